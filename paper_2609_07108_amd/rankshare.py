"""Lay out one context-parallel rank share in the library's input format.

In a real context-parallel run the data already sits on each rank in this
layout; here it is cut out of a global synthetic problem
(:mod:`paper_2609_07108_amd.workloads`) using the library's own
``zigzag_partition`` for every rank.  No attention arithmetic happens here:
rows are selected and copied, and the branch-anchor descriptors are written.

Branch-array layouts
  "group": members of each group are consecutive rows (row_stride 1).
  "depth": EAGLE-3 chains depth-major -- member i of the chain anchored at
           rank-local main row u sits at row i * n_local + u -- followed by the
           DFlash blocks, consecutive.  Rows without a member are left unused.
"""

from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np
import torch

from . import binding as B
from .workloads import KIND_DFLASH, KIND_EAGLE, GlobalProblem


@dataclasses.dataclass
class RankShare:
    prob: GlobalProblem
    plan: B.Plan
    n_local: int
    local_cu: np.ndarray
    l2g: np.ndarray                 # rank-local main row -> global main row (this rank)
    l2g_steps: List[np.ndarray]     # same for every rank j (the ring-step blocks)
    groups: np.ndarray              # [n_groups, 6] descriptors handed to the library
    group_global: np.ndarray        # global group id of each local group
    br_rows_local: np.ndarray       # local branch row of every member, in global-row order of br_rows_global
    br_rows_global: np.ndarray      # global branch row of every member
    num_branch_rows: int
    main_query_rows: np.ndarray     # rank-local main rows that are queries
    t: dict                         # device tensors


def _layout_groups(prob: GlobalProblem, r: int, l2g: np.ndarray, layout: str):
    n_local = len(l2g)
    # a group belongs to this rank iff its anchor's main token is one of the rank's tokens
    g_pos = prob.cu_seqlens[prob.g_seq] + prob.g_anchor if len(prob.g_seq) else np.zeros(0, np.int64)
    order = np.argsort(l2g, kind="stable")
    sorted_l2g = np.asarray(l2g, np.int64)[order]
    idx = np.searchsorted(sorted_l2g, g_pos)
    hit = (idx < len(sorted_l2g)) & (sorted_l2g[np.minimum(idx, len(sorted_l2g) - 1)] == g_pos) \
        if len(sorted_l2g) else np.zeros(len(g_pos), bool)
    sel = np.flatnonzero(hit).astype(np.int64)
    anchor_local = order[idx[hit]] if len(sel) else np.zeros(0, np.int64)
    desc, loc_rows, glob_rows = [], [], []
    if layout == "group":
        lens = prob.g_len[sel]
        row0 = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64) if len(sel) else lens
        desc = np.stack([prob.g_seq[sel], prob.g_anchor[sel], prob.g_kind[sel], lens, row0,
                         np.ones(len(sel), np.int64)], axis=1) if len(sel) else np.zeros((0, 6))
        member = np.arange(int(lens.sum())) - np.repeat(row0, lens) if len(sel) else np.zeros(0, np.int64)
        loc = np.arange(int(lens.sum()), dtype=np.int64)
        glob = np.repeat(prob.g_row0[sel], lens) + member if len(sel) else loc
        return (np.asarray(desc, np.int32).reshape(-1, 6), sel, loc, glob.astype(np.int64), int(lens.sum()))
    glob_to_local = {int(g): int(u) for g, u in zip(g_pos[sel], anchor_local)}
    if layout == "depth":
        eag = [g for g in sel if prob.g_kind[g] == KIND_EAGLE]
        kmax = max([int(prob.g_len[g]) for g in eag], default=0)
        row = kmax * n_local
        for g in sel:
            n = int(prob.g_len[g])
            if prob.g_kind[g] == KIND_EAGLE:
                u = glob_to_local[int(prob.cu_seqlens[prob.g_seq[g]]) + int(prob.g_anchor[g])]
                desc.append((int(prob.g_seq[g]), int(prob.g_anchor[g]), KIND_EAGLE, n, u, n_local))
                loc_rows.append(u + n_local * np.arange(n))
            else:
                desc.append((int(prob.g_seq[g]), int(prob.g_anchor[g]), int(prob.g_kind[g]), n, row, 1))
                loc_rows.append(np.arange(row, row + n))
                row += n
            glob_rows.append(np.arange(prob.g_row0[g], prob.g_row0[g] + n))
        nrows = row
    else:
        raise ValueError(layout)
    cat = lambda xs: np.concatenate(xs).astype(np.int64) if xs else np.zeros(0, np.int64)
    return (np.asarray(desc, np.int32).reshape(-1, 6), sel, cat(loc_rows), cat(glob_rows), nrows)


def build_share(prob: GlobalProblem, device: str = "cuda", layout: str = "group",
                with_grad: Optional[bool] = None, zero_q: bool = False,
                materialize: bool = True, rope_theta: float = 0.0) -> RankShare:
    C, r = prob.cp_size, prob.cp_rank
    cu = prob.cu_seqlens.astype(np.int32)
    lcu, l2g, lpos = B.zigzag_partition(cu, C, r)
    l2g_steps = [B.zigzag_partition(cu, C, j)[1] for j in range(C)]
    n_local = len(l2g)
    desc, gsel, loc_rows, glob_rows, nrows = _layout_groups(prob, r, l2g, layout)
    plan = B.Plan(cu, prob.has_main.astype(np.uint8), C, r, prob.hq, prob.hkv, prob.head_dim,
                  prob.scale, desc, nrows)
    if rope_theta:
        plan.set_rope(rope_theta)
    seq_of_local = np.searchsorted(lcu, np.arange(n_local), side="right") - 1
    mq_rows = np.flatnonzero(prob.has_main[seq_of_local]) if n_local else np.zeros(0, np.int64)
    share = RankShare(prob=prob, plan=plan, n_local=n_local, local_cu=lcu, l2g=l2g, l2g_steps=l2g_steps,
                      groups=desc, group_global=gsel, br_rows_local=loc_rows, br_rows_global=glob_rows,
                      num_branch_rows=nrows, main_query_rows=mq_rows, t={})
    if not materialize:
        return share
    with_grad = prob.backward if with_grad is None else with_grad
    H, Hk, d = prob.hq, prob.hkv, prob.head_dim
    dev = torch.device(device)

    def branch(name, heads):
        out = torch.zeros((max(nrows, 1), heads, d), dtype=torch.bfloat16)
        if len(glob_rows):
            out[torch.from_numpy(loc_rows)] = prob.draw(name, glob_rows, zero=(zero_q and name == "qb"))
        return out.to(dev)

    t = share.t
    t["q_main"] = prob.draw("qm", l2g.astype(np.int64), zero=zero_q).to(dev)
    km_all = prob.draw("km")
    vm_all = prob.draw("vm")
    t["k_step"] = [km_all[torch.from_numpy(l2g_steps[j].astype(np.int64))].to(dev) for j in range(C)]
    t["v_step"] = [vm_all[torch.from_numpy(l2g_steps[j].astype(np.int64))].to(dev) for j in range(C)]
    del km_all, vm_all
    t["q_br"] = branch("qb", H)
    t["k_br"] = branch("kb", Hk)
    t["v_br"] = branch("vb", Hk)
    if with_grad:
        t["do_main"] = prob.draw("dom", l2g.astype(np.int64)).to(dev)
        t["do_br"] = branch("dob", H)
    return share


def alloc_outputs(share: RankShare, grads: bool = False, grad_dtype=torch.bfloat16):
    """Output buffers of one call (fwd, or fwd + bwd)."""
    p = share.prob
    dev = share.t["q_main"].device
    H, Hk, d = p.hq, p.hkv, p.head_dim
    nl, nb = max(share.n_local, 1), max(share.num_branch_rows, 1)
    out = dict(o_main=torch.zeros((nl, H, d), dtype=torch.bfloat16, device=dev),
               o_br=torch.zeros((nb, H, d), dtype=torch.bfloat16, device=dev),
               lse_main=torch.zeros((H, nl), dtype=torch.float32, device=dev),
               lse_br=torch.zeros((H, nb), dtype=torch.float32, device=dev))
    if grads:
        out.update(dq_main=torch.zeros((nl, H, d), dtype=grad_dtype, device=dev),
                   dq_br=torch.zeros((nb, H, d), dtype=grad_dtype, device=dev),
                   dk_step=[torch.zeros((nl, Hk, d), dtype=grad_dtype, device=dev) for _ in range(p.cp_size)],
                   dv_step=[torch.zeros((nl, Hk, d), dtype=grad_dtype, device=dev) for _ in range(p.cp_size)],
                   dk_br=torch.zeros((nb, Hk, d), dtype=grad_dtype, device=dev),
                   dv_br=torch.zeros((nb, Hk, d), dtype=grad_dtype, device=dev))
    return out


def workspace(share: RankShare, mode: int, backward: bool = False):
    f, b = share.plan.workspace_size(mode)
    n = max(f, b if backward else 0, 256)
    return torch.empty(n, dtype=torch.uint8, device=share.t["q_main"].device)


def run_fwd(share: RankShare, out: dict, mode: int, ws, ring_events=(None, None)):
    t = share.t
    B.branch_attn_fwd(share.plan, mode, t["q_main"], t["q_br"], t["k_br"], t["v_br"], t["k_step"],
                      t["v_step"], out["o_main"], out["o_br"], out["lse_main"], out["lse_br"], ws,
                      ring_events=ring_events)


def run_bwd(share: RankShare, out: dict, mode: int, ws, ring_events=(None, None)):
    t = share.t
    gd = B.BA_DTYPE_F32 if out["dq_main"].dtype == torch.float32 else B.BA_DTYPE_BF16
    B.branch_attn_bwd(share.plan, mode, t["q_main"], t["q_br"], t["k_br"], t["v_br"], t["k_step"],
                      t["v_step"], out["o_main"], out["o_br"], out["lse_main"], out["lse_br"],
                      t["do_main"], t["do_br"], out["dq_main"], out["dq_br"], out["dk_step"],
                      out["dv_step"], out["dk_br"], out["dv_br"], gd, ws, ring_events=ring_events)
