"""fp64 oracle: masked softmax attention over the union key set.

Test infrastructure only (see the package docstring).  Every function states
the passage of the paper it follows.

Conventions (readings of points the paper leaves open):

* The causal prefix of a branch includes its anchor position (keys 0..anchor).
* An EAGLE-3 chain member at depth k (0-based index k-1 in its group) sees the
  members of depths 1..k of its own chain; a DFlash block member sees every
  member of its block.  Main queries see only main keys 0..p.
* Zigzag context parallelism: each sequence is cut into 2C equal chunks and
  rank r owns chunks r and 2C-1-r.  Branch groups live on the rank owning
  their anchor.
* LSE is the natural logarithm of the sum of exponentials of scaled scores.
* Backward differentiates sum_i <dO_i, O_i>; the LSE output carries no
  gradient unless ``dlse`` is passed explicitly.
* Grouped-query attention maps query head h to key/value head h // (Hq/Hkv).

Inputs are the problem description produced by the workload generator (any
object with the same attribute names) and float arrays holding the bf16
values; they are converted to float64 here.
"""

from __future__ import annotations

import math
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

KIND_EAGLE = 0
KIND_DFLASH = 1

_ROW_BLOCK = 256  # independent query rows processed together (memory bound only)


# ----------------------------------------------------------------------
# context-parallel ownership (Sec. 3.2: packed zigzag ring, branch groups on
# the rank owning their anchor)

def owner_rank(seqlen: int, pos, cp_size: int):
    """Rank owning main position ``pos`` of a sequence of length ``seqlen``
    under the zigzag split into 2C chunks (chunk i and 2C-1-i on rank i)."""
    c = seqlen // (2 * cp_size)
    chunk = np.asarray(pos) // c
    return np.minimum(chunk, 2 * cp_size - 1 - chunk)


def select_queries(prob, rank: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Global indices of the main queries and branch query rows of one rank.

    Main token (s, p) is a query of rank r iff the sequence trains its main
    tokens and owner(p) == r; every member of a branch group is a query of the
    rank that owns the group's anchor."""
    C = prob.cp_size
    r = prob.cp_rank if rank is None else rank
    cu = np.asarray(prob.cu_seqlens, dtype=np.int64)
    main = []
    for s in range(len(cu) - 1):
        L = int(cu[s + 1] - cu[s])
        if L % (2 * C):
            raise ValueError("sequence length not divisible by 2*cp_size")
        if not prob.has_main[s]:
            continue
        p = np.arange(L)
        main.append(cu[s] + p[owner_rank(L, p, C) == r])
    br = []
    for g in range(len(prob.g_seq)):
        s = int(prob.g_seq[g])
        L = int(cu[s + 1] - cu[s])
        if int(owner_rank(L, int(prob.g_anchor[g]), C)) == r:
            br.append(np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g]))
    cat = lambda xs: np.concatenate(xs).astype(np.int64) if xs else np.zeros(0, np.int64)
    return cat(main), cat(br)


# ----------------------------------------------------------------------
# query / key descriptors of one sequence

def _branch_row_tables(prob):
    """For every global branch row: (group id, index inside the group)."""
    nb = int(np.sum(prob.g_len)) if len(prob.g_len) else 0
    gid = np.empty(nb, dtype=np.int64)
    idx = np.empty(nb, dtype=np.int64)
    for g in range(len(prob.g_seq)):
        r0, n = int(prob.g_row0[g]), int(prob.g_len[g])
        gid[r0:r0 + n] = g
        idx[r0:r0 + n] = np.arange(n)
    return gid, idx


def _sequence_problem(prob, s, main_q, br_q, br_gid, br_idx, key_filter):
    """Queries and keys of sequence s.

    Returns query descriptors (kind, prefix limit P, group, index), key
    descriptors (is_main, position or -1, group or -1, index) and the row
    indices into the global tensors."""
    cu = prob.cu_seqlens
    lo, hi = int(cu[s]), int(cu[s + 1])
    L = hi - lo
    mq = main_q[(main_q >= lo) & (main_q < hi)]
    bq = br_q[prob.g_seq[br_gid[br_q]] == s] if len(br_q) else br_q
    q_is_main = np.r_[np.ones(len(mq), bool), np.zeros(len(bq), bool)]
    q_grp = np.r_[np.full(len(mq), -1), br_gid[bq]]
    q_idx = np.r_[np.full(len(mq), -1), br_idx[bq]]
    q_P = np.r_[mq - lo, prob.g_anchor[br_gid[bq]]] if len(bq) else (mq - lo)
    q_kind = np.r_[np.full(len(mq), -1), prob.g_kind[br_gid[bq]]] if len(bq) else np.full(len(mq), -1)
    # keys: all main keys of s, then the members of every group that has a query here
    groups = np.unique(q_grp[q_grp >= 0])
    kb_rows = np.concatenate([np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g])
                              for g in groups]).astype(np.int64) if len(groups) else np.zeros(0, np.int64)
    k_pos = np.r_[np.arange(L), np.full(len(kb_rows), -1)]
    k_grp = np.r_[np.full(L, -1), br_gid[kb_rows]] if len(kb_rows) else np.full(L, -1)
    k_idx = np.r_[np.full(L, -1), br_idx[kb_rows]] if len(kb_rows) else np.full(L, -1)
    k_is_main = np.r_[np.ones(L, bool), np.zeros(len(kb_rows), bool)]
    if key_filter is not None:
        keep = key_filter(s, L, k_is_main, k_pos)
        k_use = keep
    else:
        k_use = np.ones(len(k_pos), bool)
    return dict(mq=mq, bq=bq, q_is_main=q_is_main, q_grp=q_grp, q_idx=q_idx, q_P=q_P,
                q_kind=q_kind, km_rows=np.arange(lo, hi), kb_rows=kb_rows, k_pos=k_pos,
                k_grp=k_grp, k_idx=k_idx, k_is_main=k_is_main, k_use=k_use)


def _mask(sp, qsel):
    """Allowed (query, key) pairs for the query rows ``qsel`` of one sequence.

    Main key at position j: allowed iff j <= P (P = own position for a main
    query, the anchor for a branch query).  Branch key: allowed iff it belongs
    to the query's own group and, for an EAGLE chain, its index does not
    exceed the query's index."""
    P = sp["q_P"][qsel][:, None]
    qg = sp["q_grp"][qsel][:, None]
    qi = sp["q_idx"][qsel][:, None]
    qk = sp["q_kind"][qsel][:, None]
    main_ok = sp["k_is_main"][None, :] & (sp["k_pos"][None, :] <= P)
    same = (~sp["k_is_main"][None, :]) & (sp["k_grp"][None, :] == qg) & (qg >= 0)
    chain_ok = (qk == KIND_DFLASH) | (sp["k_idx"][None, :] <= qi)
    return (main_ok | (same & chain_ok)) & sp["k_use"][None, :]


def _gather(t, rows):
    return np.asarray(t)[rows].astype(np.float64)


# ----------------------------------------------------------------------
# forward (definition of masked softmax attention; Sec. 3.2, Eq. lse-merge)

def forward(prob, qm, km, vm, qb, kb, vb, main_q=None, br_q=None, key_filter=None):
    """O and LSE of the selected queries.

    ``qm``/``km``/``vm`` are the global main tensors ``[N, H, d]``; ``qb``/``kb``
    /``vb`` the global branch tensors.  ``main_q``/``br_q`` are global row
    indices (default: the queries of ``prob.cp_rank``).  ``key_filter``
    optionally restricts the key set (used to form partial results).

    Returns ``(o_main [n_m, Hq, d], lse_main [Hq, n_m], o_br, lse_br)`` in
    float64; rows with no allowed key get O = 0 and LSE = -inf."""
    if main_q is None or br_q is None:
        mq0, bq0 = select_queries(prob)
        main_q = mq0 if main_q is None else main_q
        br_q = bq0 if br_q is None else br_q
    main_q = np.asarray(main_q, np.int64)
    br_q = np.asarray(br_q, np.int64)
    Hq, Hkv, d = prob.hq, prob.hkv, prob.head_dim
    grp = Hq // Hkv
    br_gid, br_idx = _branch_row_tables(prob)
    o_m = np.zeros((len(main_q), Hq, d))
    l_m = np.full((Hq, len(main_q)), -np.inf)
    o_b = np.zeros((len(br_q), Hq, d))
    l_b = np.full((Hq, len(br_q)), -np.inf)
    mpos = {int(v): i for i, v in enumerate(main_q)}
    bpos = {int(v): i for i, v in enumerate(br_q)}
    for s in range(len(prob.cu_seqlens) - 1):
        sp = _sequence_problem(prob, s, main_q, br_q, br_gid, br_idx, key_filter)
        nq = len(sp["q_P"])
        if nq == 0:
            continue
        Q = np.concatenate([_gather(qm, sp["mq"]), _gather(qb, sp["bq"])], axis=0)
        K = np.concatenate([_gather(km, sp["km_rows"]), _gather(kb, sp["kb_rows"])], axis=0)
        V = np.concatenate([_gather(vm, sp["km_rows"]), _gather(vb, sp["kb_rows"])], axis=0)
        mi = np.array([mpos[int(v)] for v in sp["mq"]], np.int64)
        bi = np.array([bpos[int(v)] for v in sp["bq"]], np.int64)
        nm = len(mi)
        for r0 in range(0, nq, _ROW_BLOCK):
            qsel = np.arange(r0, min(nq, r0 + _ROW_BLOCK))
            allowed = _mask(sp, qsel)
            for h in range(Hq):
                kvh = h // grp
                S = prob.scale * (Q[qsel, h, :] @ K[:, kvh, :].T)
                S = np.where(allowed, S, -np.inf)
                m = S.max(axis=1)
                finite = np.isfinite(m)
                msafe = np.where(finite, m, 0.0)
                E = np.exp(S - msafe[:, None])
                den = E.sum(axis=1)
                lse = np.where(finite, msafe + np.log(np.where(finite, den, 1.0)), -np.inf)
                P = np.where(finite[:, None], E / np.where(finite, den, 1.0)[:, None], 0.0)
                O = P @ V[:, kvh, :]
                is_m = qsel < nm
                o_m[mi[qsel[is_m]], h] = O[is_m]
                l_m[h, mi[qsel[is_m]]] = lse[is_m]
                o_b[bi[qsel[~is_m] - nm], h] = O[~is_m]
                l_b[h, bi[qsel[~is_m] - nm]] = lse[~is_m]
    return o_m, l_m, o_b, l_b


# ----------------------------------------------------------------------
# backward (chain rule of the same definition; Sec. 3.2, the ring is replayed
# and gradients are accumulated locally)

def backward(prob, qm, km, vm, qb, kb, vb, dom, dob, main_q=None, br_q=None,
             key_filter=None, dlse_main=None, dlse_br=None):
    """Gradients of sum_i <dO_i, O_i> (+ sum_i dlse_i * LSE_i if given).

    ``dom``/``dob`` are the output gradients of the selected rows (same order
    as ``main_q``/``br_q``).  Returns a dict with ``dq_main``, ``dq_br`` (rows
    of the selected queries), and ``dk_main``, ``dv_main``, ``dk_br``,
    ``dv_br`` over the global key rows (zero where no selected query reads
    the key)."""
    if main_q is None or br_q is None:
        mq0, bq0 = select_queries(prob)
        main_q = mq0 if main_q is None else main_q
        br_q = bq0 if br_q is None else br_q
    main_q = np.asarray(main_q, np.int64)
    br_q = np.asarray(br_q, np.int64)
    Hq, Hkv, d = prob.hq, prob.hkv, prob.head_dim
    grp = Hq // Hkv
    br_gid, br_idx = _branch_row_tables(prob)
    dom = np.asarray(dom, np.float64)
    dob = np.asarray(dob, np.float64)
    out = dict(dq_main=np.zeros((len(main_q), Hq, d)), dq_br=np.zeros((len(br_q), Hq, d)),
               dk_main=np.zeros((len(km), Hkv, d)), dv_main=np.zeros((len(km), Hkv, d)),
               dk_br=np.zeros((len(kb), Hkv, d)), dv_br=np.zeros((len(kb), Hkv, d)))
    mpos = {int(v): i for i, v in enumerate(main_q)}
    bpos = {int(v): i for i, v in enumerate(br_q)}
    for s in range(len(prob.cu_seqlens) - 1):
        sp = _sequence_problem(prob, s, main_q, br_q, br_gid, br_idx, key_filter)
        nq = len(sp["q_P"])
        if nq == 0:
            continue
        Q = np.concatenate([_gather(qm, sp["mq"]), _gather(qb, sp["bq"])], axis=0)
        K = np.concatenate([_gather(km, sp["km_rows"]), _gather(kb, sp["kb_rows"])], axis=0)
        V = np.concatenate([_gather(vm, sp["km_rows"]), _gather(vb, sp["kb_rows"])], axis=0)
        mi = np.array([mpos[int(v)] for v in sp["mq"]], np.int64)
        bi = np.array([bpos[int(v)] for v in sp["bq"]], np.int64)
        dO = np.concatenate([dom[mi], dob[bi]], axis=0)
        dL = None
        if dlse_main is not None or dlse_br is not None:
            dlm = np.zeros((Hq, len(main_q))) if dlse_main is None else np.asarray(dlse_main, np.float64)
            dlb = np.zeros((Hq, len(br_q))) if dlse_br is None else np.asarray(dlse_br, np.float64)
            dL = np.concatenate([dlm[:, mi], dlb[:, bi]], axis=1)  # [Hq, nq]
        dQ = np.zeros_like(Q)
        dK = np.zeros_like(K)
        dV = np.zeros_like(V)
        for r0 in range(0, nq, _ROW_BLOCK):
            qsel = np.arange(r0, min(nq, r0 + _ROW_BLOCK))
            allowed = _mask(sp, qsel)
            for h in range(Hq):
                kvh = h // grp
                S = prob.scale * (Q[qsel, h, :] @ K[:, kvh, :].T)
                S = np.where(allowed, S, -np.inf)
                m = S.max(axis=1)
                finite = np.isfinite(m)
                msafe = np.where(finite, m, 0.0)
                E = np.exp(S - msafe[:, None])
                den = np.where(finite, E.sum(axis=1), 1.0)
                P = np.where(finite[:, None], E / den[:, None], 0.0)
                O = P @ V[:, kvh, :]
                g = dO[qsel, h, :]
                delta = np.sum(g * O, axis=1)              # D_i = <dO_i, O_i>
                dP = g @ V[:, kvh, :].T                    # dP = dO V^T
                dS = P * (dP - delta[:, None])             # dS = P o (dP - D)
                if dL is not None:
                    dS = dS + P * dL[h, qsel][:, None]     # d LSE / d S = P
                dQ[qsel, h, :] += prob.scale * (dS @ K[:, kvh, :])
                dK[:, kvh, :] += prob.scale * (dS.T @ Q[qsel, h, :])
                dV[:, kvh, :] += P.T @ g
        out["dq_main"][mi] = dQ[:len(mi)]
        out["dq_br"][bi] = dQ[len(mi):]
        L = len(sp["km_rows"])
        out["dk_main"][sp["km_rows"]] += dK[:L]
        out["dv_main"][sp["km_rows"]] += dV[:L]
        if len(sp["kb_rows"]):
            np.add.at(out["dk_br"], sp["kb_rows"], dK[L:])
            np.add.at(out["dv_br"], sp["kb_rows"], dV[L:])
    return out


# ----------------------------------------------------------------------
# Eq. lse-merge and its derivative

def lse_merge(o_a, l_a, o_b, l_b):
    """Merge two partial results (Eq. lse-merge).

    ``o_*`` are ``[rows, H, d]`` normalised partial outputs, ``l_*`` their
    natural-log LSEs ``[H, rows]``.  l = log(e^la + e^lb);
    O = e^(la-l) O_a + e^(lb-l) O_b.  A partial with LSE = -inf carries zero
    weight; if both are -inf the result is (0, -inf)."""
    la = np.asarray(l_a, np.float64)
    lb = np.asarray(l_b, np.float64)
    hi = np.maximum(la, lb)
    both_empty = ~np.isfinite(hi)
    hs = np.where(both_empty, 0.0, hi)
    ea = np.where(np.isfinite(la), np.exp(la - hs), 0.0)
    eb = np.where(np.isfinite(lb), np.exp(lb - hs), 0.0)
    tot = ea + eb
    l = np.where(both_empty, -np.inf, hs + np.log(np.where(both_empty, 1.0, tot)))
    wa = np.where(both_empty, 0.0, ea / np.where(both_empty, 1.0, tot))
    wb = np.where(both_empty, 0.0, eb / np.where(both_empty, 1.0, tot))
    o = wa.T[:, :, None] * np.asarray(o_a, np.float64) + wb.T[:, :, None] * np.asarray(o_b, np.float64)
    return o, l


def lse_merge_backward(o_a, l_a, o_b, l_b, d_o):
    """Upstream gradients of the two partials given dO of the merged output
    (the merged LSE itself receives no gradient).  With w_x = e^(lx - l):
    dO_x = w_x dO and dl_x = w_x (<dO, O_x> - <dO, O>)."""
    o, l = lse_merge(o_a, l_a, o_b, l_b)
    out = []
    for ox, lx in ((o_a, l_a), (o_b, l_b)):
        lx = np.asarray(lx, np.float64)
        w = np.where(np.isfinite(lx), np.exp(lx - np.where(np.isfinite(l), l, 0.0)), 0.0)  # [H, rows]
        dox = w.T[:, :, None] * d_o
        dlx = w * (np.sum(d_o * np.asarray(ox, np.float64), axis=2).T - np.sum(d_o * o, axis=2).T)
        out.append((dox, dlx))
    return out


# ----------------------------------------------------------------------
# counting (Sec. 4.4 workloads; useful work = allowed pairs)

def allowed_pair_counts(prob, main_q=None, br_q=None, key_filter=None):
    """Number of allowed (query, key) pairs per query head, split into the
    main-prefix part and the branch-local part, counted from the mask."""
    if main_q is None or br_q is None:
        main_q, br_q = select_queries(prob)
    br_gid, br_idx = _branch_row_tables(prob)
    n_main = n_local = 0
    for s in range(len(prob.cu_seqlens) - 1):
        sp = _sequence_problem(prob, s, np.asarray(main_q), np.asarray(br_q), br_gid, br_idx,
                               key_filter)
        nq = len(sp["q_P"])
        for r0 in range(0, nq, _ROW_BLOCK):
            qsel = np.arange(r0, min(nq, r0 + _ROW_BLOCK))
            a = _mask(sp, qsel)
            n_main += int(a[:, sp["k_is_main"]].sum())
            n_local += int(a[:, ~sp["k_is_main"]].sum())
    return n_main, n_local


def useful_flops(prob, pairs_per_head: int):
    """Useful FLOPs: 4d per allowed pair and query head forward (QK^T, PV),
    10d backward (QK^T recompute, dP, dV, dK, dQ)."""
    d = prob.head_dim
    return 4.0 * d * prob.hq * pairs_per_head, 10.0 * d * prob.hq * pairs_per_head
