"""Shared plumbing of the GPU parity tests: run the HIP path through the C ABI
on a rank share and line its outputs up with the oracle's rows.

Tolerances (bf16 inputs, fp32 accumulation, bf16 outputs; the fp64 oracle
reads the same bf16 values):
  O      max |gpu - ref| <= 2e-2
  LSE    max |gpu - ref| <= 1e-3
  dQ, dK, dV  ||gpu - ref||_2 / ||ref||_2 <= 1e-2 (whole tensor, main and
              branch rows concatenated)
"""

import numpy as np
import torch

import oracle
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS

O_TOL = 2e-2
LSE_TOL = 1e-3
GRAD_TOL = 1e-2

TENSORS = ("qm", "km", "vm", "qb", "kb", "vb")


def oracle_inputs(prob, zero_q=False):
    t = {k: prob.draw(k, zero=(zero_q and k in ("qm", "qb"))).float().numpy().astype(np.float64)
         for k in TENSORS}
    if prob.backward:
        t["dom"] = prob.draw("dom").float().numpy().astype(np.float64)
        t["dob"] = prob.draw("dob").float().numpy().astype(np.float64)
    return t


def oracle_run(prob, t, backward=True):
    mq, bq = oracle.select_queries(prob)
    args = [t[k] for k in TENSORS]
    fwd = oracle.forward(prob, *args, mq, bq)
    bwd = None
    if backward:
        bwd = oracle.backward(prob, *args, t["dom"][mq], t["dob"][bq], mq, bq)
    return mq, bq, fwd, bwd


def _maps(share, mq, bq):
    g2l = {int(g): i for i, g in enumerate(share.l2g)}
    mi = np.array([g2l[int(g)] for g in mq], np.int64)
    bmap = {int(g): int(l) for g, l in zip(share.br_rows_global, share.br_rows_local)}
    bi = np.array([bmap[int(g)] for g in bq], np.int64)
    return mi, bi


def gpu_fwd(share, mode, mq, bq, out=None, ws=None):
    out = RS.alloc_outputs(share) if out is None else out
    ws = RS.workspace(share, mode) if ws is None else ws
    RS.run_fwd(share, out, mode, ws)
    torch.cuda.synchronize()
    mi, bi = _maps(share, mq, bq)
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    return (f(out["o_main"])[mi], f(out["lse_main"])[:, mi], f(out["o_br"])[bi], f(out["lse_br"])[:, bi]), out


def gpu_bwd(share, mode, mq, bq, grad_dtype=torch.bfloat16):
    out = RS.alloc_outputs(share, grads=True, grad_dtype=grad_dtype)
    ws = RS.workspace(share, mode, backward=True)
    RS.run_fwd(share, out, mode, ws)
    RS.run_bwd(share, out, mode, ws)
    torch.cuda.synchronize()
    mi, bi = _maps(share, mq, bq)
    f = lambda x: x.float().cpu().numpy().astype(np.float64)
    p = share.prob
    g = dict(dq_main=f(out["dq_main"])[mi], dq_br=f(out["dq_br"])[bi])
    n = p.n_main
    dk = np.zeros((n, p.hkv, p.head_dim))
    dv = np.zeros((n, p.hkv, p.head_dim))
    for j in range(p.cp_size):
        rows = share.l2g_steps[j].astype(np.int64)
        dk[rows] = f(out["dk_step"][j])[:len(rows)]
        dv[rows] = f(out["dv_step"][j])[:len(rows)]
    g["dk_main"], g["dv_main"] = dk, dv
    nb = p.n_branch
    dkb = np.zeros((nb, p.hkv, p.head_dim))
    dvb = np.zeros((nb, p.hkv, p.head_dim))
    if len(share.br_rows_global):
        dkb[share.br_rows_global] = f(out["dk_br"])[share.br_rows_local]
        dvb[share.br_rows_global] = f(out["dv_br"])[share.br_rows_local]
    g["dk_br"], g["dv_br"] = dkb, dvb
    fw = (f(out["o_main"])[mi], f(out["lse_main"])[:, mi], f(out["o_br"])[bi], f(out["lse_br"])[:, bi])
    return fw, g, out


def assert_fwd_close(gpu, ref, o_tol=O_TOL, lse_tol=LSE_TOL):
    names = ("o_main", "lse_main", "o_br", "lse_br")
    for name, a, b in zip(names, gpu, ref):
        if b.size == 0:
            continue
        assert np.all(np.isfinite(a)), f"{name}: non-finite values"
        err = np.max(np.abs(a - b))
        tol = o_tol if name.startswith("o_") else lse_tol
        assert err <= tol, f"{name}: max abs error {err:.3e} > {tol}"


def rel_l2(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def assert_bwd_close(gpu, ref, tol=GRAD_TOL):
    pairs = {"dQ": ("dq_main", "dq_br"), "dK": ("dk_main", "dk_br"), "dV": ("dv_main", "dv_br")}
    for name, (m, b) in pairs.items():
        a = np.concatenate([gpu[m].ravel(), gpu[b].ravel()])
        r = np.concatenate([ref[m].ravel(), ref[b].ravel()])
        assert np.all(np.isfinite(a)), f"{name}: non-finite values"
        e = rel_l2(a, r)
        assert e <= tol, f"{name}: relative L2 error {e:.3e} > {tol}"
        # stricter than the bar: the main and the branch part each on its own,
        # so a wrong branch-local gradient cannot hide under the main one
        for part in (m, b):
            if gpu[part].size and np.linalg.norm(ref[part]) > 0:
                e = rel_l2(gpu[part].ravel(), ref[part].ravel())
                assert e <= tol, f"{name} ({part}): relative L2 error {e:.3e} > {tol}"
