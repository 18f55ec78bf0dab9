"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.

The fp64 oracle cannot afford every row at these sizes, so:
* sampled query rows (main and branch, spread over the rank's chunks and the
  branch depths) are recomputed by the oracle against all their keys: O and
  LSE of a row, and dQ of a row, depend on that row alone;
* dK and dV are checked through identities that hold at any size, per KV
  head, over the whole tensors (every main block and the branch keys):
    sum_k dV_k = sum over queries and the head's query heads of dO   (rows of P sum to 1)
    sum_k dK_k = 0                                                   (rows of dS sum to 0)
    sum_q <dQ_q, q_q> = sum_k <dK_k, k_k>                            (both equal scale sum dS o S)
  computed in fp64 from the fp32 gradients the library returns.

Tolerances: O 2e-2 max-abs and LSE 1e-3 max-abs (bf16 output vs fp64), dQ
rows 1e-2 relative L2; the identities are compared with a relative 5e-3 on
the dV sum, 2e-2 of the dK Frobenius norm for the dK sum, and 1e-2 on the
inner-product balance -- all far below what a wrong mask, a dropped ring
step or a transposed operand produces (order 1).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

# (config, schedule, sampled main rows, sampled branch rows); every workload
# runs in both schedules, the per-step one being the benchmark's launch
# configuration
CASES = [(2, "per_step", 4, 8), (2, "fused", 2, 4), (3, "per_step", 4, 8), (3, "fused", 4, 8),
         (4, "per_step", 12, 24), (4, "fused", 4, 8), (5, "per_step", 4, 8), (5, "fused", 4, 8)]


def sample_rows(prob, mq, bq, n_main=4, n_br=8, seed=0):
    """Spread the sample over both chunks of the rank and over branch depths."""
    rng = np.random.default_rng(seed)
    sm = np.sort(rng.choice(mq, size=min(n_main, len(mq)), replace=False)) if len(mq) else mq[:0]
    if len(mq) >= 2:
        sm = np.unique(np.r_[sm, mq[0], mq[-1]])  # first and last position of the share
    sb = np.sort(rng.choice(bq, size=min(n_br, len(bq)), replace=False)) if len(bq) else bq[:0]
    return sm, sb


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    return torch.device("cuda:0")


@pytest.mark.parametrize("cfg,mode,n_main,n_br", CASES)
def test_fullsize_sampled_rows_and_gradient_identities(cuda, cfg, mode, n_main, n_br):
    prob = W.config(cfg)
    md = B.BA_MODE_FUSED if mode == "fused" else B.BA_MODE_PER_STEP
    share = RS.build_share(prob, device="cuda:0", with_grad=True)
    out = RS.alloc_outputs(share, grads=True, grad_dtype=torch.float32)
    ws = RS.workspace(share, md, backward=True)
    RS.run_fwd(share, out, md, ws)
    RS.run_bwd(share, out, md, ws)
    torch.cuda.synchronize()
    print(f"[fullsize] config {cfg} ({prob.name}) {mode}: GPU done", flush=True)

    # ---- sampled rows against the oracle
    mq, bq = oracle.select_queries(prob)
    sm, sb = sample_rows(prob, mq, bq, n_main=n_main, n_br=n_br, seed=cfg)
    H_, Hk, d = prob.hq, prob.hkv, prob.head_dim

    def sparse(name, sel, total, heads):
        a = np.zeros((total, heads, d), np.float32)
        if len(sel):
            a[sel] = prob.draw(name, sel).float().numpy()
        return a

    grp = np.repeat(np.arange(len(prob.g_len)), prob.g_len)
    gsel = np.unique(grp[sb]) if len(sb) else np.zeros(0, np.int64)
    brows = np.concatenate([np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g]) for g in gsel]) \
        if len(gsel) else np.zeros(0, np.int64)
    t = dict(qm=sparse("qm", sm, prob.n_main, H_), qb=sparse("qb", sb, prob.n_branch, H_),
             km=prob.draw("km").float().numpy(), vm=prob.draw("vm").float().numpy(),
             kb=sparse("kb", brows, prob.n_branch, Hk), vb=sparse("vb", brows, prob.n_branch, Hk))
    args = [t[k] for k in ("qm", "km", "vm", "qb", "kb", "vb")]
    ref_f = oracle.forward(prob, *args, sm, sb)
    dom = prob.draw("dom", sm).float().numpy() if len(sm) else np.zeros((0, H_, d), np.float32)
    dob = prob.draw("dob", sb).float().numpy() if len(sb) else np.zeros((0, H_, d), np.float32)
    ref_b = oracle.backward(prob, *args, dom, dob, sm, sb)
    print(f"[fullsize] oracle done on {len(sm)} main + {len(sb)} branch rows", flush=True)

    g2l = {int(g): i for i, g in enumerate(share.l2g)}
    mi = np.array([g2l[int(g)] for g in sm], np.int64)
    bmap = {int(g): int(l) for g, l in zip(share.br_rows_global, share.br_rows_local)}
    bi = np.array([bmap[int(g)] for g in sb], np.int64)
    f = lambda x, idx: x[torch.from_numpy(idx).to(x.device)].float().cpu().numpy().astype(np.float64)
    got_f = (f(out["o_main"], mi), f(out["lse_main"].T, mi).T, f(out["o_br"], bi), f(out["lse_br"].T, bi).T)
    H.assert_fwd_close(got_f, ref_f)
    dq = np.concatenate([f(out["dq_main"], mi).ravel(), f(out["dq_br"], bi).ravel()])
    dq_ref = np.concatenate([ref_b["dq_main"].ravel(), ref_b["dq_br"].ravel()])
    e = H.rel_l2(dq, dq_ref)
    assert e <= H.GRAD_TOL, f"sampled dQ rows: relative L2 {e:.3e}"

    # ---- identities over the whole gradient tensors (fp64 on the GPU)
    G = H_ // Hk
    dev = cuda
    q_rows = torch.cat([share.t["q_main"][torch.from_numpy(share.main_query_rows).to(dev)],
                        share.t["q_br"][torch.from_numpy(share.br_rows_local).to(dev)]]).double()
    do_rows = torch.cat([share.t["do_main"][torch.from_numpy(share.main_query_rows).to(dev)],
                         share.t["do_br"][torch.from_numpy(share.br_rows_local).to(dev)]]).double()
    dq_rows = torch.cat([out["dq_main"][torch.from_numpy(share.main_query_rows).to(dev)],
                         out["dq_br"][torch.from_numpy(share.br_rows_local).to(dev)]]).double()
    br_idx = torch.from_numpy(share.br_rows_local).to(dev)
    dk_all = torch.cat([x.double() for x in out["dk_step"]] + [out["dk_br"][br_idx].double()])
    dv_all = torch.cat([x.double() for x in out["dv_step"]] + [out["dv_br"][br_idx].double()])
    k_all = torch.cat([x.double() for x in share.t["k_step"]] + [share.t["k_br"][br_idx].double()])

    sum_dv = dv_all.sum(0)                                      # [Hk, d]
    sum_do = do_rows.view(-1, Hk, G, d).sum((0, 2))             # [Hk, d]
    e1 = (sum_dv - sum_do).norm() / sum_do.norm()
    sum_dk = dk_all.sum(0)
    e2 = sum_dk.norm() / dk_all.norm()
    lhs = (dq_rows * q_rows).view(-1, Hk, G, d).sum((0, 2, 3))  # per KV head
    rhs = (dk_all * k_all).sum((0, 2))
    e3 = ((lhs - rhs).abs() / (dq_rows * q_rows).abs().view(-1, Hk, G, d).sum((0, 2, 3))).max()
    print(f"[fullsize] identities: dV sum {e1.item():.2e}, dK sum {e2.item():.2e}, "
          f"<dQ,Q>=<dK,K> {e3.item():.2e}", flush=True)
    assert e1 <= 5e-3, f"sum_k dV_k != sum dO: {e1.item():.3e}"
    assert e2 <= 2e-2, f"sum_k dK_k != 0: {e2.item():.3e}"
    assert e3 <= 1e-2, f"<dQ,Q> != <dK,K>: {e3.item():.3e}"


def test_fullsize_headline_with_rotary_embedding(cuda):
    """The headline share with rotary embedding (theta 5e5, positions up to
    262143, so angles of ~2.6e5 rad): sampled rows against `oracle.rope`
    (rotated queries and keys rounded to bf16), plus the two identities that
    survive the rotation: sum_k dV_k = sum dO (values are not rotated) and
    sum_q <dQ_q, q_q> = sum_k <dK_k, k_k> (the rotation is orthogonal)."""
    from oracle import rope

    theta = 5.0e5
    prob = W.config(4)
    md = B.BA_MODE_PER_STEP
    share = RS.build_share(prob, device="cuda:0", with_grad=True, rope_theta=theta)
    out = RS.alloc_outputs(share, grads=True, grad_dtype=torch.float32)
    ws = RS.workspace(share, md, backward=True)
    RS.run_fwd(share, out, md, ws)
    RS.run_bwd(share, out, md, ws)
    torch.cuda.synchronize()
    print("[fullsize] config 4 with rotary embedding: GPU done", flush=True)

    mq, bq = oracle.select_queries(prob)
    sm, sb = sample_rows(prob, mq, bq, n_main=6, n_br=12, seed=44)
    H_, Hk, d = prob.hq, prob.hkv, prob.head_dim

    def sparse(name, sel, total, heads):
        a = np.zeros((total, heads, d), np.float32)
        if len(sel):
            a[sel] = prob.draw(name, sel).float().numpy()
        return a

    grp = np.repeat(np.arange(len(prob.g_len)), prob.g_len)
    gsel = np.unique(grp[sb]) if len(sb) else np.zeros(0, np.int64)
    brows = np.concatenate([np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g]) for g in gsel]) \
        if len(gsel) else np.zeros(0, np.int64)
    t = dict(qm=sparse("qm", sm, prob.n_main, H_), qb=sparse("qb", sb, prob.n_branch, H_),
             km=prob.draw("km").float().numpy(), vm=prob.draw("vm").float().numpy(),
             kb=sparse("kb", brows, prob.n_branch, Hk), vb=sparse("vb", brows, prob.n_branch, Hk))
    args = [t[k] for k in ("qm", "km", "vm", "qb", "kb", "vb")]
    ref_f = rope.forward(prob, *args, theta, rounded=True, main_q=sm, br_q=sb)
    dom = prob.draw("dom", sm).float().numpy()
    dob = prob.draw("dob", sb).float().numpy()
    ref_b = rope.backward(prob, *args, dom, dob, theta, main_q=sm, br_q=sb, rounded=True)
    print(f"[fullsize] rotary oracle done on {len(sm)} main + {len(sb)} branch rows", flush=True)

    g2l = {int(g): i for i, g in enumerate(share.l2g)}
    mi = np.array([g2l[int(g)] for g in sm], np.int64)
    bmap = {int(g): int(l) for g, l in zip(share.br_rows_global, share.br_rows_local)}
    bi = np.array([bmap[int(g)] for g in sb], np.int64)
    f = lambda x, idx: x[torch.from_numpy(idx).to(x.device)].float().cpu().numpy().astype(np.float64)
    got_f = (f(out["o_main"], mi), f(out["lse_main"].T, mi).T, f(out["o_br"], bi), f(out["lse_br"].T, bi).T)
    H.assert_fwd_close(got_f, ref_f)
    dq = np.concatenate([f(out["dq_main"], mi).ravel(), f(out["dq_br"], bi).ravel()])
    dq_ref = np.concatenate([ref_b["dq_main"].ravel(), ref_b["dq_br"].ravel()])
    e = H.rel_l2(dq, dq_ref)
    assert e <= H.GRAD_TOL, f"sampled dQ rows: relative L2 {e:.3e}"

    G = H_ // Hk
    dev = cuda
    mrows = torch.from_numpy(share.main_query_rows).to(dev)
    br_idx = torch.from_numpy(share.br_rows_local).to(dev)
    q_rows = torch.cat([share.t["q_main"][mrows], share.t["q_br"][br_idx]]).double()
    do_rows = torch.cat([share.t["do_main"][mrows], share.t["do_br"][br_idx]]).double()
    dq_rows = torch.cat([out["dq_main"][mrows], out["dq_br"][br_idx]]).double()
    dk_all = torch.cat([x.double() for x in out["dk_step"]] + [out["dk_br"][br_idx].double()])
    dv_all = torch.cat([x.double() for x in out["dv_step"]] + [out["dv_br"][br_idx].double()])
    k_all = torch.cat([x.double() for x in share.t["k_step"]] + [share.t["k_br"][br_idx].double()])
    sum_do = do_rows.view(-1, Hk, G, d).sum((0, 2))
    e1 = (dv_all.sum(0) - sum_do).norm() / sum_do.norm()
    lhs = (dq_rows * q_rows).view(-1, Hk, G, d).sum((0, 2, 3))
    rhs = (dk_all * k_all).sum((0, 2))
    e3 = ((lhs - rhs).abs() / (dq_rows * q_rows).abs().view(-1, Hk, G, d).sum((0, 2, 3))).max()
    print(f"[fullsize] rotary identities: dV sum {e1.item():.2e}, <dQ,Q>=<dK,K> {e3.item():.2e}", flush=True)
    assert e1 <= 5e-3, f"sum_k dV_k != sum dO: {e1.item():.3e}"
    assert e3 <= 1e-2, f"<dQ,Q> != <dK,K>: {e3.item():.3e}"
