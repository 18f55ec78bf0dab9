"""The draft layer's attention block end to end on the GPU: grouped-query QKV
projection with rotary embedding (branch_attn_qkv_fwd), branch attention of
one rank share with the plan's own rotation off (branch_attn_fwd / _bwd),
and the projection's backward (branch_attn_qkv_bwd) fed with the attention's
gradients, against the same chain in the fp64 oracle: `oracle.qkv.forward`,
rounding of q / k / v to bf16 (`oracle.rope.round_bf16`), `oracle.forward`
/ `oracle.backward`, `oracle.qkv.backward`.

The rank share's ring blocks are projected the way their owners would:
block j from rank j's local rows with rank j's positions (taken from a plan
of rank j), the branch rows from the rank's branch arrays with the plan's
branch positions.  The weight gradient sums the contributions of every
block and of the branch rows (accumulated in place).  Tolerances: O max-abs
2e-2; dx (main and branch rows) and dw relative L2 1e-2.
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import qkv as OQ
from oracle import rope
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    return torch.device("cuda:0")


def bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16)


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_l2(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)


@pytest.mark.parametrize("mode,grad_dtype", [("per_step", torch.bfloat16), ("fused", torch.float32)])
def test_projection_attention_chain(cuda, mode, grad_dtype):
    prob = W.custom([512, 256], [("eagle", 3), ("dflash", 8, 32)], hq=4, hkv=2, cp_size=2, cp_rank=1, seed=501,
                    name="draft-layer")
    hidden, theta, d = 256, 1.0e4, 128
    hq, hkv = prob.hq, prob.hkv
    n = (hq + 2 * hkv) * d
    C, r = prob.cp_size, prob.cp_rank
    rng = np.random.default_rng(502)
    xm = bf16(rng.standard_normal((prob.n_main, hidden)))
    xb = bf16(rng.standard_normal((prob.n_branch, hidden)))
    w = bf16(rng.standard_normal((n, hidden)) / np.sqrt(hidden))
    dom = bf16(rng.standard_normal((prob.n_main, hq, d)))
    dob = bf16(rng.standard_normal((prob.n_branch, hq, d)))
    dev = "cuda"
    print(f"[draft layer] {mode} grads {grad_dtype}", flush=True)

    # ---- GPU: projection of every ring block by its owner, then attention
    share = RS.build_share(prob, materialize=False)
    nl, nb = share.n_local, share.num_branch_rows
    wd = w.to(dev)

    def project(x, pos):
        rows = x.shape[0]
        q = torch.empty((rows, hq, d), dtype=torch.bfloat16, device=dev)
        k = torch.empty((rows, hkv, d), dtype=torch.bfloat16, device=dev)
        v = torch.empty_like(k)
        B.branch_attn_qkv_fwd(x, wd, hq, hkv, torch.as_tensor(pos, dtype=torch.int32, device=dev), theta, q, k, v)
        return q, k, v

    blocks = []
    for j in range(C):
        sj = RS.build_share(prob.with_rank(j), materialize=False)
        pos_j, _ = sj.plan.positions(sj.n_local, sj.num_branch_rows)
        rows_j = torch.as_tensor(sj.l2g.astype(np.int64))
        assert np.array_equal(sj.l2g, share.l2g_steps[j])
        x_j = xm[rows_j].to(dev)
        blocks.append((x_j, pos_j) + project(x_j, pos_j))
    mp, bp = share.plan.positions(nl, nb)
    x_br = torch.zeros((max(nb, 1), hidden), dtype=torch.bfloat16)
    x_br[torch.as_tensor(share.br_rows_local)] = xb[torch.as_tensor(share.br_rows_global)]
    x_br = x_br.to(dev)
    bp_full = np.full(max(nb, 1), -1, np.int64)
    bp_full[:nb] = bp
    q_br, k_br, v_br = project(x_br, bp_full)
    share.t.update(q_main=blocks[r][2], k_step=[b[3] for b in blocks], v_step=[b[4] for b in blocks],
                   q_br=q_br, k_br=k_br, v_br=v_br, do_main=dom[torch.as_tensor(share.l2g.astype(np.int64))].to(dev))
    do_br = torch.zeros((max(nb, 1), hq, d), dtype=torch.bfloat16)
    do_br[torch.as_tensor(share.br_rows_local)] = dob[torch.as_tensor(share.br_rows_global)]
    share.t["do_br"] = do_br.to(dev)
    bmode = B.BA_MODE_FUSED if mode == "fused" else B.BA_MODE_PER_STEP
    out = RS.alloc_outputs(share, grads=True, grad_dtype=grad_dtype)
    ws = RS.workspace(share, bmode, backward=True)
    RS.run_fwd(share, out, bmode, ws)
    RS.run_bwd(share, out, bmode, ws)

    # ---- GPU: the projection's backward over every block and the branch rows
    dw = torch.empty((n, hidden), dtype=torch.float32, device=dev)
    dx_blocks = []
    pws = torch.empty(max(B.branch_attn_qkv_workspace_size(max(nl, nb, 1), hq, hkv), 256), dtype=torch.uint8,
                      device=dev)
    for j, (x_j, pos_j, *_rest) in enumerate(blocks):
        dq_j = out["dq_main"] if j == r else torch.zeros_like(out["dq_main"])
        dx_j = torch.empty((x_j.shape[0], hidden), dtype=torch.float32, device=dev)
        B.branch_attn_qkv_bwd(x_j, wd, hq, hkv, torch.as_tensor(pos_j, dtype=torch.int32, device=dev), theta,
                              dq_j, out["dk_step"][j], out["dv_step"][j], dx_j, dw, j > 0, pws)
        dx_blocks.append(dx_j)
    dx_br = torch.empty((x_br.shape[0], hidden), dtype=torch.float32, device=dev)
    B.branch_attn_qkv_bwd(x_br, wd, hq, hkv, torch.as_tensor(bp_full, dtype=torch.int32, device=dev), theta,
                          out["dq_br"], out["dk_br"], out["dv_br"], dx_br, dw, True, pws)
    torch.cuda.synchronize()

    # ---- oracle: the same chain in float64
    pm_g, pb_g = rope.positions(prob, prob.n_branch)
    xm64, xb64, w64 = f64(xm), f64(xb), f64(w)
    qm, km, vm = (rope.round_bf16(a) for a in OQ.forward(xm64, w64, hq, hkv, pm_g, theta))
    qb, kb, vb = (rope.round_bf16(a) for a in OQ.forward(xb64, w64, hq, hkv, pb_g, theta))
    mq, bq = oracle.select_queries(prob)
    om, _, ob, _ = oracle.forward(prob, qm, km, vm, qb, kb, vb, mq, bq)
    g = oracle.backward(prob, qm, km, vm, qb, kb, vb, f64(dom)[mq], f64(dob)[bq], mq, bq)
    dq_m = np.zeros_like(qm)
    dq_m[mq] = g["dq_main"]
    dq_b = np.zeros_like(qb)
    dq_b[bq] = g["dq_br"]
    dxm_ref, dwm = OQ.backward(xm64, w64, hq, hkv, pm_g, theta, dq_m, g["dk_main"], g["dv_main"])
    dxb_ref, dwb = OQ.backward(xb64, w64, hq, hkv, pb_g, theta, dq_b, g["dk_br"], g["dv_br"])

    # ---- compare
    g2l = {int(gr): i for i, gr in enumerate(share.l2g)}
    mi = np.array([g2l[int(gr)] for gr in mq], np.int64)
    bmap = {int(gr): int(l) for gr, l in zip(share.br_rows_global, share.br_rows_local)}
    bi = np.array([bmap[int(gr)] for gr in bq], np.int64)
    assert np.max(np.abs(f64(out["o_main"])[mi] - om)) <= 2e-2
    assert np.max(np.abs(f64(out["o_br"])[bi] - ob)) <= 2e-2
    dxm = np.zeros((prob.n_main, hidden))
    for j, dx_j in enumerate(dx_blocks):
        dxm[share.l2g_steps[j].astype(np.int64)] = f64(dx_j)
    e_m = rel_l2(dxm, dxm_ref)
    gb = share.br_rows_global.astype(np.int64)
    e_b = rel_l2(f64(dx_br)[share.br_rows_local], dxb_ref[gb])
    e_w = rel_l2(f64(dw), dwm + dwb)
    print(f"[draft layer] dx main {e_m:.2e}, dx branch {e_b:.2e}, dw {e_w:.2e}", flush=True)
    assert e_m <= 1e-2 and e_b <= 1e-2 and e_w <= 1e-2
