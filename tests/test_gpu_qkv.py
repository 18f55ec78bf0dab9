"""GPU parity of the grouped-query QKV projection with rotary embedding
(branch_attn_qkv_fwd / _bwd) against the fp64 oracle `oracle.qkv`.

Tolerances: q, k, v are one bf16 rounding (RNE, half an ulp: 2^-9 relative)
of an fp32-accumulated value, so every element is checked against
|got - ref| <= 2^-8 |ref| + 1e-4 rms(ref); dx and dw accumulate the bf16
rounding of dY (2^-9 relative per element) and are checked by relative L2
error <= 1e-2 over the tensor (sampled entries at full size: max error
<= 1e-2 of their RMS).  Inputs are seeded draws of torch's device generator:
x ~ N(0, 1), w ~ N(0, 1/hidden), gradients ~ N(0, 1).

Cases: a single row; ragged row counts (1, 129, 257, 300, 1000); GQA ratios
1, 2, 4 and 8; theta 0, 1e4 and 5e5 with positions up to 262143; negative
positions (rows left unrotated); both gradient dtypes and both dx dtypes;
dw accumulated over two calls; rows == 0 (dw cleared or kept); and the
projection of the 256K-token rank share (32768 main + 98304 branch rows,
hidden 4096, 32/8 heads, the plan's positions) on sampled rows.
"""

import numpy as np
import pytest
import torch

from oracle import qkv
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


def randn(shape, seed, scale=1.0, dtype=torch.bfloat16):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * scale).to(dtype)


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_elementwise(got, ref, what):
    got = f64(got)
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    err = np.abs(got - ref)
    bound = 2.0 ** -8 * np.abs(ref) + 1e-4 * rms
    worst = np.max(err - bound) if ref.size else -1.0
    assert worst <= 0, f"{what}: max excess {worst:.3e} (max err {err.max():.3e}, rms {rms:.3e})"


def rel_l2(got, ref):
    got = f64(got) if torch.is_tensor(got) else got
    return np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)


def run_case(rows, hidden, hq, hkv, theta, pos, grad_dtype, dx_dtype, seed):
    n = (hq + 2 * hkv) * 128
    x = randn((rows, hidden), seed)
    w = randn((n, hidden), seed + 1, 1.0 / np.sqrt(hidden))
    pos_t = torch.as_tensor(pos, dtype=torch.int32, device="cuda") if theta else None
    q = torch.empty((rows, hq, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.empty((rows, hkv, 128), dtype=torch.bfloat16, device="cuda")
    v = torch.empty_like(k)
    B.branch_attn_qkv_fwd(x, w, hq, hkv, pos_t, theta, q, k, v)
    dq = randn((rows, hq, 128), seed + 2, dtype=grad_dtype)
    dk = randn((rows, hkv, 128), seed + 3, dtype=grad_dtype)
    dv = randn((rows, hkv, 128), seed + 4, dtype=grad_dtype)
    dx = torch.empty((rows, hidden), dtype=dx_dtype, device="cuda")
    dw = torch.full((n, hidden), float("nan"), dtype=torch.float32, device="cuda")  # overwritten
    ws = torch.empty(max(B.branch_attn_qkv_workspace_size(rows, hq, hkv), 256), dtype=torch.uint8, device="cuda")
    B.branch_attn_qkv_bwd(x, w, hq, hkv, pos_t, theta, dq, dk, dv, dx, dw, False, ws)
    torch.cuda.synchronize()
    xn, wn = f64(x), f64(w)
    pn = np.asarray(pos) if theta else None
    ref_q, ref_k, ref_v = qkv.forward(xn, wn, hq, hkv, pn, theta)
    ref_dx, ref_dw = qkv.backward(xn, wn, hq, hkv, pn, theta, f64(dq), f64(dk), f64(dv))
    return (q, k, v, dx, dw), (ref_q, ref_k, ref_v, ref_dx, ref_dw), (x, w, pos_t, dq, dk, dv, ws)


CASES = [
    # rows, hidden, hq, hkv, theta, max position (None: some negative), grad dtype, dx dtype
    (1, 128, 1, 1, 1.0e4, 50, torch.bfloat16, torch.bfloat16),
    (300, 256, 4, 2, 1.0e4, 8191, torch.float32, torch.float32),
    (1000, 512, 8, 1, 5.0e5, 262143, torch.bfloat16, torch.float32),
    (257, 384, 6, 3, 0.0, 0, torch.float32, torch.bfloat16),
    (129, 128, 2, 2, 1.0e4, None, torch.bfloat16, torch.bfloat16),
    # row counts that are multiples of 64 send dW to the 256 x 256 tile
    # kernel too (dX and the forward take it whenever their reduction is a
    # multiple of 64); output widths of 640 and 384 leave its last column
    # tile part-filled, 320 rows its last row tile
    (512, 384, 3, 1, 1.0e4, 4095, torch.bfloat16, torch.float32),
    (320, 256, 4, 4, 5.0e5, 262143, torch.float32, torch.bfloat16),
]


@pytest.mark.parametrize("rows,hidden,hq,hkv,theta,maxpos,gd,xd", CASES)
def test_qkv_parity(cuda, rows, hidden, hq, hkv, theta, maxpos, gd, xd):
    print(f"[qkv] rows {rows} hidden {hidden} heads {hq}/{hkv} theta {theta}", flush=True)
    rng = np.random.default_rng(rows + hidden)
    if maxpos is None:
        pos = rng.integers(-3, 500, rows)
        pos[::7] = -1
    else:
        pos = rng.integers(0, maxpos + 1, rows)
        pos[0] = maxpos
    got, ref, _ = run_case(rows, hidden, hq, hkv, theta, pos, gd, xd, seed=rows * 7 + hidden)
    for g, r, name in zip(got[:3], ref[:3], "qkv"):
        assert_elementwise(g, r, name)
    assert rel_l2(got[3], ref[3]) <= 1e-2, ("dx", rel_l2(got[3], ref[3]))
    assert rel_l2(got[4], ref[4]) <= 1e-2, ("dw", rel_l2(got[4], ref[4]))


def test_qkv_dw_accumulates_and_empty_calls(cuda):
    hidden, hq, hkv, theta = 256, 4, 1, 1.0e4
    n = (hq + 2 * hkv) * 128
    rng = np.random.default_rng(5)
    pos_a, pos_b = rng.integers(0, 3000, 200), rng.integers(0, 3000, 77)
    got_a, ref_a, (xa, w, pa, dqa, dka, dva, ws) = run_case(200, hidden, hq, hkv, theta, pos_a, torch.float32,
                                                            torch.float32, seed=11)
    got_b, ref_b, (xb, wb, pb, dqb, dkb, dvb, wsb) = run_case(77, hidden, hq, hkv, theta, pos_b, torch.float32,
                                                              torch.float32, seed=11)
    assert torch.equal(w, wb)  # same weight seed
    dw = got_a[4].clone()
    dx = torch.empty((77, hidden), dtype=torch.float32, device="cuda")
    B.branch_attn_qkv_bwd(xb, w, hq, hkv, pb, theta, dqb, dkb, dvb, dx, dw, True, wsb)
    torch.cuda.synchronize()
    assert rel_l2(dw, ref_a[4] + ref_b[4]) <= 1e-2
    # rows == 0: dw cleared without accumulation, kept with it
    empty = torch.empty((0, hidden), dtype=torch.bfloat16, device="cuda")
    g0 = torch.empty((0, hq, 128), dtype=torch.float32, device="cuda")
    g1 = torch.empty((0, hkv, 128), dtype=torch.float32, device="cuda")
    keep = dw.clone()
    B.branch_attn_qkv_bwd(empty, w, hq, hkv, None, 0.0, g0, g1, g1, empty, dw, True, None)
    torch.cuda.synchronize()
    assert torch.equal(dw, keep)
    B.branch_attn_qkv_bwd(empty, w, hq, hkv, None, 0.0, g0, g1, g1, empty, dw, False, None)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dw).item() == 0
    assert dw.shape == (n, hidden)


def test_qkv_fullsize_headline_share(cuda):
    """Projection of the 256K-token rank share (CP=8 rank 0, EAGLE-3 depth 3):
    32768 main rows and 98304 branch rows, hidden 4096, 32/8 heads, theta 5e5,
    the plan's positions; the weight gradient accumulated over both calls."""
    prob = W.config(4)
    share = RS.build_share(prob, materialize=False)
    mp, bp = share.plan.positions(share.n_local, share.num_branch_rows)
    hidden, hq, hkv, theta = 4096, prob.hq, prob.hkv, 5.0e5
    n = (hq + 2 * hkv) * 128
    print(f"[qkv full] main {len(mp)} branch {len(bp)} rows, hidden {hidden}", flush=True)
    w = randn((n, hidden), 41, 1.0 / np.sqrt(hidden))
    dw = torch.empty((n, hidden), dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(42)
    cols = rng.integers(0, hidden, 6)
    heads = [0, hq - 1, hq, hq + hkv - 1, hq + hkv, n // 128 - 1]  # q, k and v heads
    dw_ref = np.zeros((len(heads), 128, len(cols)))
    for part, pos in enumerate((mp, bp)):
        rows = len(pos)
        x = randn((rows, hidden), 43 + part)
        pos_t = torch.as_tensor(pos, dtype=torch.int32, device="cuda")
        q = torch.empty((rows, hq, 128), dtype=torch.bfloat16, device="cuda")
        k = torch.empty((rows, hkv, 128), dtype=torch.bfloat16, device="cuda")
        v = torch.empty_like(k)
        B.branch_attn_qkv_fwd(x, w, hq, hkv, pos_t, theta, q, k, v)
        dq = randn((rows, hq, 128), 45 + part)
        dk = randn((rows, hkv, 128), 47 + part)
        dv = randn((rows, hkv, 128), 49 + part)
        dx = torch.empty((rows, hidden), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(B.branch_attn_qkv_workspace_size(rows, hq, hkv), dtype=torch.uint8, device="cuda")
        B.branch_attn_qkv_bwd(x, w, hq, hkv, pos_t, theta, dq, dk, dv, dx, dw, part == 1, ws)
        torch.cuda.synchronize()
        sel = np.r_[0, rows - 1, rng.integers(0, rows, 30)]
        st = torch.as_tensor(sel, device="cuda")
        xs, wn = f64(x[st]), f64(w)
        rq, rk, rv = qkv.forward(xs, wn, hq, hkv, pos[sel], theta)
        for g, r, name in zip((q[st], k[st], v[st]), (rq, rk, rv), "qkv"):
            assert_elementwise(g, r, f"{name} part {part}")
        rdx, _ = qkv.backward(xs, wn, hq, hkv, pos[sel], theta, f64(dq[st]), f64(dk[st]), f64(dv[st]))
        assert rel_l2(dx[st], rdx) <= 1e-2, ("dx", part, rel_l2(dx[st], rdx))
        # dw columns `cols` of the sampled heads: sum over every row of dY[:, head] x[:, cols]
        xc = f64(x[:, torch.as_tensor(cols, device="cuda")])
        for hi, h in enumerate(heads):
            if h < hq:
                dy = qkv.grad_y(f64(dq[:, h:h + 1]), f64(dk[:, :1]), f64(dv[:, :1]), pos, theta)[:, :128]
            elif h < hq + hkv:
                dy = qkv.grad_y(f64(dq[:, :1]), f64(dk[:, h - hq:h - hq + 1]), f64(dv[:, :1]), pos, theta)[:, 128:256]
            else:
                dy = f64(dv[:, h - hq - hkv])
            dw_ref[hi] += dy.T @ xc
        del x, q, k, v, dq, dk, dv, dx, ws
    got = np.stack([f64(dw[h * 128:(h + 1) * 128][:, torch.as_tensor(cols, device="cuda")]) for h in heads])
    rms = np.sqrt(np.mean(dw_ref ** 2))
    assert np.max(np.abs(got - dw_ref)) <= 1e-2 * rms, (np.max(np.abs(got - dw_ref)), rms)
