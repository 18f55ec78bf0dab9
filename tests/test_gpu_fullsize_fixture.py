"""Element-wise GPU parity at full workload size against stored fp64 oracle
values (``tests/golden/fullsize_c{3,4}.npz``, written by
``tests/golden/make_fullsize_fixture.py``, which calls only the oracle and
the seeded input generator).

* Config 3 (32768-token DFlash sequence, 64/8 heads): the per-ring-block
  dK/dV that the backward hands back to the block owners (Sec. 3.2: the
  backward replays the ring and the gradients of every block are
  accumulated on the rank that holds its queries) are compared element by
  element on 2048 sampled (key row, KV head) pairs covering every position
  inside a 128-key tile, plus 256 groups of branch-local dK/dV, plus O, LSE
  and dQ of 128 query rows.  The earliest key tiles are read by all 8192
  block queries: the unsplit long walks of the dK/dV kernel.
* Config 4 (the 256K-token share): O, LSE and dQ of 256 rows over both of
  the rank's chunks and every branch depth.

Both schedules run; the per-step one (the benchmark's launch configuration)
with bf16 gradients as the benchmark returns them, the fused one with fp32.
Tolerances are the path's bar: O max-abs 2e-2, LSE max-abs 1e-3, gradients
relative L2 1e-2 on the sample (main and branch parts held separately).
"""

import os

import numpy as np
import pytest
import torch

from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

CASES = [pytest.param(3, "per_step", torch.bfloat16, id="c3-per_step-bf16"),
         pytest.param(3, "fused", torch.float32, id="c3-fused-f32"),
         pytest.param(4, "per_step", torch.bfloat16, id="c4-per_step-bf16"),
         pytest.param(4, "fused", torch.float32, id="c4-fused-f32")]


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    return torch.device("cuda:0")


def load_fixture(cfg):
    path = os.path.join(GOLDEN, f"fullsize_c{cfg}.npz")
    assert os.path.exists(path), f"missing {path}: run tests/golden/make_fullsize_fixture.py --config {cfg}"
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def _take(x, rows, heads):
    """x[rows[i], heads[i, j]] -> [n, m, d] as float64 (device gather, then host)."""
    dev = x.device
    r = torch.from_numpy(np.repeat(rows, heads.shape[1])).to(dev)
    h = torch.from_numpy(heads.reshape(-1)).to(dev)
    return x[r, h].double().cpu().numpy().reshape(heads.shape + (x.shape[-1],))


def _report(name, got, ref):
    e = H.rel_l2(got.ravel(), ref.ravel())
    mx = float(np.max(np.abs(got - ref))) if got.size else 0.0
    print(f"[fixture] {name}: rel L2 {e:.3e}, max abs {mx:.3e}, ref norm {np.linalg.norm(ref):.3e}", flush=True)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert e <= H.GRAD_TOL, f"{name}: relative L2 {e:.3e} > {H.GRAD_TOL}"
    return e


@pytest.mark.parametrize("cfg,mode,gdt", CASES)
def test_fullsize_fixture(cuda, cfg, mode, gdt):
    fx = load_fixture(cfg)
    assert int(fx["config"]) == cfg
    prob = W.config(cfg)
    md = B.BA_MODE_FUSED if mode == "fused" else B.BA_MODE_PER_STEP
    print(f"[fixture] config {cfg} ({prob.name}) {mode} grads {gdt}", flush=True)
    share = RS.build_share(prob, device="cuda:0", with_grad=True)
    out = RS.alloc_outputs(share, grads=True, grad_dtype=gdt)
    ws = RS.workspace(share, md, backward=True)
    RS.run_fwd(share, out, md, ws)
    RS.run_bwd(share, out, md, ws)
    torch.cuda.synchronize()
    print("[fixture] GPU done", flush=True)

    # ---- query rows: global -> rank-local rows
    g2l = {int(g): i for i, g in enumerate(share.l2g)}
    bmap = {int(g): int(l) for g, l in zip(share.br_rows_global, share.br_rows_local)}
    mi = np.array([g2l[int(g)] for g in fx["q_main_rows"]], np.int64)
    bi = np.array([bmap[int(g)] for g in fx["q_br_rows"]], np.int64)
    for part, idx in (("main", mi), ("br", bi)):
        if not len(idx):
            continue
        heads = fx[f"q_{part}_heads"]
        o = _take(out[f"o_{part}"], idx, heads)
        err = float(np.max(np.abs(o - fx[f"o_{part}"])))
        lse = out[f"lse_{part}"][:, torch.from_numpy(idx).to(cuda)].double().cpu().numpy()
        lerr = float(np.max(np.abs(lse - fx[f"lse_{part}"])))
        print(f"[fixture] o_{part}: max abs {err:.3e}; lse_{part}: max abs {lerr:.3e}", flush=True)
        assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
        assert err <= H.O_TOL, f"o_{part}: max abs {err:.3e}"
        assert lerr <= H.LSE_TOL, f"lse_{part}: max abs {lerr:.3e}"
        _report(f"dq_{part}", _take(out[f"dq_{part}"], idx, heads), fx[f"dq_{part}"])

    # ---- per-ring-block dK/dV of sampled main keys: global row -> (block j, local row)
    if len(fx["key_rows"]):
        where = np.full(prob.n_main, -1, np.int64)
        local = np.full(prob.n_main, -1, np.int64)
        for j, rows in enumerate(share.l2g_steps):
            where[rows] = j
            local[rows] = np.arange(len(rows))
        kr, kh = fx["key_rows"], fx["key_heads"]
        assert np.all(where[kr] >= 0)
        dk = np.zeros((len(kr), prob.head_dim))
        dv = np.zeros((len(kr), prob.head_dim))
        for j in range(prob.cp_size):
            s = np.flatnonzero(where[kr] == j)
            if len(s):
                dk[s] = _take(out["dk_step"][j], local[kr[s]], kh[s, None])[:, 0]
                dv[s] = _take(out["dv_step"][j], local[kr[s]], kh[s, None])[:, 0]
        _report("dk_step (sampled keys)", dk, fx["dk_main"])
        _report("dv_step (sampled keys)", dv, fx["dv_main"])
    if len(fx["br_key_rows"]):
        bk = np.array([bmap[int(g)] for g in fx["br_key_rows"]], np.int64)
        hh = fx["br_key_heads"][:, None]
        _report("dk_br (sampled groups)", _take(out["dk_br"], bk, hh)[:, 0], fx["dk_br"])
        _report("dv_br (sampled groups)", _take(out["dv_br"], bk, hh)[:, 0], fx["dv_br"])
