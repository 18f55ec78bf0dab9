"""branch_attn_fwd_noalloc: the forward with the library's static per-GPU
scratch instead of a caller workspace, for callers that cannot allocate.

Its kernels are those of branch_attn_fwd, so with the same plan and mode the
outputs must be bit-identical.  Two calls in a row share the scratch, the
second on a smaller problem (in the other schedule), so a stale table or
running sum left by the first call would show; the first problem is then run
again.  A plan whose scratch need exceeds the static array is refused before
anything touches the GPU.
"""

import ctypes

import pytest
import torch

from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W


def _problems():
    big = W.custom([2048, 1024, 512], [("eagle", 3), ("dflash", 16, 64), ("eagle", 2)], hq=8, hkv=2,
                   cp_size=2, cp_rank=1, seed=71, name="noalloc-big", backward=False)
    small = W.custom([256], [("eagle", 2)], hq=4, hkv=4, cp_size=1, cp_rank=0, seed=72, name="noalloc-small",
                     backward=False)
    return big, small


def _run(share, mode, noalloc):
    out = RS.alloc_outputs(share)
    t = share.t
    args = (share.plan, mode, t["q_main"], t["q_br"], t["k_br"], t["v_br"], t["k_step"], t["v_step"],
            out["o_main"], out["o_br"], out["lse_main"], out["lse_br"])
    if noalloc:
        B.branch_attn_fwd_noalloc(*args)
    else:
        B.branch_attn_fwd(*args, RS.workspace(share, mode))
    torch.cuda.synchronize()
    return out


def _same(a, b, what):
    for k in ("o_main", "o_br", "lse_main", "lse_br"):
        assert torch.equal(a[k], b[k]), f"{what}: {k} differs from branch_attn_fwd"
        assert torch.isfinite(a[k].float()).all() or k.startswith("lse"), f"{what}: {k} not finite"


def test_noalloc_refuses_oversized_plan_without_gpu():
    prob = W.config(4)
    share = RS.build_share(prob, materialize=False)
    io = B.BaFwdIO()
    rc = B.lib().branch_attn_fwd_noalloc(None, share.plan.handle, B.BA_MODE_PER_STEP, ctypes.byref(io))
    assert rc == B.BA_E_WORKSPACE
    assert b"static scratch" in B.lib().branch_attn_last_error()


@pytest.mark.gpu
def test_noalloc_forward_matches_workspace_forward():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    big, small = _problems()
    sb = RS.build_share(big, device="cuda:0", with_grad=False)
    ss = RS.build_share(small, device="cuda:0", with_grad=False)
    print("[noalloc] first call: fused, 3 sequences, CP=2 rank 1", flush=True)
    a1 = _run(sb, B.BA_MODE_FUSED, noalloc=True)
    print("[noalloc] second call: per-step, one 256-token sequence", flush=True)
    a2 = _run(ss, B.BA_MODE_PER_STEP, noalloc=True)
    print("[noalloc] third call: per-step on the first problem", flush=True)
    a3 = _run(sb, B.BA_MODE_PER_STEP, noalloc=True)
    _same(a1, _run(sb, B.BA_MODE_FUSED, noalloc=False), "first call")
    _same(a2, _run(ss, B.BA_MODE_PER_STEP, noalloc=False), "second call")
    _same(a3, _run(sb, B.BA_MODE_PER_STEP, noalloc=False), "third call")
