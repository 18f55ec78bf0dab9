"""GPU parity of the path with rotary position embedding in front of the
attention (queries and keys rotated by their positions: main token at p,
branch member i at anchor + 1 + i) against the fp64 oracle `oracle.rope`,
which rounds the rotated queries and keys to bfloat16 as the library hands
them to its bfloat16 kernels.  Same tolerances as the plain path.  Cases:
both branch kinds, both ring schedules, both gradient dtypes, both
branch-array layouts, GQA ratios 1, 4, 8 and 64, an empty sequence, DFlash
blocks in a sequence that also trains its main tokens, a DFlash-only share,
EAGLE chains of the maximum 64 members, and positions up to 8191 with theta
1e4 (angles of thousands of radians, so the turn reduction of the angles
matters).
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import rope
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

MODES = {"per_step": B.BA_MODE_PER_STEP, "fused": B.BA_MODE_FUSED}


def case(name):
    if name == "mixed_cp2":
        return W.custom([1024, 384], [("eagle", 3), ("dflash", 16, 64)], hq=16, hkv=4, cp_size=2, cp_rank=1,
                        seed=301, name=name)
    if name == "long_cp4":
        return W.custom([8192], [("eagle", 2)], hq=8, hkv=1, cp_size=4, cp_rank=1, seed=302, name=name)
    if name == "edges_g1":
        # G = 1, an empty sequence, DFlash blocks of 8 (two per window) in a
        # sequence that also trains its main tokens, an EAGLE chain of 64
        return W.custom([0, 512, 64], [None, ("dflash", 8, 32, 2), ("eagle", 64)], hq=2, hkv=2, cp_size=2,
                        cp_rank=0, seed=303, has_main=[True, True, True], name=name)
    if name == "dflash_only_g64":
        # G = 64 and a share whose only queries are DFlash blocks
        return W.custom([1024], [("dflash", 16, 64)], hq=64, hkv=1, cp_size=2, cp_rank=1, seed=304, name=name)
    raise KeyError(name)


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    return torch.device("cuda:0")


def oracle_rope_run(prob, t, theta):
    mq, bq = oracle.select_queries(prob)
    args = [t[k] for k in H.TENSORS]
    fwd = rope.forward(prob, *args, theta, rounded=True, main_q=mq, br_q=bq)
    bwd = rope.backward(prob, *args, t["dom"][mq], t["dob"][bq], theta, main_q=mq, br_q=bq, rounded=True)
    return mq, bq, fwd, bwd


@pytest.mark.parametrize("name,mode,layout,grad_dtype,theta", [
    ("mixed_cp2", "per_step", "group", torch.bfloat16, 1.0e4),
    ("mixed_cp2", "fused", "depth", torch.float32, 5.0e5),
    ("long_cp4", "per_step", "depth", torch.float32, 1.0e4),
    ("long_cp4", "fused", "group", torch.bfloat16, 1.0e4),
    ("edges_g1", "per_step", "depth", torch.bfloat16, 1.0e4),
    ("dflash_only_g64", "fused", "group", torch.float32, 1.0e6),
])
def test_rope_forward_backward_parity(cuda, name, mode, layout, grad_dtype, theta):
    prob = case(name)
    t = H.oracle_inputs(prob)
    mq, bq, ref_f, ref_b = oracle_rope_run(prob, t, theta)
    share = RS.build_share(prob, device="cuda", layout=layout, rope_theta=theta)
    got_f, got_b, _ = H.gpu_bwd(share, MODES[mode], mq, bq, grad_dtype=grad_dtype)
    H.assert_fwd_close(got_f, ref_f)
    H.assert_bwd_close(got_b, ref_b)


def test_rope_off_again_is_the_plain_path(cuda):
    prob = case("mixed_cp2")
    share = RS.build_share(prob, device="cuda", rope_theta=1.0e4)
    share.plan.set_rope(0.0)
    t = H.oracle_inputs(prob)
    mq, bq, ref_f, _ = H.oracle_run(prob, t, backward=False)
    got, _ = H.gpu_fwd(share, B.BA_MODE_PER_STEP, mq, bq)
    H.assert_fwd_close(got, ref_f)
