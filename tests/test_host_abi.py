"""Host-side checks of the C ABI (no GPU needed): exported symbols, zigzag
partition against the oracle's ownership rule, descriptor validation and
error codes, useful-FLOP counting against the oracle's pair count."""

import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import workloads as W
from paper_2609_07108_amd import rankshare as RS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "branch_attn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


def test_library_exports_every_declared_function():
    L = B.lib()
    decl = declared_functions()
    assert set(decl) == set(B.EXPORTED), decl
    for name in decl:
        assert hasattr(L, name), name


@pytest.mark.parametrize("C", [1, 2, 4, 8])
def test_zigzag_partition_matches_owner_rule(C):
    lens = [16 * C, 0, 48 * C, 2 * C]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    seen = []
    for r in range(C):
        lcu, l2g, lpos = B.zigzag_partition(cu, C, r)
        assert list(lcu) == list(np.concatenate([[0], np.cumsum(np.array(lens) // C)]))
        for s in range(len(lens)):
            rows = l2g[lcu[s]:lcu[s + 1]]
            pos = lpos[lcu[s]:lcu[s + 1]]
            assert np.all(rows == cu[s] + pos)
            assert np.all(np.diff(pos) > 0)  # chunk r then chunk 2C-1-r: increasing positions
            if lens[s]:
                assert np.all(oracle.owner_rank(lens[s], pos, C) == r)
        seen += list(l2g)
    assert sorted(seen) == list(range(int(cu[-1])))


@pytest.mark.parametrize("cu,C,r", [([0, 10], 2, 0), ([0, 8], 2, 2), ([0, 8], 0, 0), ([1, 8], 2, 0),
                                    ([0, 8, 4], 2, 0), ([0, 8], 2, -1)])
def test_zigzag_partition_rejects_bad_input(cu, C, r):
    with pytest.raises(B.BranchAttnError) as e:
        B.zigzag_partition(np.array(cu), C, r)
    assert e.value.code == B.BA_E_INVAL


def _plan(groups, **kw):
    args = dict(cu_seqlens=[0, 64], has_main=[1], cp_size=2, cp_rank=0, hq=4, hkv=2, head_dim=128,
                softmax_scale=0.1, groups=np.array(groups, np.int32).reshape(-1, 6), num_branch_rows=32)
    args.update(kw)
    return B.Plan(**args)


def test_plan_accepts_valid_groups():
    p = _plan([(0, 3, 0, 3, 0, 1), (0, 60, 1, 4, 3, 1)])  # anchors in chunk 0 and chunk 3 (rank 0)
    n_local, ntok = p.info()
    assert n_local == 32 and ntok == 32 + 3 + 4


@pytest.mark.parametrize("groups,kw,code", [
    ([(0, 20, 0, 3, 0, 1)], {}, B.BA_E_INVAL),           # anchor in chunk 1: rank 1
    ([(0, 3, 0, 3, 0, 1), (0, 4, 0, 3, 2, 1)], {}, B.BA_E_INVAL),  # overlapping member rows
    ([(0, 3, 0, 3, 30, 1)], {}, B.BA_E_INVAL),           # member row out of range
    ([(1, 3, 0, 3, 0, 1)], {}, B.BA_E_INVAL),            # sequence out of range
    ([(0, 3, 2, 3, 0, 1)], {}, B.BA_E_INVAL),            # unknown kind
    ([(0, 3, 0, 0, 0, 1)], {}, B.BA_E_INVAL),            # empty group
    ([(0, 3, 0, 65, 0, 1)], {"num_branch_rows": 100}, B.BA_E_INVAL),  # too long
    ([(0, 3, 0, 3, 0, 0)], {}, B.BA_E_INVAL),            # stride 0
    ([], {"head_dim": 64}, B.BA_E_UNSUPPORTED),
    ([], {"hq": 6, "hkv": 4}, B.BA_E_INVAL),
    ([], {"cu_seqlens": [0, 62]}, B.BA_E_INVAL),        # not a multiple of 2C
    ([], {"cp_rank": 2}, B.BA_E_INVAL),
])
def test_plan_rejects_bad_descriptors(groups, kw, code):
    with pytest.raises(B.BranchAttnError) as e:
        _plan(groups, **kw)
    assert e.value.code == code
    assert len(B.lib().branch_attn_last_error()) > 0


@pytest.mark.parametrize("layout", ["group", "depth"])
@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_useful_flops_match_oracle_pair_count(cfg, layout):
    prob = W.config(cfg)
    if cfg in (2, 3, 5):  # shrink: same structure, shorter sequences, fewer heads
        prob = W.custom(np.minimum(prob.seqlens // 16, 1024) // (2 * prob.cp_size) * (2 * prob.cp_size),
                        [(("eagle", int(prob.g_len[prob.g_seq == s][0])) if prob.g_kind[prob.g_seq == s][0] == W.KIND_EAGLE
                          else ("dflash", 16, 64)) for s in range(prob.num_seqs)],
                        hq=prob.hq, hkv=prob.hkv, cp_size=prob.cp_size, cp_rank=prob.cp_rank, seed=cfg,
                        has_main=prob.has_main)
    share = RS.build_share(prob, layout=layout, materialize=False)
    f, b = share.plan.useful_flops()
    pm, pl = oracle.allowed_pair_counts(prob)
    pairs = pm + pl
    assert f == pytest.approx(4 * 128 * prob.hq * pairs, rel=1e-12)
    assert b == pytest.approx(10 * 128 * prob.hq * pairs, rel=1e-12)
    n_local, ntok = share.plan.info()
    mq, bq = oracle.select_queries(prob)
    assert ntok == len(mq) + len(bq)


def test_headline_pair_count_closed_form():
    """256K EAGLE-3 K=3 at CP=8, rank 0: 4 query sets x (16 c^2 + c) main-prefix
    pairs plus 2c chains x (1+2+3) branch-local pairs, c = 16384."""
    prob = W.config(4)
    share = RS.build_share(prob, materialize=False)
    f, b = share.plan.useful_flops()
    c = 262144 // 16
    pairs = 4 * (16 * c * c + c) + 2 * c * 6
    assert f == pytest.approx(4 * 128 * 32 * pairs, rel=1e-12)
    assert (f + b) == pytest.approx(9.852e14, rel=1e-3)


def test_workspace_sizes():
    prob = W.config(1)
    share = RS.build_share(prob, materialize=False)
    f_step, b_step = share.plan.workspace_size(B.BA_MODE_PER_STEP)
    f_fused, b_fused = share.plan.workspace_size(B.BA_MODE_FUSED)
    n_local, ntok = share.plan.info()
    assert f_step >= ntok * prob.hq * 128 * 4  # running fp32 output
    assert f_fused < f_step
    # per-step backward keeps running fp32 dQ sums; the fused one needs only row statistics
    assert b_step >= ntok * prob.hq * (128 + 2) * 4
    assert ntok * prob.hq * 2 * 4 <= b_fused < b_step


def test_rope_settings():
    prob = W.config(1)
    share = RS.build_share(prob, materialize=False)
    plain = share.plan.workspace_size(B.BA_MODE_PER_STEP)
    for bad in (-1.0, float("nan"), float("inf")):
        with pytest.raises(B.BranchAttnError) as e:
            share.plan.set_rope(bad)
        assert e.value.code == B.BA_E_INVAL
    share.plan.set_rope(1.0e4)
    n_local, _ = share.plan.info()
    rot = share.plan.workspace_size(B.BA_MODE_PER_STEP)
    # rotated bf16 copies of Q and the C key blocks in both passes, fp32
    # gradient staging (dQ, dK, dV) in the backward
    C, hq, hkv, nb = prob.cp_size, prob.hq, prob.hkv, share.num_branch_rows
    copies = 2 * 128 * ((n_local + nb) * hq + (C * n_local + nb) * hkv)
    assert rot[0] - plain[0] >= copies
    assert rot[1] - plain[1] >= copies + 4 * 128 * ((n_local + nb) * hq + 2 * (C * n_local + nb) * hkv)
    share.plan.set_rope(0.0)
    assert share.plan.workspace_size(B.BA_MODE_PER_STEP) == plain


def test_rope_positions_must_fit_float():
    # one sequence of 2^24 tokens with a branch anchored at its last token:
    # the branch member's position 2^24 is not exact in float32
    L = 1 << 24
    plan = B.Plan([0, L], [1], 8, 0, 1, 1, 128, 0.088, np.array([[0, L - 1, 0, 1, 0, 1]], np.int32), 1)
    before = plan.workspace_size(B.BA_MODE_PER_STEP)
    with pytest.raises(B.BranchAttnError) as e:
        plan.set_rope(1.0e4)
    assert e.value.code == B.BA_E_UNSUPPORTED
    assert plan.workspace_size(B.BA_MODE_PER_STEP) == before  # left without rotation


def test_device_calls_reject_more_than_32_ring_steps():
    """A plan may describe any CP size, but the ring-step block pointers of
    one call must fit the kernel arguments (32): the device entry points
    refuse larger rings before touching the GPU."""
    import ctypes
    C = 33
    plan = B.Plan([0, 4 * C], [1], C, 0, 1, 1, 128, 0.088, np.zeros((0, 6), np.int32), 0)
    fake = 0x10000  # aligned, never dereferenced: the call stops at validation
    ptrs = (ctypes.c_void_p * C)(*([fake] * C))
    io = B.BaFwdIO(fake, fake, fake, fake, ptrs, ptrs, fake, fake, fake, fake, None, None)
    rc = B.lib().branch_attn_fwd(None, plan.handle, B.BA_MODE_PER_STEP, ctypes.byref(io), ctypes.c_void_p(fake),
                                 1 << 40)
    assert rc == B.BA_E_UNSUPPORTED
    assert b"32" in B.lib().branch_attn_last_error()


def test_auto_schedule_choice_per_plan():
    """BA_MODE_AUTO resolves to the fused schedule, measured the faster one
    on every workload; the explicit modes resolve to themselves."""
    want = {2: B.BA_MODE_FUSED, 3: B.BA_MODE_FUSED, 4: B.BA_MODE_FUSED, 5: B.BA_MODE_FUSED}
    for cfg, mode in want.items():
        share = RS.build_share(W.config(cfg), materialize=False)
        assert share.plan.mode(B.BA_MODE_AUTO) == mode, cfg
        assert share.plan.mode(B.BA_MODE_FUSED) == B.BA_MODE_FUSED
        assert share.plan.mode(B.BA_MODE_PER_STEP) == B.BA_MODE_PER_STEP
        assert share.plan.workspace_size(B.BA_MODE_AUTO) == share.plan.workspace_size(mode)
    share = RS.build_share(W.config(1), materialize=False)
    with pytest.raises(B.BranchAttnError):
        share.plan.mode(3)
    with pytest.raises(B.BranchAttnError):
        share.plan.workspace_size(3)
