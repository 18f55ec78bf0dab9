"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

P1 brute force, P2 depth-0 == textbook causal attention, P3 Q = 0 closed form,
P4 merge identity (Eq. lse-merge), P5 chain rule through the merge (backward
by ring replay, Sec. 3.2), P6 finite differences and autograd, P7 reassembly
of all context-parallel ranks, P8 zigzag load-balance closed form, P9 DFlash
block symmetry.  The paper prints no worked numeric example for branch
attention, so raw values are pinned by these properties instead.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_07108_amd import workloads as W
from tests import bruteforce as BF

TENSORS = ("qm", "km", "vm", "qb", "kb", "vb")


def draw_all(p, zero_q=False):
    t = {}
    for k in TENSORS:
        t[k] = p.draw(k, zero=(zero_q and k in ("qm", "qb"))).float().numpy().astype(np.float64)
    return t


def tiny_problems():
    return [
        W.custom([16], [("eagle", 2)], hq=2, hkv=1, head_dim=4, cp_size=2, cp_rank=1, seed=11),
        W.custom([8, 16], [("eagle", 3), ("dflash", 4, 8)], hq=2, hkv=2, head_dim=4,
                 cp_size=2, cp_rank=0, seed=12),
        W.custom([12], [("dflash", 3, 4)], hq=4, hkv=2, head_dim=3, cp_size=1, cp_rank=0,
                 seed=13, has_main=[True]),
        W.custom([8, 8], [None, ("eagle", 1)], hq=1, hkv=1, head_dim=5, cp_size=2, cp_rank=1,
                 seed=14),
    ]


def small_problem(seed=21, C=2, r=0):
    return W.custom([64, 32, 96], [("eagle", 3), ("dflash", 8, 16), ("eagle", 2)], hq=4, hkv=2,
                    head_dim=16, cp_size=C, cp_rank=r, seed=seed)


# ---------------------------------------------------------------- P1
@pytest.mark.parametrize("pi", range(4))
def test_p1_bruteforce_forward_backward(pi):
    p = tiny_problems()[pi]
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    rng = np.random.default_rng(100 + pi)
    dom = rng.standard_normal((len(mq), p.hq, p.head_dim))
    dob = rng.standard_normal((len(bq), p.hq, p.head_dim))
    om, lm, ob, lb = oracle.forward(p, *[t[k] for k in TENSORS], mq, bq)
    g = oracle.backward(p, *[t[k] for k in TENSORS], dom, dob, mq, bq)

    T = {k: t[k].tolist() for k in TENSORS}
    dO = {("m", int(r)): dom[i].tolist() for i, r in enumerate(mq)}
    dO.update({("b", int(r)): dob[i].tolist() for i, r in enumerate(bq)})
    O, LSE, G = BF.forward_backward(p, T, dO)
    assert set(O) == set(dO)  # the same query set
    for i, r in enumerate(mq):
        np.testing.assert_allclose(om[i], O[("m", int(r))], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lm[:, i], LSE[("m", int(r))], rtol=0, atol=1e-12)
        np.testing.assert_allclose(g["dq_main"][i], G[("dq", "m", int(r))], rtol=0, atol=1e-12)
    for i, r in enumerate(bq):
        np.testing.assert_allclose(ob[i], O[("b", int(r))], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lb[:, i], LSE[("b", int(r))], rtol=0, atol=1e-12)
        np.testing.assert_allclose(g["dq_br"][i], G[("dq", "b", int(r))], rtol=0, atol=1e-12)
    for name, arr_m, arr_b in (("dk", g["dk_main"], g["dk_br"]), ("dv", g["dv_main"], g["dv_br"])):
        for row in range(len(arr_m)):
            ref = G.get((name, "m", row), np.zeros_like(arr_m[row]))
            np.testing.assert_allclose(arr_m[row], ref, rtol=0, atol=1e-12)
        for row in range(len(arr_b)):
            ref = G.get((name, "b", row), np.zeros_like(arr_b[row]))
            np.testing.assert_allclose(arr_b[row], ref, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- P2
@pytest.mark.parametrize("C,r", [(1, 0), (2, 1), (4, 2)])
def test_p2_depth0_is_textbook_causal_attention(C, r):
    p = W.custom([64, 128, 32], [None, ("eagle", 0), None], hq=4, hkv=2, head_dim=16,
                 cp_size=C, cp_rank=r, seed=31)
    assert len(p.g_seq) == 0
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    om, lm, _, _ = oracle.forward(p, *[t[k] for k in TENSORS], mq, bq)
    row_of = {int(v): i for i, v in enumerate(mq)}
    G = p.hq // p.hkv
    for s in range(p.num_seqs):
        lo, hi = int(p.cu_seqlens[s]), int(p.cu_seqlens[s + 1])
        q = torch.from_numpy(t["qm"][lo:hi]).permute(1, 0, 2)  # [H, L, d]
        k = torch.from_numpy(t["km"][lo:hi]).permute(1, 0, 2).repeat_interleave(G, 0)
        v = torch.from_numpy(t["vm"][lo:hi]).permute(1, 0, 2).repeat_interleave(G, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
        sc = (q @ k.transpose(1, 2)) / math.sqrt(p.head_dim)
        causal = torch.ones(hi - lo, hi - lo, dtype=torch.bool).tril()
        lse = torch.logsumexp(sc.masked_fill(~causal, -math.inf), dim=-1)  # [H, L]
        for pos in range(hi - lo):
            i = row_of.get(lo + pos)
            if i is None:
                continue
            np.testing.assert_allclose(om[i], ref[:, pos, :].numpy(), rtol=0, atol=1e-12)
            np.testing.assert_allclose(lm[:, i], lse[:, pos].numpy(), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- P3
@pytest.mark.parametrize("C,r", [(1, 0), (2, 0), (2, 1), (4, 3)])
def test_p3_zero_queries_closed_form(C, r):
    """Q = 0: every allowed score is 0, so LSE = ln(#allowed keys) and O is
    the mean of the allowed values.  #allowed is P+1 for a main query at P,
    anchor+1+(k) for the depth-k member of a chain, anchor+1+len for a block
    member."""
    p = W.custom([64, 32, 96], [("eagle", 3), ("dflash", 8, 16), ("eagle", 2)], hq=4, hkv=2,
                 head_dim=8, cp_size=C, cp_rank=r, seed=41)
    t = draw_all(p, zero_q=True)
    mq, bq = oracle.select_queries(p)
    om, lm, ob, lb = oracle.forward(p, *[t[k] for k in TENSORS], mq, bq)
    seq_of = np.searchsorted(p.cu_seqlens, mq, side="right") - 1
    for i, row in enumerate(mq):
        P = row - p.cu_seqlens[seq_of[i]]
        np.testing.assert_allclose(lm[:, i], math.log(P + 1), rtol=0, atol=1e-13)
        mean = t["vm"][p.cu_seqlens[seq_of[i]]:row + 1].mean(axis=0)
        np.testing.assert_allclose(om[i], np.repeat(mean, p.hq // p.hkv, axis=0), atol=1e-13)
    grp_of = np.repeat(np.arange(len(p.g_len)), p.g_len)
    for i, row in enumerate(bq):
        g = grp_of[row]
        k = row - p.g_row0[g]
        a = p.g_anchor[g]
        n_local = (k + 1) if p.g_kind[g] == W.KIND_EAGLE else p.g_len[g]
        np.testing.assert_allclose(lb[:, i], math.log(a + 1 + n_local), rtol=0, atol=1e-13)
        base = p.cu_seqlens[p.g_seq[g]]
        vals = np.concatenate([t["vm"][base:base + a + 1],
                               t["vb"][p.g_row0[g]:p.g_row0[g] + n_local]], axis=0)
        np.testing.assert_allclose(ob[i], np.repeat(vals.mean(axis=0), p.hq // p.hkv, axis=0),
                                   atol=1e-13)


# ---------------------------------------------------------------- P4
def _chunk_filter(C, j):
    def f(s, L, is_main, pos):
        c = L // (2 * C)
        ch = np.where(is_main, pos // max(c, 1), -1)
        return is_main & ((ch == j) | (ch == 2 * C - 1 - j))
    return f


def test_p4_merge_of_main_and_branch_partials_equals_union():
    p = small_problem()
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    args = [t[k] for k in TENSORS]
    full = oracle.forward(p, *args, mq, bq)
    main = oracle.forward(p, *args, mq, bq, key_filter=lambda s, L, m, pos: m)
    br = oracle.forward(p, *args, mq, bq, key_filter=lambda s, L, m, pos: ~m)
    # main queries have no branch-local keys: their branch partial is empty
    assert np.all(np.isneginf(br[1]))
    for a, b, o_full, l_full in ((0, 1, 0, 1), (2, 3, 2, 3)):
        o, l = oracle.lse_merge(main[a], main[b], br[a], br[b])
        np.testing.assert_allclose(o, full[o_full], rtol=0, atol=1e-12)
        np.testing.assert_allclose(l, full[l_full], rtol=0, atol=1e-12)


@pytest.mark.parametrize("C", [2, 4])
def test_p4_merge_of_ring_steps_equals_main_prefix(C):
    p = W.custom([64, 128], [("eagle", 2), ("dflash", 8, 32)], hq=2, hkv=1, head_dim=8,
                 cp_size=C, cp_rank=1, seed=42)
    t = draw_all(p)
    args = [t[k] for k in TENSORS]
    mq, bq = oracle.select_queries(p)
    ref = oracle.forward(p, *args, mq, bq, key_filter=lambda s, L, m, pos: m)
    acc = None
    for i in range(C):
        j = (p.cp_rank - i) % C
        part = oracle.forward(p, *args, mq, bq, key_filter=_chunk_filter(C, j))
        if acc is None:
            acc = list(part)
        else:
            acc[0], acc[1] = oracle.lse_merge(acc[0], acc[1], part[0], part[1])
            acc[2], acc[3] = oracle.lse_merge(acc[2], acc[3], part[2], part[3])
    for k in range(4):
        np.testing.assert_allclose(acc[k], ref[k], rtol=0, atol=1e-12)


def test_p4_merge_algebra():
    rng = np.random.default_rng(5)
    o = [rng.standard_normal((7, 3, 4)) for _ in range(3)]
    l = [rng.standard_normal((3, 7)) * 3 for _ in range(3)]
    l[1][0, 2] = -np.inf
    # identity element (O=0, LSE=-inf)
    e_o, e_l = np.zeros_like(o[0]), np.full_like(l[0], -np.inf)
    oo, ll = oracle.lse_merge(o[0], l[0], e_o, e_l)
    np.testing.assert_array_equal(ll, l[0])
    np.testing.assert_allclose(oo, o[0], atol=1e-15)
    # both empty -> (0, -inf), no NaN
    oo, ll = oracle.lse_merge(e_o, e_l, e_o, e_l)
    assert np.all(np.isneginf(ll)) and np.all(oo == 0)
    # commutative and associative
    a = oracle.lse_merge(o[0], l[0], o[1], l[1])
    b = oracle.lse_merge(o[1], l[1], o[0], l[0])
    np.testing.assert_allclose(a[0], b[0], atol=1e-14)
    np.testing.assert_allclose(a[1], b[1], atol=1e-14)
    x = oracle.lse_merge(*oracle.lse_merge(o[0], l[0], o[1], l[1]), o[2], l[2])
    y = oracle.lse_merge(o[0], l[0], *oracle.lse_merge(o[1], l[1], o[2], l[2]))
    np.testing.assert_allclose(x[0], y[0], atol=1e-13)
    np.testing.assert_allclose(x[1], y[1], atol=1e-13)
    # the LSE is log(e^la + e^lb) computed without overflow
    big = oracle.lse_merge(o[0], np.full_like(l[0], 800.0), o[1], np.full_like(l[0], 800.0))
    np.testing.assert_allclose(big[1], 800.0 + math.log(2.0), atol=1e-12)


# ---------------------------------------------------------------- P5
def test_p5_backward_through_merge_equals_global_lse_backward():
    p = small_problem(seed=51)
    t = draw_all(p)
    args = [t[k] for k in TENSORS]
    mq, bq = oracle.select_queries(p)
    rng = np.random.default_rng(52)
    dom = rng.standard_normal((len(mq), p.hq, p.head_dim))
    dob = rng.standard_normal((len(bq), p.hq, p.head_dim))
    ref = oracle.backward(p, *args, dom, dob, mq, bq)
    fm = lambda s, L, m, pos: m
    fb = lambda s, L, m, pos: ~m
    pm = oracle.forward(p, *args, mq, bq, key_filter=fm)
    pb = oracle.forward(p, *args, mq, bq, key_filter=fb)
    (dom_m, dl_m), (dom_b, dl_b) = oracle.lse_merge_backward(pm[0], pm[1], pb[0], pb[1], dom)
    (dob_m, dlb_m), (dob_b, dlb_b) = oracle.lse_merge_backward(pm[2], pm[3], pb[2], pb[3], dob)
    gm = oracle.backward(p, *args, dom_m, dob_m, mq, bq, key_filter=fm, dlse_main=dl_m, dlse_br=dlb_m)
    gb = oracle.backward(p, *args, dom_b, dob_b, mq, bq, key_filter=fb, dlse_main=dl_b, dlse_br=dlb_b)
    for k in ref:
        np.testing.assert_allclose(gm[k] + gb[k], ref[k], rtol=0, atol=1e-11)


# ---------------------------------------------------------------- P6
def _loss(p, t, dom, dob, mq, bq):
    om, _, ob, _ = oracle.forward(p, *[t[k] for k in TENSORS], mq, bq)
    return float(np.sum(om * dom) + np.sum(ob * dob))


def test_p6_finite_differences():
    p = W.custom([32, 16], [("eagle", 2), ("dflash", 4, 8)], hq=2, hkv=1, head_dim=8,
                 cp_size=2, cp_rank=0, seed=61)
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    rng = np.random.default_rng(62)
    dom = rng.standard_normal((len(mq), p.hq, p.head_dim))
    dob = rng.standard_normal((len(bq), p.hq, p.head_dim))
    g = oracle.backward(p, *[t[k] for k in TENSORS], dom, dob, mq, bq)
    h = 1e-6
    checks = 0
    for name, grad_name, rows in (("qm", "dq_main", mq), ("qb", "dq_br", bq), ("km", "dk_main", None),
                                  ("vm", "dv_main", None), ("kb", "dk_br", None), ("vb", "dv_br", None)):
        for _ in range(6):
            if rows is not None:
                i = int(rng.integers(len(rows)))
                row = int(rows[i])
                gi = i
            else:
                row = int(rng.integers(len(t[name])))
                gi = row
            hh = int(rng.integers(t[name].shape[1]))
            dd = int(rng.integers(p.head_dim))
            old = t[name][row, hh, dd]
            t[name][row, hh, dd] = old + h
            lp = _loss(p, t, dom, dob, mq, bq)
            t[name][row, hh, dd] = old - h
            lm = _loss(p, t, dom, dob, mq, bq)
            t[name][row, hh, dd] = old
            fd = (lp - lm) / (2 * h)
            an = g[grad_name][gi, hh, dd]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, row, hh, dd, fd, an)
            checks += 1
    assert checks == 36


def test_p6_autograd_of_dense_masked_attention():
    p = W.custom([16, 8], [("eagle", 2), ("dflash", 4, 8)], hq=2, hkv=1, head_dim=4,
                 cp_size=1, cp_rank=0, seed=63)
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    rng = np.random.default_rng(64)
    dom = rng.standard_normal((len(mq), p.hq, p.head_dim))
    dob = rng.standard_normal((len(bq), p.hq, p.head_dim))
    g = oracle.backward(p, *[t[k] for k in TENSORS], dom, dob, mq, bq)
    # dense autograd over the concatenation of every main and branch row; the
    # mask comes from the brute-force key enumeration
    Q = torch.tensor(np.concatenate([t["qm"], t["qb"]]), requires_grad=True)
    K = torch.tensor(np.concatenate([t["km"], t["kb"]]), requires_grad=True)
    V = torch.tensor(np.concatenate([t["vm"], t["vb"]]), requires_grad=True)
    nm = len(t["qm"])
    qs = BF.queries(p, 0)
    mask = torch.zeros(len(qs), len(K), dtype=torch.bool)
    qrows = []
    for i, q in enumerate(qs):
        qrows.append(q[5] if q[0] == "m" else nm + q[5])
        for kk, row in BF.keys_of(p, q):
            mask[i, row if kk == "m" else nm + row] = True
    qrows = torch.tensor(qrows)
    loss = 0
    for h in range(p.hq):
        S = p.scale * Q[qrows, h] @ K[:, h // (p.hq // p.hkv)].T
        P = torch.softmax(S.masked_fill(~mask, -math.inf), dim=-1)
        O = P @ V[:, h // (p.hq // p.hkv)]
        dO = torch.tensor(np.stack([dom[list(mq).index(q[5])][h] if q[0] == "m"
                                    else dob[list(bq).index(q[5])][h] for q in qs]))
        loss = loss + (O * dO).sum()
    loss.backward()
    np.testing.assert_allclose(g["dk_main"], K.grad[:nm].numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dk_br"], K.grad[nm:].numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dv_main"], V.grad[:nm].numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dv_br"], V.grad[nm:].numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dq_main"], Q.grad[mq].numpy(), atol=1e-12)
    np.testing.assert_allclose(g["dq_br"], Q.grad[nm + bq].numpy(), atol=1e-12)


# ---------------------------------------------------------------- P7
@pytest.mark.parametrize("C", [2, 4])
def test_p7_all_ranks_reassemble_the_unsharded_result(C):
    base = W.custom([64, 128], [("eagle", 2), ("dflash", 8, 32)], hq=2, hkv=1, head_dim=8,
                    cp_size=1, cp_rank=0, seed=71)
    t = draw_all(base)
    args = [t[k] for k in TENSORS]
    rng = np.random.default_rng(72)
    mq1, bq1 = oracle.select_queries(base)
    dom = rng.standard_normal((base.n_main, base.hq, base.head_dim))
    dob = rng.standard_normal((base.n_branch, base.hq, base.head_dim))
    ref = oracle.forward(base, *args, mq1, bq1)
    gref = oracle.backward(base, *args, dom[mq1], dob[bq1], mq1, bq1)
    seen_m, seen_b = [], []
    acc = {k: 0 for k in ("dk_main", "dv_main", "dk_br", "dv_br")}
    import dataclasses
    for r in range(C):
        p = dataclasses.replace(base, cp_size=C, cp_rank=r)
        mq, bq = oracle.select_queries(p)
        seen_m += list(mq)
        seen_b += list(bq)
        out = oracle.forward(p, *args, mq, bq)
        im = np.searchsorted(mq1, mq)
        ib = np.searchsorted(bq1, bq)
        np.testing.assert_allclose(out[0], ref[0][im], atol=1e-12)
        np.testing.assert_allclose(out[1], ref[1][:, im], atol=1e-12)
        np.testing.assert_allclose(out[2], ref[2][ib], atol=1e-12)
        np.testing.assert_allclose(out[3], ref[3][:, ib], atol=1e-12)
        g = oracle.backward(p, *args, dom[mq], dob[bq], mq, bq)
        np.testing.assert_allclose(g["dq_main"], gref["dq_main"][im], atol=1e-12)
        np.testing.assert_allclose(g["dq_br"], gref["dq_br"][ib], atol=1e-12)
        for k in acc:
            acc[k] = acc[k] + g[k]
    assert sorted(seen_m) == list(mq1) and sorted(seen_b) == list(bq1)
    for k in acc:
        np.testing.assert_allclose(acc[k], gref[k], atol=1e-12)


# ---------------------------------------------------------------- P8
@pytest.mark.parametrize("C", [1, 2, 4])
def test_p8_zigzag_pair_counts_closed_form(C):
    """Per sequence and query set, rank r holds 2C c^2 + c main-prefix pairs
    (c = L/2C); the ring step that brings the rank's own block holds 2c^2 + c
    of them and every other step 2c^2."""
    K = 3
    lens = [32 * C, 64 * C]
    p = W.custom(lens, [("eagle", K), ("eagle", K)], hq=1, hkv=1, head_dim=4, cp_size=C,
                 cp_rank=0, seed=81)
    for r in range(C):
        pr = p.with_rank(r)
        n_main, n_local = oracle.allowed_pair_counts(pr)
        cs = [L // (2 * C) for L in lens]
        assert n_main == (K + 1) * sum(2 * C * c * c + c for c in cs)
        assert n_local == sum(2 * c * K * (K + 1) // 2 for c in cs)
        for j in range(C):
            nm_j, _ = oracle.allowed_pair_counts(pr, key_filter=_chunk_filter(C, j))
            per = sum((2 * c * c + c) if j == r else 2 * c * c for c in cs)
            assert nm_j == (K + 1) * per


def test_p8_dflash_pair_counts():
    p = W.custom([128], [("dflash", 16, 64)], hq=1, hkv=1, head_dim=4, cp_size=1, seed=82)
    n_main, n_local = oracle.allowed_pair_counts(p)
    assert n_main == sum(16 * (a + 1) for a in p.g_anchor)
    assert n_local == 256 * len(p.g_anchor)


# ---------------------------------------------------------------- P9
def test_p9_dflash_block_is_permutation_equivariant():
    p = W.custom([32], [("dflash", 8, 16)], hq=2, hkv=1, head_dim=8, cp_size=1, seed=91)
    t = draw_all(p)
    mq, bq = oracle.select_queries(p)
    out = oracle.forward(p, *[t[k] for k in TENSORS], mq, bq)
    perm = np.random.default_rng(92).permutation(8)
    t2 = dict(t)
    for k in ("qb", "kb", "vb"):
        a = t[k].copy()
        a[p.g_row0[0]:p.g_row0[0] + 8] = t[k][p.g_row0[0] + perm]
        t2[k] = a
    out2 = oracle.forward(p, *[t2[k] for k in TENSORS], mq, bq)
    r0 = np.searchsorted(bq, p.g_row0[0])
    np.testing.assert_allclose(out2[2][r0:r0 + 8], out[2][r0 + perm], atol=1e-13)
    np.testing.assert_allclose(out2[3][:, r0:r0 + 8], out[3][:, r0 + perm], atol=1e-13)
