"""Pins of the QKV-projection oracle (`oracle.qkv`) and host-side checks of
the projection's C entry points (argument validation only: no GPU here).

Q1 torch's linear layer in float64 followed by the Llama rotary routine of
the transformers library (a library composition that fixes the weight
layout, the q / k / v head order and which heads turn), Q2 central finite
differences of sum <dq, q> + <dk, k> + <dv, v> with respect to x and w (pins
the transposed rotation and both products of the backward), Q3 theta 0 and
negative positions leave rows unrotated, Q4 the plan's positions match the
oracle's position rule on every rank of two workloads.
"""

import ctypes

import numpy as np
import pytest
import torch

from oracle import qkv, rope
from paper_2609_07108_amd import binding as B
from paper_2609_07108_amd import rankshare as RS
from paper_2609_07108_amd import workloads as W


def _draw(rng, rows, hidden, hq, hkv, d):
    x = rng.standard_normal((rows, hidden))
    w = rng.standard_normal(((hq + 2 * hkv) * d, hidden)) / np.sqrt(hidden)
    return x, w


@pytest.mark.parametrize("hq,hkv,theta", [(4, 2, 1.0e4), (2, 2, 5.0e5), (8, 1, 50.0)])
def test_q1_linear_then_llama_rotary(hq, hkv, theta):
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb

    d, hidden, rows = 128, 256, 24
    rng = np.random.default_rng(81)
    x, w = _draw(rng, rows, hidden, hq, hkv, d)
    pos = rng.integers(0, 300, rows)  # float32 angle tables of the library stay accurate here
    y = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(w))  # float64
    q = y[:, : hq * d].reshape(rows, hq, d)
    k = y[:, hq * d: (hq + hkv) * d].reshape(rows, hkv, d)
    v = y[:, (hq + hkv) * d:].reshape(rows, hkv, d)
    cfg = LlamaConfig(hidden_size=hq * d, num_attention_heads=hq, num_key_value_heads=hkv, head_dim=d,
                      rope_theta=theta)
    cos, sin = LlamaRotaryEmbedding(config=cfg)(torch.zeros(1, dtype=torch.float32), torch.as_tensor(pos)[None])
    qr, kr = apply_rotary_pos_emb(q.permute(1, 0, 2)[None], k.permute(1, 0, 2)[None], cos.double(), sin.double())
    ref = (qr[0].permute(1, 0, 2).numpy(), kr[0].permute(1, 0, 2).numpy(), v.numpy())
    got = qkv.forward(x, w, hq, hkv, pos, theta)
    for g, r in zip(got, ref):
        assert g.shape == r.shape
        # the library tabulates cos / sin in float32
        assert np.max(np.abs(g - r)) <= 5e-5 * np.max(np.abs(r))
    # and the rotation did act on q and k
    plain = qkv.forward(x, w, hq, hkv, pos, 0.0)
    assert np.max(np.abs(plain[0] - got[0])) > 0.1 and np.max(np.abs(plain[1] - got[1])) > 0.1
    assert np.array_equal(plain[2], got[2])


def test_q2_finite_differences():
    d, hidden, rows, hq, hkv, theta = 8, 6, 5, 4, 2, 20.0
    rng = np.random.default_rng(82)
    x, w = _draw(rng, rows, hidden, hq, hkv, d)
    pos = np.array([0, 3, -1, 17, 40])
    dq = rng.standard_normal((rows, hq, d))
    dk = rng.standard_normal((rows, hkv, d))
    dv = rng.standard_normal((rows, hkv, d))

    def loss(x_, w_):
        q, k, v = qkv.forward(x_, w_, hq, hkv, pos, theta, head_dim=d)
        return float(np.sum(q * dq) + np.sum(k * dk) + np.sum(v * dv))

    dx, dw = qkv.backward(x, w, hq, hkv, pos, theta, dq, dk, dv)
    h = 1e-6
    for a, g in ((x, dx), (w, dw)):
        for _ in range(25):
            idx = tuple(int(rng.integers(n)) for n in a.shape)
            old = a[idx]
            a[idx] = old + h
            lp = loss(x, w)
            a[idx] = old - h
            lm = loss(x, w)
            a[idx] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g[idx]) <= 1e-6 * max(1.0, abs(g[idx])), (idx, fd, g[idx])


def test_q3_unrotated_rows():
    d, hidden, rows, hq, hkv = 16, 32, 6, 2, 1
    rng = np.random.default_rng(83)
    x, w = _draw(rng, rows, hidden, hq, hkv, d)
    pos = np.array([5, -1, 7, -3, 0, 9])
    y = x @ w.T
    q, k, v = qkv.forward(x, w, hq, hkv, pos, 1.0e4, head_dim=d)
    for r in (1, 3, 4):  # negative positions and position 0 (angle 0)
        assert np.allclose(q[r].ravel(), y[r, : hq * d], rtol=0, atol=1e-12)
        assert np.allclose(k[r].ravel(), y[r, hq * d: (hq + hkv) * d], rtol=0, atol=1e-12)
    assert np.max(np.abs(q[0].ravel() - y[0, : hq * d])) > 1e-3
    q0, k0, _ = qkv.forward(x, w, hq, hkv, pos, 0.0, head_dim=d)
    assert np.allclose(q0.reshape(rows, -1), y[:, : hq * d], atol=1e-12)


@pytest.mark.parametrize("cfg", [2, 5])
def test_q4_plan_positions_match_oracle(cfg):
    base = W.config(cfg)
    for r in range(base.cp_size):
        prob = base.with_rank(r)
        share = RS.build_share(prob, materialize=False)
        mp, bp = share.plan.positions(share.n_local, share.num_branch_rows)
        pm, pb = rope.positions(prob)
        assert np.array_equal(mp, pm[share.l2g])
        ref = np.full(share.num_branch_rows, -1, np.int64)
        ref[share.br_rows_local] = pb[share.br_rows_global]
        assert np.array_equal(bp, ref)


# ------------------------------------------------- host-side validation


def _fwd(rows, hidden, hq, hkv, theta=0.0, ptr=None):
    return B.lib().branch_attn_qkv_fwd(None, rows, hidden, hq, hkv, ptr, ptr, ptr, theta, ptr, ptr, ptr)


def test_qkv_argument_checks():
    assert _fwd(0, 128, 4, 2) == B.BA_OK  # nothing to do, nothing launched
    assert _fwd(0, 96, 4, 2) == B.BA_E_UNSUPPORTED
    assert _fwd(0, 128, 4, 3) == B.BA_E_INVAL
    assert _fwd(0, 128, 4, 2, theta=-1.0) == B.BA_E_INVAL
    assert _fwd(0, 128, 4, 2, theta=float("nan")) == B.BA_E_INVAL
    assert _fwd(5, 128, 4, 2) == B.BA_E_INVAL  # NULL x / w
    assert _fwd(5, 128, 4, 2, ptr=ctypes.c_void_p(0x1008)) == B.BA_E_INVAL  # misaligned
    assert B.branch_attn_qkv_workspace_size(10, 4, 2) == 10 * 8 * 128 * 2
    L = B.lib()
    fake = ctypes.c_void_p(0x10000)  # aligned, never dereferenced: validation fails first
    rc = L.branch_attn_qkv_bwd(None, 4, 128, 4, 2, fake, fake, None, 0.0, fake, fake, fake, B.BA_DTYPE_BF16, fake,
                               B.BA_DTYPE_F32, fake, 0, fake, 100)
    assert rc == B.BA_E_WORKSPACE
    rc = L.branch_attn_qkv_bwd(None, 4, 128, 4, 2, fake, fake, None, 0.0, fake, fake, fake, 7, fake,
                               B.BA_DTYPE_F32, fake, 0, fake, 1 << 20)
    assert rc == B.BA_E_INVAL
    rc = L.branch_attn_qkv_bwd(None, 4, 128, 4, 2, fake, fake, None, 1.0e4, fake, fake, fake, B.BA_DTYPE_BF16, fake,
                               B.BA_DTYPE_F32, fake, 0, fake, 1 << 20)
    assert rc == B.BA_E_INVAL  # theta > 0 without positions
