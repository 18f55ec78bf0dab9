"""fp64 oracle: grouped-query QKV projection with rotary embedding, the step
in front of branch attention inside a draft layer.

Test infrastructure only (see the package docstring).

The draft layer (the paper gives no projection detail; reading R20 of the
design notes takes it to be a Llama-style decoder layer) projects hidden states x [rows, hidden] with one fused linear
weight w [(hq + 2 hkv) d, hidden] (output-major, as a linear layer stores it):
y = x w^T, whose consecutive d-column blocks are the hq query heads, then the
hkv key heads, then the hkv value heads.  Queries and keys are then rotated
by their positions (:mod:`oracle.rope`: pairs j, j + d/2 by
pos * theta^(-2j/d)); a row with a negative position is left unrotated.

Backward of sum <dq, q> + <dk, k> + <dv, v>: the gradient of the unrotated
projection is dy = [R^T dq, R^T dk, dv] (the rotation is orthogonal), then
dx = dy w and dw = dy^T x.
"""

from __future__ import annotations

import numpy as np

from . import rope


def _split(y, rows, hq, hkv, d):
    q = y[:, : hq * d].reshape(rows, hq, d)
    k = y[:, hq * d: (hq + hkv) * d].reshape(rows, hkv, d)
    v = y[:, (hq + hkv) * d:].reshape(rows, hkv, d)
    return q, k, v


def _turn(a, pos, theta, inverse):
    """Rotate the rows of ``a [rows, H, d]`` whose position is >= 0."""
    if not theta:
        return a
    pos = np.asarray(pos, np.int64)
    out = a.copy()
    m = pos >= 0
    if m.any():
        out[m] = rope.rotate(a[m], pos[m], theta, inverse=inverse)
    return out


def forward(x, w, hq: int, hkv: int, pos, theta: float, head_dim: int = 128):
    """(q [rows, hq, d], k [rows, hkv, d], v [rows, hkv, d]) in float64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    rows = x.shape[0]
    assert w.shape == ((hq + 2 * hkv) * head_dim, x.shape[1])
    q, k, v = _split(x @ w.T, rows, hq, hkv, head_dim)
    return _turn(q, pos, theta, False), _turn(k, pos, theta, False), v


def grad_y(dq, dk, dv, pos, theta: float):
    """dy [rows, (hq + 2 hkv) d]: the gradient of the unrotated projection."""
    dq, dk, dv = (np.asarray(a, np.float64) for a in (dq, dk, dv))
    rows = dq.shape[0]
    parts = [_turn(dq, pos, theta, True), _turn(dk, pos, theta, True), dv]
    return np.concatenate([p.reshape(rows, -1) for p in parts], axis=1)


def backward(x, w, hq: int, hkv: int, pos, theta: float, dq, dk, dv):
    """(dx [rows, hidden], dw [(hq + 2 hkv) d, hidden]) in float64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    dy = grad_y(dq, dk, dv, pos, theta)
    return dy @ w, dy.T @ x
