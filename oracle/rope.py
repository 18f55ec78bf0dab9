"""fp64 oracle: rotary position embedding on the inputs of branch attention.

Test infrastructure only (see the package docstring).

Inside a draft layer the step right before branch attention rotates every
query and key by its position (rotary position embedding, as in the Llama
family of target models that the paper's drafts attach to).  The paper names
no positional scheme for branch tokens; the readings taken here:

* a main token at position p of its sequence has position p;
* member i (0-based) of a branch group anchored at a has position a + 1 + i:
  an EAGLE-3 chain member of depth k = i + 1 stands k positions after its
  anchor (the draft step it simulates), a DFlash block member i stands i + 1
  positions after the anchor (the block continues the sequence);
* the rotation pairs dims j and j + d/2 (j < d/2) and turns them by the angle
  pos * theta^(-2j/d):  x_j' = x_j cos - x_{j+d/2} sin,
  x_{j+d/2}' = x_{j+d/2} cos + x_j sin.

Values (V) are not rotated.  The gradient of a rotated input maps back to the
unrotated one through the transposed rotation (the rotation is orthogonal).
"""

from __future__ import annotations

import numpy as np

from . import attention


def positions(prob, n_br=None):
    """Positions of every global main row and branch row: ``(pos_main [N],
    pos_br [n_br])``; branch rows outside every group get 0.  ``n_br``
    defaults to the end of the last group's rows."""
    cu = np.asarray(prob.cu_seqlens, np.int64)
    pos_main = np.concatenate([np.arange(cu[s + 1] - cu[s]) for s in range(len(cu) - 1)]) \
        if len(cu) > 1 else np.zeros(0, np.int64)
    if n_br is None:
        n_br = int(np.max(np.asarray(prob.g_row0) + np.asarray(prob.g_len))) if len(prob.g_len) else 0
    pos_br = np.zeros(int(n_br), np.int64)
    for g in range(len(prob.g_len)):
        r0, n = int(prob.g_row0[g]), int(prob.g_len[g])
        pos_br[r0:r0 + n] = int(prob.g_anchor[g]) + 1 + np.arange(n)
    return pos_main.astype(np.int64), pos_br


def angles(pos, head_dim: int, theta: float):
    """Rotation angle of every (row, pair j): pos * theta^(-2j/d), [rows, d/2]."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(float(theta), -2.0 * j / head_dim)
    return np.asarray(pos, np.float64)[:, None] * inv_freq[None, :]


def rotate(x, pos, theta: float, inverse: bool = False):
    """Rotate rows ``x [rows, H, d]`` by their positions ``pos [rows]``;
    ``inverse`` applies the transposed rotation."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    a = angles(pos, d, theta)[:, None, :]
    c, s = np.cos(a), np.sin(a)
    if inverse:
        s = -s
    lo, hi = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def round_bf16(x):
    """Round to the nearest bfloat16 value (8 significant bits, ties to
    even); values are assumed inside bfloat16's normal range or zero."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)  # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def _rotated_inputs(prob, qm, km, qb, kb, theta, rounded):
    pm, pb = positions(prob, len(np.asarray(qb)))
    rq = round_bf16 if rounded else (lambda a: a)
    return (rq(rotate(qm, pm, theta)), rq(rotate(km, pm, theta)), rq(rotate(qb, pb, theta)),
            rq(rotate(kb, pb, theta)), pm, pb)


def forward(prob, qm, km, vm, qb, kb, vb, theta: float, rounded: bool = False, **kw):
    """Branch attention of the rotated queries and keys (see
    :func:`attention.forward` for the arguments and results).  ``rounded``
    rounds the rotated queries and keys to bfloat16 before attending (a
    draft layer computing in bfloat16 hands them over in that type)."""
    rqm, rkm, rqb, rkb, _, _ = _rotated_inputs(prob, qm, km, qb, kb, theta, rounded)
    return attention.forward(prob, rqm, rkm, vm, rqb, rkb, vb, **kw)


def backward(prob, qm, km, vm, qb, kb, vb, dom, dob, theta: float, main_q=None, br_q=None,
             rounded: bool = False, **kw):
    """Gradients with respect to the unrotated inputs: the attention backward
    on the rotated inputs, then the transposed rotation of dQ and dK (the
    bfloat16 rounding of ``rounded`` passes gradients through unchanged)."""
    if main_q is None or br_q is None:
        mq0, bq0 = attention.select_queries(prob)
        main_q = mq0 if main_q is None else main_q
        br_q = bq0 if br_q is None else br_q
    main_q = np.asarray(main_q, np.int64)
    br_q = np.asarray(br_q, np.int64)
    rqm, rkm, rqb, rkb, pm, pb = _rotated_inputs(prob, qm, km, qb, kb, theta, rounded)
    g = attention.backward(prob, rqm, rkm, vm, rqb, rkb, vb, dom, dob, main_q=main_q, br_q=br_q, **kw)
    g["dq_main"] = rotate(g["dq_main"], pm[main_q], theta, inverse=True)
    g["dq_br"] = rotate(g["dq_br"], pb[br_q], theta, inverse=True)
    g["dk_main"] = rotate(g["dk_main"], pm, theta, inverse=True)
    g["dk_br"] = rotate(g["dk_br"], pb, theta, inverse=True)
    return g
