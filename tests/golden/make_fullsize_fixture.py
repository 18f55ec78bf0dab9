"""Write the full-size parity fixtures from the fp64 oracle.

    python tests/golden/make_fullsize_fixture.py --config 3   # ~45 min on 8 cores
    python tests/golden/make_fullsize_fixture.py --config 4   # ~8 min

Calls only ``oracle`` and the seeded input generator (``workloads``, which
draws inputs and holds no attention arithmetic).  Nothing here comes from the
HIP path.  The stored values are the oracle's float64 results rounded to
float32, so storage adds at most 2^-24 relative error.

What is stored (every choice seeded; the seed is the config number + 1000):

config 3 (one 32768-token sequence, DFlash 16-token blocks per 64 positions,
64/8 heads, CP=1, block queries only).  The oracle runs the backward over
*every* query of the share, so the gradient of every key is exact:
  * rows: 128 branch query rows spread over the share (first and last
    included), each with one query head per KV group (1024 (row, head)
    pairs): O and dQ; LSE for all 64 heads of those rows;
  * dk/dv main: 2048 (key row, KV head) pairs, 16 at each of the 128 key
    positions inside a 128-key tile, tiles drawn over the whole sequence
    (keys near the start are read by every block query: the longest walks);
  * dk/dv branch: 256 groups, 4 members and one KV head each.

config 4 (the 256K-token share, EAGLE-3 depth 3, CP=8 rank 0): 256 query rows
(32 main rows from each of the rank's two chunks, first and last included;
64 branch rows at each depth 1..3, anchors in both chunks), each against all
its keys: O and dQ at one query head per KV group, LSE at all 32 heads.  The
dK/dV of this share would need the oracle's forward over all 131072 query
rows (about 12 h on this scale of host), so its gradients are checked at
config 3 instead.
"""

from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2609_07108_amd import workloads as W  # noqa: E402

TENSORS = ("qm", "km", "vm", "qb", "kb", "vb")


def fixture_path(cfg: int) -> str:
    return os.path.join(HERE, f"fullsize_c{cfg}.npz")


def _heads_per_group(rng, n, hq, hkv):
    """One query head per KV group for each of n rows: [n, hkv]."""
    G = hq // hkv
    return (np.arange(hkv)[None, :] * G + rng.integers(0, G, size=(n, hkv))).astype(np.int64)


def _log(msg):
    print(f"[fixture] {msg}", flush=True)


def config3():
    prob = W.config(3)
    rng = np.random.default_rng(1003)
    mq, bq = oracle.select_queries(prob)
    assert len(mq) == 0
    t0 = time.time()
    t = {k: prob.draw(k).float().numpy() for k in TENSORS}
    dob = prob.draw("dob").float().numpy()
    _log(f"inputs drawn in {time.time() - t0:.0f} s")

    # sampled query rows (global branch rows)
    rows = np.unique(np.r_[rng.choice(bq, 126, replace=False), bq[0], bq[-1]])
    heads = _heads_per_group(rng, len(rows), prob.hq, prob.hkv)
    t0 = time.time()
    _, _, o_b, l_b = oracle.forward(prob, *[t[k] for k in TENSORS], mq, rows)
    _log(f"forward of {len(rows)} rows in {time.time() - t0:.0f} s")

    t0 = time.time()
    g = oracle.backward(prob, *[t[k] for k in TENSORS], np.zeros((0, prob.hq, prob.head_dim)), dob[bq], mq, bq)
    _log(f"backward of all {len(bq)} rows in {time.time() - t0:.0f} s")
    pos_in_bq = np.searchsorted(bq, rows)
    assert np.all(bq[pos_in_bq] == rows)

    # main keys: 16 at each position inside a 128-key tile
    L = prob.n_main
    ntile = L // 128
    key_rows = (rng.integers(0, ntile, size=2048) * 128 + np.tile(np.arange(128), 16)).astype(np.int64)
    key_heads = rng.integers(0, prob.hkv, size=2048).astype(np.int64)
    # branch keys: 256 groups x 4 members, one KV head each
    ng = len(prob.g_len)
    gsel = np.sort(rng.choice(ng, 256, replace=False))
    mem = np.stack([np.sort(rng.choice(int(prob.g_len[gg]), 4, replace=False)) for gg in gsel])
    br_key_rows = (prob.g_row0[gsel][:, None] + mem).reshape(-1).astype(np.int64)
    br_key_heads = np.repeat(rng.integers(0, prob.hkv, size=256), 4).astype(np.int64)

    ri = np.arange(len(rows))[:, None]
    out = dict(
        config=np.int64(3),
        q_main_rows=np.zeros(0, np.int64), q_main_heads=np.zeros((0, prob.hkv), np.int64),
        o_main=np.zeros((0, prob.hkv, prob.head_dim), np.float32),
        lse_main=np.zeros((prob.hq, 0), np.float32),
        dq_main=np.zeros((0, prob.hkv, prob.head_dim), np.float32),
        q_br_rows=rows, q_br_heads=heads,
        o_br=o_b[ri, heads].astype(np.float32),
        lse_br=l_b.astype(np.float32),
        dq_br=g["dq_br"][pos_in_bq[:, None], heads].astype(np.float32),
        key_rows=key_rows, key_heads=key_heads,
        dk_main=g["dk_main"][key_rows, key_heads].astype(np.float32),
        dv_main=g["dv_main"][key_rows, key_heads].astype(np.float32),
        br_key_rows=br_key_rows, br_key_heads=br_key_heads,
        dk_br=g["dk_br"][br_key_rows, br_key_heads].astype(np.float32),
        dv_br=g["dv_br"][br_key_rows, br_key_heads].astype(np.float32),
    )
    return out


def config4():
    prob = W.config(4)
    rng = np.random.default_rng(1004)
    mq, bq = oracle.select_queries(prob)
    L = prob.n_main
    c = L // (2 * prob.cp_size)
    lo_chunk = mq[mq < c]
    hi_chunk = mq[mq >= c]
    sm = np.unique(np.r_[rng.choice(lo_chunk, 31, replace=False), lo_chunk[0],
                         rng.choice(hi_chunk, 31, replace=False), hi_chunk[-1]])
    # branch rows: members of the groups are consecutive (g_row0 + depth - 1)
    grp = np.repeat(np.arange(len(prob.g_len)), prob.g_len)
    depth = np.arange(prob.n_branch) - prob.g_row0[grp]
    sb = []
    for k in range(3):
        cand = bq[depth[bq] == k]
        anch = prob.g_anchor[grp[cand]]
        sb.append(rng.choice(cand[anch < c], 32, replace=False))
        sb.append(rng.choice(cand[anch >= c], 32, replace=False))
    sb = np.unique(np.concatenate(sb))

    H, Hk, d = prob.hq, prob.hkv, prob.head_dim

    def sparse(name, sel, total, heads):
        a = np.zeros((total, heads, d), np.float32)
        if len(sel):
            a[sel] = prob.draw(name, sel).float().numpy()
        return a

    gsel = np.unique(grp[sb])
    brows = np.concatenate([np.arange(prob.g_row0[g], prob.g_row0[g] + prob.g_len[g]) for g in gsel])
    t0 = time.time()
    t = dict(qm=sparse("qm", sm, prob.n_main, H), qb=sparse("qb", sb, prob.n_branch, H),
             km=prob.draw("km").float().numpy(), vm=prob.draw("vm").float().numpy(),
             kb=sparse("kb", brows, prob.n_branch, Hk), vb=sparse("vb", brows, prob.n_branch, Hk))
    dom = prob.draw("dom", sm).float().numpy()
    dob = prob.draw("dob", sb).float().numpy()
    _log(f"inputs drawn in {time.time() - t0:.0f} s")
    args = [t[k] for k in TENSORS]
    t0 = time.time()
    o_m, l_m, o_b, l_b = oracle.forward(prob, *args, sm, sb)
    _log(f"forward of {len(sm)} + {len(sb)} rows in {time.time() - t0:.0f} s")
    t0 = time.time()
    g = oracle.backward(prob, *args, dom, dob, sm, sb)
    _log(f"backward in {time.time() - t0:.0f} s")
    hm = _heads_per_group(rng, len(sm), H, Hk)
    hb = _heads_per_group(rng, len(sb), H, Hk)
    im = np.arange(len(sm))[:, None]
    ib = np.arange(len(sb))[:, None]
    empty_k = np.zeros((0, d), np.float32)
    return dict(
        config=np.int64(4),
        q_main_rows=sm, q_main_heads=hm, o_main=o_m[im, hm].astype(np.float32),
        lse_main=l_m.astype(np.float32), dq_main=g["dq_main"][im, hm].astype(np.float32),
        q_br_rows=sb, q_br_heads=hb, o_br=o_b[ib, hb].astype(np.float32),
        lse_br=l_b.astype(np.float32), dq_br=g["dq_br"][ib, hb].astype(np.float32),
        key_rows=np.zeros(0, np.int64), key_heads=np.zeros(0, np.int64), dk_main=empty_k, dv_main=empty_k,
        br_key_rows=np.zeros(0, np.int64), br_key_heads=np.zeros(0, np.int64), dk_br=empty_k, dv_br=empty_k,
    )


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, choices=(3, 4), required=True)
    a = ap.parse_args()
    t0 = time.time()
    data = config3() if a.config == 3 else config4()
    path = fixture_path(a.config)
    np.savez(path, **data)
    _log(f"wrote {path} ({os.path.getsize(path) / 1e6:.1f} MB) in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()
