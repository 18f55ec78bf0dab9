"""Seeded synthetic workloads for draft branch attention.

This module only *describes and draws* inputs: sequence lengths, where the
draft branches sit, and the bf16 tensors.  It contains no attention
arithmetic, no context-parallel partitioning and no masking; both the HIP
path and the CPU oracle consume what it produces and interpret it on their
own.

Problem description (global, i.e. before any context-parallel split):

* ``cu_seqlens`` -- int64 ``[S+1]`` prefix sums of the packed main sequences.
* ``has_main`` -- bool ``[S]``: whether the main-sequence tokens of a sequence
  are themselves queries (EAGLE-3 training trains depth 0 too; a DFlash-style
  draft only trains its blocks).
* Branch groups, one entry per branch: ``g_seq``, ``g_anchor`` (position in
  the sequence the branch hangs off), ``g_kind`` (``KIND_EAGLE`` = chain in
  which member i sees members 0..i, ``KIND_DFLASH`` = block in which every
  member sees every member), ``g_len`` and ``g_row0`` (first row of the group
  in the global branch arrays; the members of a group are consecutive rows).
* Heads ``hq``/``hkv``, ``head_dim`` and the softmax ``scale``.
* ``cp_size``/``cp_rank`` -- which context-parallel rank share is evaluated.

Tensor draws are row-addressable: row block ``b`` (``ROW_BLOCK`` rows) of
tensor ``t`` is ``default_rng([seed, t, b]).standard_normal((rows, H, d))``
in float32, rounded to bf16 (round-to-nearest-even).  A rank share is thus a
row selection of one global problem, and any subset of rows can be drawn
without drawing the rest.

The five named workloads follow the evaluation configurations of the
branch-attention study (Sec. 4.4 of the paper describes the CP benchmark;
the shapes here are synthetic stand-ins, see the ``describe`` strings).
"""

from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

KIND_EAGLE = 0
KIND_DFLASH = 1

ROW_BLOCK = 1024

# tensor ids of the row-addressable draws
TENSOR_IDS = {"qm": 0, "km": 1, "vm": 2, "qb": 3, "kb": 4, "vb": 5, "dom": 6, "dob": 7}


@dataclasses.dataclass
class GlobalProblem:
    name: str
    seed: int
    cu_seqlens: np.ndarray          # int64 [S+1]
    has_main: np.ndarray            # bool  [S]
    g_seq: np.ndarray               # int64 [G]
    g_anchor: np.ndarray            # int64 [G]
    g_kind: np.ndarray              # int64 [G]
    g_len: np.ndarray               # int64 [G]
    g_row0: np.ndarray              # int64 [G]
    hq: int
    hkv: int
    head_dim: int
    scale: float
    cp_size: int
    cp_rank: int
    backward: bool = True
    describe: str = ""

    # ------------------------------------------------------------------
    @property
    def num_seqs(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def seqlens(self) -> np.ndarray:
        return np.diff(self.cu_seqlens)

    @property
    def n_main(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def n_branch(self) -> int:
        return int(self.g_len.sum()) if len(self.g_len) else 0

    def with_rank(self, rank: int) -> "GlobalProblem":
        return dataclasses.replace(self, cp_rank=int(rank))

    def heads_of(self, tensor: str) -> int:
        return self.hq if tensor in ("qm", "qb", "dom", "dob") else self.hkv

    # ------------------------------------------------------------------
    def draw(self, tensor: str, rows: Optional[np.ndarray] = None,
             zero: bool = False) -> torch.Tensor:
        """bf16 CPU tensor ``[len(rows), H, d]`` of the given global rows.

        ``rows`` defaults to every row of that tensor.  ``zero`` returns zeros
        of the same shape (used for closed-form tests with Q = 0)."""
        total = self.n_main if tensor in ("qm", "km", "vm", "dom") else self.n_branch
        if rows is None:
            rows = np.arange(total, dtype=np.int64)
        rows = np.asarray(rows, dtype=np.int64)
        H, d = self.heads_of(tensor), self.head_dim
        if zero or len(rows) == 0:
            return torch.zeros((len(rows), H, d), dtype=torch.bfloat16)
        if rows.min() < 0 or rows.max() >= total:
            raise IndexError(f"row out of range for tensor {tensor}")
        tid = TENSOR_IDS[tensor]
        out = torch.empty((len(rows), H, d), dtype=torch.bfloat16)
        blocks = rows // ROW_BLOCK
        order = np.argsort(blocks, kind="stable")
        sb = blocks[order]
        starts = np.flatnonzero(np.r_[True, sb[1:] != sb[:-1]])
        ends = np.r_[starts[1:], len(sb)]

        def one(se):
            st, en = se
            b = int(sb[st])
            nrows = min(ROW_BLOCK, total - b * ROW_BLOCK)
            blk = np.random.default_rng([self.seed, tid, b]).standard_normal(
                (nrows, H, d), dtype=np.float32)
            blk_t = torch.from_numpy(blk).to(torch.bfloat16)
            sel = order[st:en]
            out[torch.from_numpy(sel)] = blk_t[torch.from_numpy(rows[sel] - b * ROW_BLOCK)]

        jobs = list(zip(starts, ends))
        if len(jobs) > 4:
            # block streams are independent, so the draw order does not matter
            with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
                list(ex.map(one, jobs))
        else:
            for j in jobs:
                one(j)
        return out


# ----------------------------------------------------------------------
# construction helpers

def _groups_for(cu: np.ndarray, spec: Sequence[Tuple], rng: Optional[np.random.Generator]):
    """Lay out the branch groups of every sequence.

    ``spec[s]`` is ``None`` (no branches), ``("eagle", K)`` (one chain of K
    tokens at every position) or ``("dflash", block, window[, nblocks])``
    (``nblocks``, default 1, blocks of ``block`` tokens per ``window``
    positions, each anchored at a uniform position inside its window; anchors
    are drawn from ``rng`` in sequence order, window by window)."""
    g_seq, g_anchor, g_kind, g_len = [], [], [], []
    for s, sp in enumerate(spec):
        L = int(cu[s + 1] - cu[s])
        if sp is None:
            continue
        if sp[0] == "eagle":
            K = int(sp[1])
            if K <= 0:
                continue
            g_seq.append(np.full(L, s))
            g_anchor.append(np.arange(L))
            g_kind.append(np.full(L, KIND_EAGLE))
            g_len.append(np.full(L, K))
        elif sp[0] == "dflash":
            block, window = int(sp[1]), int(sp[2])
            nb = int(sp[3]) if len(sp) > 3 else 1
            nwin = L // window
            offs = rng.integers(0, window, size=nwin * nb) if nb > 1 else rng.integers(0, window, size=nwin)
            g_seq.append(np.full(nwin * nb, s))
            g_anchor.append(np.repeat(np.arange(nwin) * window, nb) + offs)
            g_kind.append(np.full(nwin * nb, KIND_DFLASH))
            g_len.append(np.full(nwin * nb, block))
        else:
            raise ValueError(sp)
    cat = lambda xs: (np.concatenate(xs).astype(np.int64) if xs else np.zeros(0, np.int64))
    g_seq, g_anchor, g_kind, g_len = map(cat, (g_seq, g_anchor, g_kind, g_len))
    g_row0 = np.concatenate([[0], np.cumsum(g_len)[:-1]]).astype(np.int64) if len(g_len) else g_len.copy()
    return g_seq, g_anchor, g_kind, g_len, g_row0


def custom(seqlens: Sequence[int], spec: Sequence[Optional[Tuple]], *, hq: int, hkv: int,
           head_dim: int = 128, cp_size: int = 1, cp_rank: int = 0, seed: int = 0,
           has_main: Optional[Sequence[bool]] = None, anchor_seed: Optional[int] = None,
           scale: Optional[float] = None, name: str = "custom",
           backward: bool = True) -> GlobalProblem:
    """Build a problem from explicit lengths and per-sequence branch specs.
    By default a sequence has main queries unless its spec is DFlash."""
    seqlens = np.asarray(seqlens, dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int64)
    rng = np.random.default_rng(seed if anchor_seed is None else anchor_seed)
    g = _groups_for(cu, spec, rng)
    if has_main is None:
        has_main = [not (sp is not None and sp[0] == "dflash") for sp in spec]
    return GlobalProblem(
        name=name, seed=seed, cu_seqlens=cu, has_main=np.asarray(has_main, dtype=bool),
        g_seq=g[0], g_anchor=g[1], g_kind=g[2], g_len=g[3], g_row0=g[4],
        hq=hq, hkv=hkv, head_dim=head_dim,
        scale=(1.0 / math.sqrt(head_dim)) if scale is None else float(scale),
        cp_size=cp_size, cp_rank=cp_rank, backward=backward)


def config(n: int) -> GlobalProblem:
    """The five named workloads (structure RNG seeded with the config number)."""
    if n == 1:
        p = custom([1024], [("eagle", 3)], hq=8, hkv=8, cp_size=4, cp_rank=0, seed=1,
                   name="eagle3-K3-L1024-cp4", backward=False)
        p.describe = ("single 1024-token sequence, 8/8 heads, EAGLE-3 chains of depth 3, "
                      "CP=4 zigzag (every rank evaluated), forward only")
        return p
    if n == 2:
        rng = np.random.default_rng(2)
        L = rng.integers(2048, 16384, 8, endpoint=True)
        L = np.clip(np.rint(L / 128).astype(np.int64) * 128, 2048, 16384)
        p = custom(L, [("eagle", 7)] * 8, hq=32, hkv=8, cp_size=4, cp_rank=0, seed=2,
                   name="varlen8-eagle3-K7-cp4r0")
        p.describe = (f"8 packed sequences (sum {int(L.sum())} tokens), 32/8 heads, EAGLE-3 "
                      "depth 7, CP=4 rank 0, fwd+bwd")
        return p
    if n == 3:
        p = custom([32768], [("dflash", 16, 64)], hq=64, hkv=8, cp_size=1, cp_rank=0, seed=3,
                   anchor_seed=3, name="dflash16-L32768")
        p.describe = ("single 32768-token sequence, 64/8 heads, one 16-token DFlash block per "
                      "64 positions, block queries only, fwd+bwd")
        return p
    if n == 4:
        p = custom([262144], [("eagle", 3)], hq=32, hkv=8, cp_size=8, cp_rank=0, seed=4,
                   name="eagle3-K3-L262144-cp8r0")
        p.describe = ("one 262144-token sequence, 32/8 heads, EAGLE-3 depth 3, CP=8 rank 0 "
                      "share (32768 main + 98304 branch queries vs 262144 main keys), fwd+bwd")
        return p
    if n == 5:
        rng = np.random.default_rng(5)
        x = rng.lognormal(math.log(6144), 0.7585, 16)
        x = np.clip(x, 1024, 32768)
        x = x * 131072 / x.sum()
        x = np.clip(x, 1024, 32768)
        L = (np.rint(x / 128) * 128).astype(np.int64)
        L[int(np.argmax(L))] += 131072 - int(L.sum())
        spec = [("eagle", 5) if s % 2 == 0 else ("dflash", 16, 64) for s in range(16)]
        cu = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
        g = _groups_for(cu, spec, rng)  # anchors drawn after the lengths, same stream
        p = GlobalProblem(
            name="mixed16-eagle5-dflash16-cp8r3", seed=5, cu_seqlens=cu,
            has_main=np.array([s % 2 == 0 for s in range(16)]),
            g_seq=g[0], g_anchor=g[1], g_kind=g[2], g_len=g[3], g_row0=g[4],
            hq=64, hkv=4, head_dim=128, scale=1.0 / math.sqrt(128), cp_size=8, cp_rank=3)
        p.describe = ("16 packed lognormal sequences (sum 131072), 64/4 heads, even sequences "
                      "EAGLE-3 depth 5, odd sequences DFlash 16-token blocks per 64, CP=8 rank 3")
        return p
    raise ValueError(f"unknown config {n}")


CONFIG_IDS = (1, 2, 3, 4, 5)
