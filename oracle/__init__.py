"""Plain fp64 CPU oracle for draft branch attention under context parallelism.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package; only the tests, the smoke check and the benchmark's CPU-baseline
leg do.  It shares no code with the HIP library: it re-derives every quantity
(rank ownership, masks, softmax, merge, gradients) from the paper's
definitions, written out in numpy float64 with no blocking beyond independent
query rows.

What the method computes (Sec. 3.2 of the paper): each branch query attends a
causal prefix of its main sequence plus its branch-local keys; the two partial
results are merged with the log-sum-exp rule (Eq. lse-merge).  In exact
arithmetic that equals ordinary masked softmax attention over the union of the
two key sets, which is what :func:`forward` materialises.

Pinning (see tests/test_oracle_*.py): brute-force scalar loops, the depth-0
reduction to textbook causal attention (torch SDPA in float64), the Q = 0
closed form of every row's key count, the merge identity of Eq. lse-merge,
the chain rule through the merge, central finite differences, reassembly of
all context-parallel ranks, and the closed-form zigzag pair counts.
:mod:`oracle.rope` adds rotary position embedding in front of the op
(pinned against the Llama rotary routine of the transformers library, the
relative-position identity and finite differences); :mod:`oracle.qkv` the
grouped-query QKV projection with that rotation (pinned against torch's
linear layer plus the same library routine, and finite differences).
"""

from .attention import (  # noqa: F401
    KIND_EAGLE, KIND_DFLASH, owner_rank, select_queries, forward, backward,
    lse_merge, lse_merge_backward, allowed_pair_counts, useful_flops,
)
from . import rope  # noqa: F401
from . import qkv  # noqa: F401
