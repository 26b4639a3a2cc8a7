"""CPU oracle for CaDDTree draft-tree construction (TEST INFRASTRUCTURE).

This package is a plain, slow, deliberately literal fp64 implementation of what
the GPU hot path computes, written from the paper (Cost-Aware Diffusion Draft
Trees for Speculative Decoding, arXiv 2606.01813).  It exists to check the GPU
library and nothing else: only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import it.  The product path never calls it, and it
shares no code with the HIP library or its Python binding.

Contents
--------
``vocab``      per-position log-normaliser and top-K (Sec. 3.2, eq. marginals;
               the Require line of Algorithm 1).
``alg1``       Algorithm 1 (Sec. 4.5): best-first expansion with the greedy
               throughput stop, plus a fixed-budget mode (the DDTree heap of
               Sec. 3.4) used by the tests.
``layout``     canonical output order, parent indices, tree-attention mask and
               position ids (Sec. 3.3).
``pipeline``   one round end to end, and the decision margins used by the
               input guard.
``cost``       context-aware verification cost: linear interpolation between
               cost tables profiled on a grid of context lengths (Sec. 4.6,
               eq. cv-interp).
``accept``     synthetic acceptance: a target path drawn from the drafter's
               factorised distribution, the accepted length under tree
               verification (Sec. 3.3, eq. surrogate) and the throughput
               sum (1 + alpha) / sum C (Sec. 4.2).
``costfit``    convex non-decreasing least-squares fit of a cost profile and the
               cost table built from it (Sec. 4.6, eq. convex-reg).

Precision: fp64 throughout (bf16 and fp32 logits are widened exactly).
"""

from .vocab import widen, log_normalizer, top_k, marginals
from .alg1 import expand, Expansion
from .layout import canonical_order, emit_mask, TreeOut
from .pipeline import build_round, RoundResult, Margins, decision_margins
from .cost import context_cost
from . import accept, costfit

__all__ = [
    "widen", "log_normalizer", "top_k", "marginals",
    "expand", "Expansion",
    "canonical_order", "emit_mask", "TreeOut",
    "build_round", "RoundResult", "Margins", "decision_margins",
    "context_cost", "accept", "costfit",
]
