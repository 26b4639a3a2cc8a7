"""One round end to end, and decision margins (oracle; test infrastructure).

``build_round`` chains the three steps of the hot path for one round: the
per-position marginals and top-K (Sec. 3.2), Algorithm 1 (Sec. 4.5), and the
tree layout with its attention mask and position ids (Sec. 3.3).

``decision_margins`` measures how close a round sits to a decision boundary,
for the input guard that keeps floating-point decisions unambiguous:

* stop margins: at every tested pop, Lemma 1 (eq. stopping) says the node is
  kept iff delta * C(n) > (1 + Phi) * c_{n+1}, where c_{n+1} = C(n+1) - C(n);
  the margin is |delta C(n) - (1 + Phi) c_{n+1}| / (delta C(n) + (1 + Phi)
  c_{n+1}), and 1 when c_{n+1} = 0 (the node is always kept then);
* cross-depth gap: a perturbation of the log-normalisers shifts every sigma at
  depth d by the same amount, so the kept set can only change through a
  comparison between a kept node and a frontier node at a different depth;
  the gap is min over depths d != d' of (min sigma of kept nodes at d) - (max
  sigma of frontier nodes at d').
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

from .vocab import marginals
from .alg1 import expand, Expansion
from .layout import canonical_order, emit_mask, TreeOut


@dataclasses.dataclass
class RoundResult:
    marg: dict
    exp: Expansion
    tree: TreeOut
    mask: Optional[np.ndarray]

    @property
    def n_star(self) -> int:
        return self.exp.n_star


def build_round(logits: np.ndarray, dtype: str, K: int, t_draft: float, t_verify: np.ndarray,
                cap: int, pos_offset: int = 0, mask: str = "u8",
                budget: Optional[int] = None) -> RoundResult:
    marg = marginals(logits, dtype, K)
    ex = expand(marg["logit"], marg["lse"], t_draft, t_verify, cap, budget=budget)
    tree = canonical_order([nd.ranks for nd in ex.selected], ex.deltas, marg["ids"], pos_offset)
    m = None if mask == "none" else emit_mask(tree.parent, mask, cap)
    return RoundResult(marg, ex, tree, m)


def decision_margins(ex: Expansion):
    """Returns (min stop margin over tested pops, min cross-depth gap); inf if none apply."""
    stop = math.inf
    for s in ex.steps:
        c = s.c_next - s.c_n
        if c == 0.0:
            continue
        a = s.delta * s.c_n
        b = (1.0 + s.phi) * c
        stop = min(stop, abs(a - b) / (abs(a) + abs(b)))
    kept_min = {}
    for nd in ex.selected:
        kept_min[nd.depth] = min(kept_min.get(nd.depth, math.inf), nd.sigma)
    front_max = {}
    for nd in ex.frontier:
        front_max[nd.depth] = max(front_max.get(nd.depth, -math.inf), nd.sigma)
    gap = math.inf
    for d, lo in kept_min.items():
        for d2, hi in front_max.items():
            if d2 != d:
                gap = min(gap, lo - hi)
    return stop, gap
