"""One round end to end, and decision margins (oracle; test infrastructure).

``build_round`` chains the three steps of the hot path for one round: the
per-position marginals and top-K (Sec. 3.2), Algorithm 1 (Sec. 4.5), and the
tree layout with its attention mask and position ids (Sec. 3.3).

``decision_margins`` lists every floating-point decision of a round with its
distance from a tie, for the input guard that keeps such decisions unambiguous.
A GPU log-normaliser LSE_i may differ from the oracle's by a tiny error e_i;
that shifts sigma at depth d by -(e_1 + .. + e_d).  So each margin comes with
its depth span, the number of normalisers whose error it can carry:

* stop margins: at every stop test, Lemma 1 (eq. stopping) keeps the node iff
  delta * C(n) > (1 + Phi) * c_{n+1}, where c_{n+1} = C(n+1) - C(n); the
  margin is |delta C(n) - (1 + Phi) c_{n+1}| / (delta C(n) + (1 + Phi)
  c_{n+1}) (no margin when c_{n+1} = 0: the node is always kept then).  delta
  carries the error of the tested node's depth and Phi that of the deepest
  node kept so far; the span is the larger of the two depths;
* cross-depth gaps: the selected set can change only through a comparison
  between a selected node and a frontier node (an unselected node that would
  come next along its branch) at a different depth, since same-depth
  comparisons reduce to the raw-logit sums Lambda, which carry no normaliser.
  For depths d != d' the gap is (min sigma of selected nodes at d) - (max sigma
  of frontier nodes at d'), with span |d - d'|.
"""

from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Tuple

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


@dataclasses.dataclass
class Margins:
    stop: List[Tuple[float, int]]     # (relative stop margin, depth span), one per stop test
    cross: List[Tuple[float, int]]    # (sigma gap, depth span), one per pair of depths

    @property
    def min_stop(self) -> float:
        return min((m for m, _ in self.stop), default=math.inf)

    @property
    def min_gap(self) -> float:
        return min((g for g, _ in self.cross), default=math.inf)


def decision_margins(ex: Expansion) -> Margins:
    stop = []
    deepest = 0
    for s in ex.steps:
        c = s.c_next - s.c_n
        if c != 0.0:
            a = s.delta * s.c_n
            b = (1.0 + s.phi) * c
            stop.append((abs(a - b) / (abs(a) + abs(b)), max(s.depth, deepest)))
        if s.kept:
            deepest = max(deepest, s.depth)
    kept_min = {}
    for nd in ex.selected:
        kept_min[nd.depth] = min(kept_min.get(nd.depth, math.inf), nd.sigma)
    front_max = {}
    for nd in ex.frontier:
        front_max[nd.depth] = max(front_max.get(nd.depth, -math.inf), nd.sigma)
    cross = []
    for d, lo in kept_min.items():
        for d2, hi in front_max.items():
            if d2 != d:
                cross.append((lo - hi, abs(d - d2)))
    return Margins(stop, cross)
