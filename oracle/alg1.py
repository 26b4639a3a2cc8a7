"""Algorithm 1 (CaDDTree): best-first expansion with the greedy throughput stop.

Oracle; test infrastructure.  Follows Sec. 4.5 (Algorithm 1) in the paper's
order, in fp64:

* A node s = (s_1 .. s_d) of the draft tree is identified here by its 0-based
  rank tuple (rank k-1 stands for the paper's k-th most likely token).  Its
  log prefix probability (eq. prefix-prob) is
  sigma(s) = sum_{i<=d} log q_i^(s_i) = Lambda(s) - A_d with
  Lambda(s) = sum_{i<=d} l_i^(s_i) (raw logits) and A_d = sum_{i<=d} LSE_i,
  both summed in depth order.  The key is clamped, sigma(s) =
  min(Lambda(s) - A_d, sigma(parent)) with sigma(root) = 0, so a child never
  ranks above its parent under rounding (the parent-dominates-child fact used
  in the proof of Prop. 1).  The sibling key of Algorithm 1,
  sigma(s) - log q_d^(s_d) + log q_d^(s_d + 1), is the same quantity and is
  computed directly.
* The max-heap order is the canonical total order on nodes:
  sigma descending, then depth ascending, then Lambda descending, then the
  rank tuple lexicographically ascending.  The paper leaves ties open; this
  order makes every node's predecessor (previous sibling, or parent for a
  first child) come before it, so the heap pops the nodes in exactly this
  order.
* Stop rule (Algorithm 1, eq. stopping): with C(n) = C_d + C_v(n), the
  popped node is kept iff theta_new = (1 + Phi + delta) / C(n + 1) is strictly
  greater than theta_prev; ties stop.  1 + Phi + delta is formed left to
  right.  The loop also ends when the heap is empty or n reaches the budget
  cap (the cap is this library's addition; Algorithm 1 has none).
"""

from __future__ import annotations

import dataclasses
import heapq
import math
from typing import List, Optional, Tuple

import numpy as np


@dataclasses.dataclass
class Node:
    ranks: Tuple[int, ...]
    sigma: float
    lam: float

    @property
    def depth(self) -> int:
        return len(self.ranks)

    def key(self):
        return (-self.sigma, self.depth, -self.lam, self.ranks)


@dataclasses.dataclass
class Step:
    """One tested pop: the decision of Algorithm 1 at budget n."""
    n: int
    delta: float
    phi: float          # Phi before adding delta
    c_n: float          # C_d + C_v(n)
    c_next: float       # C_d + C_v(n + 1)
    theta_prev: float
    theta_new: float
    kept: bool


@dataclasses.dataclass
class Expansion:
    selected: List[Node]         # kept nodes, in pop order
    deltas: List[float]          # exp(sigma) of each kept node
    n_star: int
    phi: float
    theta: float                 # theta_prev at exit = theta_hat*(n_star)
    stop: str                    # "rule", "cap" or "exhausted"
    steps: List[Step]
    frontier: List[Node]         # unselected nodes whose predecessor was kept (incl. a rejected pop)


def _prefix_lse(lse: np.ndarray) -> np.ndarray:
    A = np.zeros(len(lse) + 1, dtype=np.float64)
    for d in range(1, len(lse) + 1):
        A[d] = A[d - 1] + float(lse[d - 1])
    return A


def expand(logit: np.ndarray, lse: np.ndarray, t_draft: float, t_verify: np.ndarray,
           cap: int, budget: Optional[int] = None) -> Expansion:
    """Run Algorithm 1 on one round.

    ``logit`` float64 [L, K]: raw top-K logits per position (value desc);
    ``lse`` float64 [L]; ``t_verify`` float64, at least cap + 1 entries.
    ``budget``: if given, run the fixed-budget heap instead (pop exactly
    min(budget, cap, #nodes) nodes, no stop rule) -- the DDTree construction
    of Sec. 3.4, used to obtain T*_n for every n.
    """
    logit = np.asarray(logit, dtype=np.float64)
    L, K = logit.shape
    A = _prefix_lse(np.asarray(lse, dtype=np.float64))
    t_verify = np.asarray(t_verify, dtype=np.float64)
    if len(t_verify) < cap + 1:
        raise ValueError("t_verify needs cap + 1 entries")
    if not t_draft > 0:
        raise ValueError("t_draft must be positive")

    def C(n: int) -> float:
        return t_draft + float(t_verify[n])

    def make(parent: Optional[Node], ranks: Tuple[int, ...]) -> Node:
        d = len(ranks)
        base_lam = 0.0 if parent is None else parent.lam
        base_sig = 0.0 if parent is None else parent.sigma
        lam = base_lam + float(logit[d - 1, ranks[-1]])
        sig = min(lam - float(A[d]), base_sig)
        return Node(ranks, sig, lam)

    parents = {(): None}
    selected: List[Node] = []
    deltas: List[float] = []
    steps: List[Step] = []
    phi, n = 0.0, 0
    theta_prev = 1.0 / C(0)
    heap = []
    first = make(None, (0,))
    heapq.heappush(heap, (first.key(), first))
    stop = "exhausted"
    rejected = None
    limit = cap if budget is None else min(cap, budget)
    while heap:
        if n >= limit:
            stop = "cap"
            break
        _, node = heapq.heappop(heap)
        delta = math.exp(node.sigma)
        theta_new = (1.0 + phi + delta) / C(n + 1)
        if budget is None:
            kept = not (theta_new <= theta_prev)
            steps.append(Step(n, delta, phi, C(n), C(n + 1), theta_prev, theta_new, kept))
            if not kept:
                stop = "rule"
                rejected = node
                break
        selected.append(node)
        deltas.append(delta)
        phi += delta
        n += 1
        theta_prev = theta_new
        parents[node.ranks] = node
        d, r = node.depth, node.ranks[-1]
        if r + 1 < K:
            sib = make(parents[node.ranks[:-1]], node.ranks[:-1] + (r + 1,))
            heapq.heappush(heap, (sib.key(), sib))
        if d < L:
            child = make(node, node.ranks + (0,))
            heapq.heappush(heap, (child.key(), child))
    frontier = [nd for _, nd in heap]
    if rejected is not None:
        frontier.append(rejected)
    if budget is not None:
        theta_prev = (1.0 + phi) / C(n)
    return Expansion(selected, deltas, n, phi, theta_prev, stop, steps, frontier)
