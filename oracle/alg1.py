"""The throughput-optimal draft tree of one round, computed from its definition.

Oracle; test infrastructure.  fp64 throughout.

What the method returns (Sec. 4.3-4.5):

* A node s = (s_1 .. s_d) of the draft tree is identified by its 0-based rank
  tuple (rank k-1 stands for the paper's k-th most likely token at that
  position).  Its log prefix probability (eq. prefix-prob) is
  sigma(s) = sum_{i<=d} log q_i^(s_i) = Lambda(s) - A_d with
  Lambda(s) = sum_{i<=d} l_i^(s_i) (raw logits) and A_d = sum_{i<=d} LSE_i,
  both summed in depth order.  The value is clamped,
  sigma(s) = min(Lambda(s) - A_d, sigma(parent)), sigma(root) = 0, so a child
  never ranks above its parent under rounding (the parent-dominates-child fact
  in the proof of Prop. 1).
* Nodes are ranked by one total order: sigma descending, then depth ascending,
  then Lambda descending, then the rank tuple lexicographically ascending (the
  paper leaves ties open).
* T*_n is the first n nodes in that order: the n prefixes of largest path
  probability (eq. phistar), a tree that maximises Phi among trees of n nodes
  (Prop. 1).  Phi*(n) is the sum of their exp(sigma), added in that order.
* theta*(n) = (1 + Phi*(n)) / C(n) with C(n) = C_d + C_v(n) (eq. per-round).
  The chosen budget n* is the first n at which the next node does not raise
  theta (Lemma 1, eq. stopping: it is kept only if theta*(n + 1) > theta*(n));
  under a convex cost this is the first maximiser of theta* (Thm. 1, Cor. 2).
  theta*(n + 1) is formed as ((1 + Phi*(n)) + delta) / C(n + 1).  The budget
  also ends at the cap (this library's addition) and when no node is left.
* Fixed-budget mode (the DDTree construction, Sec. 3.4): n* = min(budget, cap,
  number of nodes), with no stop rule.

How the first nodes of the order are found without listing the whole tree:
for a level tau the set T(tau) = {s : sigma(s) >= tau} contains, with every
node, its parent and its previous siblings (sigma does not rise along either
step), so it is listed by descending from the root through children of rank
0, 1, .. while they pass.  Every node outside T(tau) has sigma < tau and so
comes after every node of T(tau): sorted, T(tau) is exactly the first |T(tau)|
nodes of the whole order.  tau is lowered one nat at a time until that prefix
holds the stop, reaches the cap, or is the whole tree.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

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
    """One stop test: is the next node worth adding at budget n?"""
    n: int
    depth: int          # depth of the node tested
    delta: float
    phi: float          # Phi*(n), before adding delta
    c_n: float          # C_d + C_v(n)
    c_next: float       # C_d + C_v(n + 1)
    theta_prev: float   # theta*(n)
    theta_new: float    # theta*(n + 1)
    kept: bool


@dataclasses.dataclass
class Expansion:
    selected: List[Node]         # T*_{n*}, in the order above
    deltas: List[float]          # exp(sigma) of each selected node
    n_star: int
    phi: float
    theta: float                 # theta*(n_star)
    stop: str                    # "rule", "cap" or "exhausted"
    steps: List[Step]
    frontier: List[Node]         # unselected nodes whose parent (or root) and previous sibling are selected


def _prefix_lse(lse: np.ndarray) -> np.ndarray:
    A = np.zeros(len(lse) + 1, dtype=np.float64)
    for d in range(1, len(lse) + 1):
        A[d] = A[d - 1] + float(lse[d - 1])
    return A


class _Tree:
    """The K-ary, depth-L tree of rank tuples with the log prefix probability of each node."""

    def __init__(self, logit: np.ndarray, lse: np.ndarray):
        self.logit = np.asarray(logit, dtype=np.float64)
        self.L, self.K = self.logit.shape
        self.A = _prefix_lse(np.asarray(lse, dtype=np.float64))
        self.total = sum(self.K ** d for d in range(1, self.L + 1))
        self._memo: Dict[Tuple[int, ...], Node] = {}

    def node(self, ranks: Tuple[int, ...]) -> Node:
        nd = self._memo.get(ranks)
        if nd is None:
            d = len(ranks)
            if d == 1:
                base_lam, base_sig = 0.0, 0.0
            else:
                parent = self.node(ranks[:-1])
                base_lam, base_sig = parent.lam, parent.sigma
            lam = base_lam + float(self.logit[d - 1, ranks[-1]])
            sig = min(lam - float(self.A[d]), base_sig)
            nd = self._memo[ranks] = Node(ranks, sig, lam)
        return nd

    def at_or_above(self, tau: float) -> List[Node]:
        """T(tau): every node with sigma >= tau."""
        out: List[Node] = []
        stack: List[Tuple[int, ...]] = [()]
        while stack:
            prefix = stack.pop()
            if len(prefix) == self.L:
                continue
            for r in range(self.K):
                child = self.node(prefix + (r,))
                if child.sigma < tau:
                    break               # later ranks have no larger sigma
                out.append(child)
                stack.append(child.ranks)
        return out


def expand(logit: np.ndarray, lse: np.ndarray, t_draft: float, t_verify: np.ndarray,
           cap: int, budget: Optional[int] = None) -> Expansion:
    """T*_{n*} of one round.

    ``logit`` float64 [L, K]: raw top-K logits per position (value desc);
    ``lse`` float64 [L]; ``t_verify`` float64, at least cap + 1 entries.
    ``budget``: if given, return T*_n at n = min(budget, cap, #nodes) with no
    stop rule (the fixed-budget construction).
    """
    t_verify = np.asarray(t_verify, dtype=np.float64)
    if len(t_verify) < cap + 1:
        raise ValueError("t_verify needs cap + 1 entries")
    if not t_draft > 0:
        raise ValueError("t_draft must be positive")
    tree = _Tree(logit, lse)
    limit = cap if budget is None else min(cap, budget)

    def C(n: int) -> float:
        return t_draft + float(t_verify[n])

    tau = tree.node((0,)).sigma
    while True:
        tau -= 1.0
        listed = tree.at_or_above(tau)
        complete = len(listed) == tree.total
        order = sorted(listed, key=Node.key)   # the first len(listed) nodes of the whole order
        selected: List[Node] = []
        deltas: List[float] = []
        steps: List[Step] = []
        phi, n = 0.0, 0
        theta_prev = 1.0 / C(0)
        stop = None
        for nd in order:
            if n >= limit:
                stop = "cap"
                break
            delta = math.exp(nd.sigma)
            theta_new = (1.0 + phi + delta) / C(n + 1)
            if budget is None:
                kept = not (theta_new <= theta_prev)
                steps.append(Step(n, nd.depth, delta, phi, C(n), C(n + 1), theta_prev, theta_new, kept))
                if not kept:
                    stop = "rule"
                    break
            selected.append(nd)
            deltas.append(delta)
            phi += delta
            n += 1
            theta_prev = theta_new
        if stop is None:
            if complete:
                stop = "exhausted"          # no node is left
            elif n >= limit:
                stop = "cap"                # nodes outside the listed set remain
        if stop is not None:
            break
    if budget is not None:
        theta_prev = (1.0 + phi) / C(n)
    return Expansion(selected, deltas, n, phi, theta_prev, stop, steps, _frontier(tree, selected))


def _frontier(tree: _Tree, selected: List[Node]) -> List[Node]:
    """Unselected nodes that would come next along some branch: the first depth-1 node, the next
    sibling and the first child of every selected node, when they exist and are not selected."""
    kept = {nd.ranks for nd in selected}
    cand = [(0,)]
    for nd in selected:
        r = nd.ranks[-1]
        if r + 1 < tree.K:
            cand.append(nd.ranks[:-1] + (r + 1,))
        if nd.depth < tree.L:
            cand.append(nd.ranks + (0,))
    out, seen = [], set()
    for rk in cand:
        if rk not in kept and rk not in seen:
            seen.add(rk)
            out.append(tree.node(rk))
    return out
