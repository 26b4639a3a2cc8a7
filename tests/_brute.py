"""Brute-force checkers that pin the oracle on tiny inputs.

Independent of ``oracle/``: probabilities are formed directly as products of
softmax values (no log-sum-exp, no heap), and trees are enumerated
exhaustively.
"""

from __future__ import annotations

import itertools
from typing import Dict, List, Tuple

import numpy as np


def softmax_direct(x: np.ndarray) -> np.ndarray:
    e = np.exp(np.asarray(x, dtype=np.float64))
    return e / e.sum(axis=-1, keepdims=True)


def topk_by_sort(x: np.ndarray, K: int) -> np.ndarray:
    """Top-K ids via Python's stable sort of (value desc) over ascending ids."""
    ids = sorted(range(len(x)), key=lambda v: -float(x[v]))  # stable: equal values keep id order
    return np.array(ids[:K], dtype=np.int64)


def all_nodes(q: np.ndarray, ids: np.ndarray) -> Dict[Tuple[int, ...], float]:
    """Every node of the K-ary, depth-L tree with its prefix probability pi."""
    L, K = ids.shape
    out = {}
    for d in range(1, L + 1):
        for ranks in itertools.product(range(K), repeat=d):
            p = 1.0
            for i, r in enumerate(ranks):
                p *= float(q[i, ids[i, r]])
            out[ranks] = p
    return out


def sorted_deltas(nodes: Dict[Tuple[int, ...], float]) -> List[float]:
    return sorted(nodes.values(), reverse=True)


def theta_curve(deltas: List[float], t_draft: float, t_verify: np.ndarray, cap: int) -> np.ndarray:
    """theta*(n) = (1 + Phi*(n)) / (C_d + C_v(n)) for n = 0 .. min(cap, #nodes)."""
    nmax = min(cap, len(deltas))
    phi = np.concatenate([[0.0], np.cumsum(deltas[:nmax])])
    return (1.0 + phi) / (t_draft + np.asarray(t_verify[: nmax + 1], dtype=np.float64))


def enumerate_trees(nodes: Dict[Tuple[int, ...], float], L: int, K: int):
    """All prefix-closed subtrees, as (size, Phi) pairs (the empty tree included)."""

    def forests(prefix: Tuple[int, ...]):
        # all ways to hang subtrees below `prefix`: each child absent or present with a forest
        d = len(prefix)
        if d == L:
            return [(0, 0.0)]
        per_child = []
        for r in range(K):
            child = prefix + (r,)
            opts = [(0, 0.0)]
            for n, phi in forests(child):
                opts.append((n + 1, phi + nodes[child]))
            per_child.append(opts)
        out = []
        for combo in itertools.product(*per_child):
            out.append((sum(c[0] for c in combo), sum(c[1] for c in combo)))
        return out

    return forests(())


def best_phi_by_size(trees) -> Dict[int, float]:
    best: Dict[int, float] = {}
    for n, phi in trees:
        if phi > best.get(n, -1.0):
            best[n] = phi
    return best
