"""Draft-tree output: canonical order, parents, mask, position ids (oracle; test infrastructure).

The paper returns the tree as a node set (Algorithm 1) and verifies it with tree
attention, where each node attends to the shared context and to its own
ancestors (Sec. 3.3).  This module fixes the output layout:

* order: depth ascending, then rank tuple lexicographically ascending (a
  breadth-first order; every parent precedes its children);
* parent[i]: index of node i's parent in that order, -1 for depth-1 nodes
  (whose parent is the bonus token, the root, which is not a node);
* mask[i][j] = 1 iff node j is node i or one of its ancestors, over the
  n x n block of non-root nodes; attention to the root and the context is
  implicit;
* pos[i] = pos_offset + depth(i), so the root sits at pos_offset.

Packed masks use u32 words, bit (j mod 32) of word (j div 32), least
significant bit first, ceil(cap / 32) words per row.
"""

from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np


@dataclasses.dataclass
class TreeOut:
    ranks: List[Tuple[int, ...]]   # canonical order
    token_ids: np.ndarray          # int64 [n]
    parent: np.ndarray             # int64 [n]
    depth: np.ndarray              # int64 [n]
    path_prob: np.ndarray          # float64 [n], exp(sigma)
    pos_ids: np.ndarray            # int64 [n]


def canonical_order(ranks: Sequence[Tuple[int, ...]], deltas: Sequence[float],
                    topk_ids: np.ndarray, pos_offset: int = 0) -> TreeOut:
    """Lay out a prefix-closed node set (rank tuples) in canonical order."""
    order = sorted(range(len(ranks)), key=lambda i: (len(ranks[i]), ranks[i]))
    rk = [tuple(ranks[i]) for i in order]
    index = {r: i for i, r in enumerate(rk)}
    n = len(rk)
    tok = np.empty(n, dtype=np.int64)
    par = np.empty(n, dtype=np.int64)
    dep = np.empty(n, dtype=np.int64)
    for i, r in enumerate(rk):
        d = len(r)
        dep[i] = d
        tok[i] = int(topk_ids[d - 1, r[-1]])
        if d == 1:
            par[i] = -1
        else:
            if r[:-1] not in index:
                raise ValueError("node set is not prefix-closed")
            par[i] = index[r[:-1]]
    prob = np.array([deltas[i] for i in order], dtype=np.float64)
    return TreeOut(rk, tok, par, dep, prob, pos_offset + dep)


def emit_mask(parent: np.ndarray, kind: str = "u8", cap: int | None = None) -> np.ndarray:
    """Ancestor-or-self mask of a tree in canonical order.

    kind "u8": uint8 [n, n].  kind "bits": uint32 [n, ceil(cap/32)] with only
    the first ceil(n/32) words of each row meaningful (the rest zero here).
    """
    parent = np.asarray(parent, dtype=np.int64)
    n = len(parent)
    dense = np.zeros((n, n), dtype=np.uint8)
    for i in range(n):
        j = i
        while j >= 0:
            dense[i, j] = 1
            j = int(parent[j])
    if kind == "u8":
        return dense
    if kind == "bits":
        cap = n if cap is None else cap
        words = (cap + 31) // 32
        out = np.zeros((n, words), dtype=np.uint32)
        for j in range(n):          # column j sets bit j % 32 of word j // 32 in every row
            out[:, j // 32] |= dense[:, j].astype(np.uint32) << np.uint32(j % 32)
        return out
    raise ValueError(kind)
