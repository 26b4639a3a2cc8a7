"""Context-aware verification cost (oracle; test infrastructure).

The verification cost depends on the current context length l as well as on
the node count n (Sec. 4.2).  It is profiled offline on a grid of context
lengths L_0 < L_1 < ... < L_{J-1}, one table C_v(.; L_j) per grid point
(Sec. 4.6).  At run time l is known exactly, and for L_j <= l < L_{j+1} the
cost is the linear interpolation of eq. cv-interp:

    alpha = (l - L_j) / (L_{j+1} - L_j)
    C_v(n; l) = (1 - alpha) * C_v(n; L_j) + alpha * C_v(n; L_{j+1})

Readings (the paper defines only the interior case):

* l below L_0 takes the L_0 table, and l at or above L_{J-1} takes the
  L_{J-1} table.  Linear extrapolation is not used, because weights outside
  [0, 1] could break the convexity and monotonicity that Cor. 3 needs.
* alpha is the correctly rounded quotient of the two integer differences.
  Each product and the sum are rounded separately, with no fused multiply-add.
"""

from __future__ import annotations

import numpy as np


def context_cost(tables: np.ndarray, grid, ell: int) -> np.ndarray:
    """C_v(0..cap; ell) from J tables [J, cap + 1] on the integer grid ``grid`` (eq. cv-interp)."""
    tables = np.asarray(tables, dtype=np.float64)
    grid = [int(g) for g in grid]
    if tables.ndim != 2 or tables.shape[0] != len(grid) or len(grid) == 0:
        raise ValueError("need one table per grid point")
    if any(b <= a for a, b in zip(grid, grid[1:])):
        raise ValueError("grid must be strictly increasing")
    ell = int(ell)
    if ell <= grid[0]:
        return tables[0].copy()
    if ell >= grid[-1]:
        return tables[-1].copy()
    j = 0
    while grid[j + 1] <= ell:
        j += 1
    alpha = (ell - grid[j]) / (grid[j + 1] - grid[j])   # Python int division: correctly rounded
    lo, hi = tables[j], tables[j + 1]
    return np.array([(1.0 - alpha) * float(lo[n]) + alpha * float(hi[n]) for n in range(tables.shape[1])],
                    dtype=np.float64)
