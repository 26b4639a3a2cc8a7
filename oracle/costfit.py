"""Convex non-decreasing regression of a verification-cost profile (oracle; test infrastructure).

Sec. 4.6 fits, per context length, the least-squares function over the
profiled node counts that is convex and non-decreasing (eq. convex-reg), a
convex quadratic program whose solution is piecewise linear with breakpoints
chosen by the data.  On a strictly increasing grid x_1 < .. < x_N such
functions are exactly

    f(x) = c + b_0 (x - x_1) + sum_{k=2}^{N-1} b_k max(0, x - x_k),  b >= 0,

(b_0 is the first slope, b_k the slope increase at x_k; c is free), so the
program is a non-negative least-squares problem in b once c is eliminated by
centring the columns and the data.  ``fit_convex`` solves it with a library
NNLS routine on the dense hinge design.  ``cost_table`` evaluates the fitted
piecewise-linear function at n = 0 .. cap: linear interpolation between the
fitted points, and beyond either end the end segment continued (which keeps
it convex and non-decreasing).
"""

from __future__ import annotations

import numpy as np
from scipy.optimize import nnls


def hinge_design(x: np.ndarray) -> np.ndarray:
    """[N, N - 1]: the column (x - x_1), then max(0, x - x_k) for k = 2 .. N - 1."""
    x = np.asarray(x, dtype=np.float64)
    N = len(x)
    cols = [x - x[0]] + [np.maximum(0.0, x - x[k]) for k in range(1, N - 1)]
    return np.stack(cols, axis=1) if cols else np.zeros((N, 0))


def fit_convex(x, y) -> np.ndarray:
    """Least-squares fit of y at the points x by a convex non-decreasing function (eq. convex-reg)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    if x.ndim != 1 or x.shape != y.shape or len(x) == 0:
        raise ValueError("x and y must be 1-d of equal, non-zero length")
    if not (np.all(np.isfinite(x)) and np.all(np.isfinite(y))):
        raise ValueError("x and y must be finite")
    if np.any(np.diff(x) <= 0):
        raise ValueError("x must be strictly increasing")
    if len(x) == 1:
        return y.copy()
    A = hinge_design(x)
    Ac = A - A.mean(axis=0)
    yc = y - y.mean()
    b, _ = nnls(Ac, yc, maxiter=50 * A.shape[1])
    c = float(np.mean(y - A @ b))
    return c + A @ b


def cost_table(x, f, cap: int) -> np.ndarray:
    """The piecewise-linear function through (x_j, f_j), at n = 0 .. cap, end segments continued."""
    x = np.asarray(x, dtype=np.float64)
    f = np.asarray(f, dtype=np.float64)
    n = np.arange(cap + 1, dtype=np.float64)
    if len(x) == 1:
        return np.full(cap + 1, f[0])
    out = np.interp(n, x, f)
    lo, hi = n < x[0], n > x[-1]
    out[lo] = f[0] + (n[lo] - x[0]) * (f[1] - f[0]) / (x[1] - x[0])
    out[hi] = f[-1] + (n[hi] - x[-1]) * (f[-1] - f[-2]) / (x[-1] - x[-2])
    return out
