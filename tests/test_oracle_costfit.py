"""Pins for the oracle's convex non-decreasing cost regression (Sec. 4.6, eq. convex-reg).

* KKT certificate: the fit is feasible, and its residual is a non-negative
  combination of the active constraints' normals (stationarity, dual
  feasibility, complementary slackness), which proves optimality of the
  convex program whatever routine produced it;
* brute force on tiny grids: every choice of active constraints, the
  equality-constrained least-squares fit, the best feasible one;
* closed forms: convex non-decreasing data is its own fit, decreasing data
  fits to its mean;
* the cost table built from a fit is convex and non-decreasing and passes
  through the fitted points;
* planted mistakes must fail one of these pins.
"""

import itertools

import numpy as np
import pytest

from oracle import costfit as ofit
from tests.test_oracle_pins import _plant


def constraint_matrix(x):
    """G [N-1, N]: row 0 = first slope, row j = slope_{j+1} - slope_j; the fit needs G f >= 0."""
    x = np.asarray(x, dtype=np.float64)
    N = len(x)
    S = np.zeros((N - 1, N))                 # slopes
    for j in range(N - 1):
        h = x[j + 1] - x[j]
        S[j, j], S[j, j + 1] = -1.0 / h, 1.0 / h
    G = np.zeros((N - 1, N))
    G[0] = S[0]
    for j in range(1, N - 1):
        G[j] = S[j] - S[j - 1]
    return G


def check_kkt(x, y, f, tol=1e-7):
    x, y, f = (np.asarray(v, dtype=np.float64) for v in (x, y, f))
    scale = max(1.0, float(np.max(np.abs(y))))
    G = constraint_matrix(x)
    g = G @ f
    gscale = scale / max(float(np.min(np.diff(x))), 1e-300)
    assert np.all(g >= -tol * gscale), ("infeasible", g.min())
    lam, *_ = np.linalg.lstsq(G.T, f - y, rcond=None)
    assert np.max(np.abs(G.T @ lam - (f - y))) <= tol * scale, "stationarity"
    lscale = scale * float(x[-1] - x[0]) + 1.0
    assert np.all(lam >= -tol * lscale), ("dual infeasible", lam.min())
    assert np.max(np.abs(lam * g)) <= tol * lscale * gscale, "complementary slackness"


def brute_force(x, y):
    G = constraint_matrix(x)
    best, best_obj = None, np.inf
    m = G.shape[0]
    for r in range(m + 1):
        for S in itertools.combinations(range(m), r):
            if S:
                Gs = G[list(S)]
                # projection of y onto the null space of Gs
                P = np.eye(len(x)) - Gs.T @ np.linalg.solve(Gs @ Gs.T, Gs)
                f = P @ y
            else:
                f = np.asarray(y, dtype=np.float64).copy()
            if np.all(G @ f >= -1e-9):
                obj = float(np.sum((f - y) ** 2))
                if obj < best_obj - 1e-12:
                    best, best_obj = f, obj
    return best


def check_fit_random(seed=0, N=60):
    rng = np.random.default_rng(seed)
    x = np.cumsum(rng.uniform(0.5, 2.0, size=N))
    y = 1.0 + 0.002 * x + 1e-4 * x * x + rng.normal(0, 0.05, size=N)
    f = ofit.fit_convex(x, y)
    check_kkt(x, y, f)


def check_brute_force(seed=1, N=5):
    rng = np.random.default_rng(seed)
    x = np.sort(rng.choice(np.arange(1, 30), size=N, replace=False)).astype(np.float64)
    y = rng.normal(0, 1, size=N)
    f = ofit.fit_convex(x, y)
    np.testing.assert_allclose(f, brute_force(x, y), atol=1e-9)


def check_closed_forms():
    x = np.arange(1.0, 41.0)
    y = 2.0 + 0.1 * x + 0.003 * x * x
    np.testing.assert_allclose(ofit.fit_convex(x, y), y, atol=1e-9)
    yd = 5.0 - 0.3 * x
    np.testing.assert_allclose(ofit.fit_convex(x, yd), np.full_like(x, yd.mean()), atol=1e-9)


def check_table():
    x = np.array([1.0, 2.0, 4.0, 8.0, 16.0])
    f = ofit.fit_convex(x, np.array([1.0, 1.1, 1.5, 2.0, 4.0]))
    t = ofit.cost_table(x, f, 20)
    assert np.allclose(t[[1, 2, 4, 8, 16]], f)
    assert np.all(np.diff(t) >= -1e-12) and np.all(np.diff(t, 2) >= -1e-12)
    # the end segments continue: beyond x_N the last slope, before x_1 the first
    assert abs((t[20] - t[16]) / 4 - (f[-1] - f[-2]) / (x[-1] - x[-2])) < 1e-12
    assert abs((t[1] - t[0]) - (f[1] - f[0]) / (x[1] - x[0])) < 1e-12


@pytest.mark.parametrize("seed", range(4))
def test_kkt_certificate(seed):
    check_fit_random(seed)


def test_kkt_certificate_large():
    rng = np.random.default_rng(9)
    x = np.arange(1.0, 1025.0)
    y = 10 + 0.01 * x + 2e-5 * x * x + rng.normal(0, 0.5, size=len(x))
    check_kkt(x, y, ofit.fit_convex(x, y))


@pytest.mark.parametrize("seed,N", [(1, 3), (2, 4), (3, 5), (4, 6), (5, 6), (6, 7)])
def test_brute_force(seed, N):
    check_brute_force(seed, N)


def test_closed_forms():
    check_closed_forms()


def test_table():
    check_table()


def test_edge_sizes():
    assert ofit.fit_convex([3.0], [7.0]).tolist() == [7.0]
    np.testing.assert_allclose(ofit.fit_convex([1.0, 2.0], [3.0, 1.0]), [2.0, 2.0])
    np.testing.assert_allclose(ofit.fit_convex([1.0, 2.0], [1.0, 3.0]), [1.0, 3.0])
    with pytest.raises(ValueError):
        ofit.fit_convex([1.0, 1.0], [1.0, 2.0])


MUTATIONS = [
    ("oracle.costfit", "cols = [x - x[0]] + ", "cols = [x[0] - x] + ", check_fit_random, ()),
    ("oracle.costfit", "c = float(np.mean(y - A @ b))", "c = 0.0", check_closed_forms, ()),
    ("oracle.costfit", "[np.maximum(0.0, x - x[k]) for k in range(1, N - 1)]",
     "[np.maximum(0.0, x - x[k]) for k in range(2, N - 1)]", check_brute_force, ()),
    ("oracle.costfit", "out[hi] = f[-1] + (n[hi] - x[-1]) * (f[-1] - f[-2]) / (x[-1] - x[-2])",
     "out[hi] = f[-1] + (n[hi] - x[-1]) * (f[1] - f[0]) / (x[1] - x[0])", check_table, ()),
]


@pytest.mark.parametrize("i", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(monkeypatch, i):
    modname, old, new, check, args = MUTATIONS[i]
    check(*args)
    _plant(monkeypatch, modname, old, new)
    with pytest.raises(Exception):
        check(*args)
