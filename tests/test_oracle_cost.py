"""Pins for the oracle's context-aware cost (Sec. 4.6, eq. cv-interp).

* a hand-worked round under two context tables (tests/golden/hand_example_ctx.json);
* closed form: tables affine in the context length interpolate to the affine
  value at any context length;
* grid points reproduce their table bit for bit, and contexts outside the grid
  take the nearest end table;
* the paper's claim that interpolation keeps C_v convex and non-decreasing in n;
* planted mistakes in the interpolation must fail one of these pins.
"""

import json
import os

import numpy as np
import pytest

import oracle
from oracle import cost as ocost
from tests.test_oracle_pins import _plant

HERE = os.path.dirname(os.path.abspath(__file__))


def _hand_ctx():
    with open(os.path.join(HERE, "golden", "hand_example_ctx.json")) as f:
        return json.load(f)


def _tables_linear(slopes, cap):
    n = np.arange(cap + 1, dtype=np.float64)
    return np.stack([1.0 + s * n for s in slopes])


def check_hand_ctx():
    g = _hand_ctx()
    logits = np.log(np.array(g["q"], dtype=np.float64)).astype(np.float32)
    tables = _tables_linear(g["slopes"], g["cap"])
    for case in g["cases"]:
        tv = oracle.context_cost(tables, g["grid"], case["ell"])
        r = oracle.build_round(logits, "f32", g["K"], g["t_draft"], tv, g["cap"])
        assert r.n_star == case["n_star"], (case["ell"], r.n_star)
        assert r.tree.token_ids.tolist() == case["token_ids"]
        assert r.tree.parent.tolist() == case["parent"]
        assert abs(r.exp.phi - case["phi"]) < 1e-6
        assert abs(r.exp.theta - case["theta"]) < 1e-6 * case["theta"]


def check_affine_closed_form(seed=0):
    """C_v(n; L_j) = a(n) + L_j b(n) for every j  =>  C_v(n; l) = a(n) + l b(n) for every l in the grid's span."""
    rng = np.random.default_rng(seed)
    cap = 40
    n = np.arange(cap + 1, dtype=np.float64)
    a = 1.0 + 0.01 * n + 1e-4 * n * n
    bcoef = 1e-4 + 1e-6 * n
    grid = [0, 700, 1000, 2500, 4096, 8000]
    tables = np.stack([a + g * bcoef for g in grid])
    for ell in list(rng.integers(0, 8000, size=40)) + [1, 699, 701, 4095, 7999]:
        want = a + float(ell) * bcoef
        got = ocost.context_cost(tables, grid, int(ell))
        np.testing.assert_allclose(got, want, rtol=1e-13, atol=0)


def check_grid_points_and_clamp():
    cap = 16
    rng = np.random.default_rng(3)
    grid = [100, 1000, 3000]
    tables = np.sort(rng.uniform(1, 2, size=(3, cap + 1)), axis=1)
    for j, g in enumerate(grid):
        assert np.array_equal(ocost.context_cost(tables, grid, g), tables[j])
    assert np.array_equal(ocost.context_cost(tables, grid, -5), tables[0])
    assert np.array_equal(ocost.context_cost(tables, grid, 50), tables[0])
    assert np.array_equal(ocost.context_cost(tables, grid, 10 ** 9), tables[-1])
    # just above a grid point stays close to that point's table
    near = ocost.context_cost(tables, grid, 1001)
    assert np.max(np.abs(near - tables[1])) <= np.max(np.abs(tables[2] - tables[1])) / 1000


def test_hand_ctx():
    check_hand_ctx()


def test_affine_closed_form():
    check_affine_closed_form()


def test_grid_points_and_clamp():
    check_grid_points_and_clamp()


def test_single_table_ignores_context():
    t = 1.0 + 0.01 * np.arange(9)
    for ell in (-1, 0, 5, 10 ** 6):
        assert np.array_equal(ocost.context_cost(t[None, :], [0], ell), t)


@pytest.mark.parametrize("seed", range(5))
def test_interpolation_keeps_convex_nondecreasing(seed):
    """Convex combinations of convex non-decreasing tables stay convex and non-decreasing (Sec. 4.6)."""
    rng = np.random.default_rng(100 + seed)
    cap, J = 64, 5
    n = np.arange(cap + 1, dtype=np.float64)
    tables = []
    for _ in range(J):
        slopes = np.sort(rng.uniform(0, 0.05, size=cap))
        tables.append(rng.uniform(0.5, 2) + np.concatenate([[0.0], np.cumsum(slopes)]))
    tables = np.stack(tables)
    grid = sorted(rng.choice(10000, size=J, replace=False).tolist())
    for ell in rng.integers(grid[0], grid[-1], size=20):
        c = ocost.context_cost(tables, grid, int(ell))
        scale = np.max(np.abs(c))
        assert np.all(np.diff(c) >= -1e-13 * scale)
        assert np.all(np.diff(c, 2) >= -1e-13 * scale)
    assert n.shape[0] == cap + 1


def test_rejects_bad_grid():
    t = np.ones((2, 5))
    with pytest.raises(ValueError):
        ocost.context_cost(t, [5, 5], 3)
    with pytest.raises(ValueError):
        ocost.context_cost(t, [0], 3)


MUTATIONS = [
    ("oracle.cost", "(1.0 - alpha) * float(lo[n]) + alpha * float(hi[n])",
     "alpha * float(lo[n]) + (1.0 - alpha) * float(hi[n])", check_affine_closed_form, ()),
    ("oracle.cost", "lo, hi = tables[j], tables[j + 1]", "lo, hi = tables[j - 1], tables[j]",
     check_affine_closed_form, ()),
    ("oracle.cost", "if ell <= grid[0]:", "if ell <= grid[1]:", check_grid_points_and_clamp, ()),
    ("oracle.cost", "alpha = (ell - grid[j]) / (grid[j + 1] - grid[j])",
     "alpha = (ell - grid[j]) / (grid[-1] - grid[0])", check_affine_closed_form, ()),
    ("oracle.cost", "return tables[-1].copy()", "return tables[-2].copy()", check_hand_ctx, ()),
]


@pytest.mark.parametrize("i", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(monkeypatch, i):
    modname, old, new, check, args = MUTATIONS[i]
    check(*args)
    _plant(monkeypatch, modname, old, new)
    with pytest.raises(Exception):
        check(*args)
