"""The library's cost fitter (caddtree_fit_cost, host code) against the oracle's, and its own
optimality certificate; runs without a GPU."""

import numpy as np
import pytest

from oracle import costfit as ofit
from paper_2606_01813_amd import CaddtreeError, _lib, fit_cost
from tests.test_oracle_costfit import check_kkt

CASES = [
    # name, x, y
    ("quad+noise", np.arange(1.0, 257.0), lambda x, r: 1 + 0.004 * x + 3e-5 * x * x + r.normal(0, 0.05, len(x))),
    ("heavy noise", np.arange(1.0, 101.0), lambda x, r: 1 + 0.01 * x + r.normal(0, 1.0, len(x))),
    ("flat then steep", np.arange(1.0, 129.0), lambda x, r: np.where(x < 64, 1.0, 1 + 0.02 * (x - 64))
     + r.normal(0, 0.01, len(x))),
    ("decreasing", np.arange(1.0, 51.0), lambda x, r: 5 - 0.1 * x + r.normal(0, 0.01, len(x))),
    ("concave", np.arange(1.0, 81.0), lambda x, r: np.sqrt(x) + r.normal(0, 0.01, len(x))),
    ("non-uniform grid", np.cumsum(np.linspace(0.5, 9.0, 70)), lambda x, r: 2 + 1e-3 * x ** 1.5
     + r.normal(0, 0.02, len(x))),
    ("profile grid 1..1024", np.arange(1.0, 1025.0), lambda x, r: 12 + 0.01 * x + 1.5e-5 * x * x
     + r.normal(0, 0.3, len(x))),
    ("tiny", np.array([1.0, 2.0, 3.0]), lambda x, r: np.array([3.0, 1.0, 2.0])),
]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_fit_matches_oracle_and_is_optimal(i):
    name, x, gen = CASES[i]
    y = gen(x, np.random.default_rng(100 + i))
    f = fit_cost(x, y)
    g = ofit.fit_convex(x, y)
    scale = max(1.0, float(np.max(np.abs(y))))
    assert np.max(np.abs(f - g)) <= 1e-8 * scale, (name, np.max(np.abs(f - g)))
    check_kkt(x, y, f)


def test_cost_table_matches_oracle_and_builds_a_plan():
    x = np.arange(1.0, 513.0)
    y = 1 + 0.002 * x + 2e-5 * x * x + np.random.default_rng(5).normal(0, 0.02, len(x))
    f, table = fit_cost(x, y, cap=600)
    np.testing.assert_allclose(table, ofit.cost_table(x, f, 600), rtol=1e-13, atol=1e-13)
    d1, d2 = np.diff(table), np.diff(table, 2)
    assert d1.min() >= -1e-12 * table.max() and d2.min() >= -1e-12 * table.max()
    # the table is acceptable as a plan's verification cost (validation runs before any HIP call)
    import ctypes
    cfg = _lib.Config(16, 151936, 8, 600, 1, 1, 0, 1.0, table.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                      0, None)
    h = ctypes.c_void_p()
    st = _lib.lib().caddtree_plan_create(ctypes.byref(cfg), ctypes.byref(h))
    assert st in (_lib.OK, _lib.E_HIP), _lib.lib().caddtree_last_error()
    if st == _lib.OK:
        _lib.lib().caddtree_plan_destroy(h)


def test_edge_sizes():
    assert fit_cost([4.0], [2.5]).tolist() == [2.5]
    np.testing.assert_allclose(fit_cost([1.0, 2.0], [3.0, 1.0]), [2.0, 2.0])
    f, t = fit_cost([7.0], [1.5], cap=3)
    assert t.tolist() == [1.5] * 4


@pytest.mark.parametrize("x,y", [
    ([1.0, 1.0], [1.0, 2.0]),
    ([2.0, 1.0], [1.0, 2.0]),
    ([1.0, np.nan], [1.0, 2.0]),
    ([1.0, 2.0], [1.0, np.inf]),
    ([], []),
])
def test_invalid_profiles(x, y):
    with pytest.raises(CaddtreeError):
        fit_cost(x, y)


def test_invalid_cap():
    with pytest.raises(CaddtreeError):
        fit_cost([1.0, 2.0], [1.0, 2.0], cap=5000)
