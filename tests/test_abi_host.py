"""The C ABI without a GPU: the library loads, exports what include/caddtree.h declares,
and validates plans on the host before any HIP call."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_01813_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "caddtree.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(caddtree_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return _lib.lib()


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert len(names) >= 9
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(names) == sorted(_lib.EXPORTS)


def test_status_strings(lib):
    for st in range(6):
        assert lib.caddtree_status_string(st)
    assert lib.caddtree_status_string(99) == b"unknown status"


def _cfg(**kw):
    d = dict(L=4, V=1024, K=4, budget_cap=32, dtype=0, mask=1, flags=0, t_draft=1.0, n_ctx=0)
    tv = kw.pop("tv", None)
    grid = kw.pop("grid", None)
    d.update(kw)
    cap = d["budget_cap"]
    if tv is None:
        n = np.arange(max(cap, 0) + 1, dtype=np.float64)
        tv = 1.0 + 0.01 * n + 0.0005 * n * n
        if d["n_ctx"] >= 2:
            tv = np.stack([tv * (1 + 0.1 * j) for j in range(d["n_ctx"])])
    tv = np.ascontiguousarray(tv, dtype=np.float64)
    gp = None
    if grid is not None:
        grid = np.ascontiguousarray(grid, dtype=np.int64)
        gp = grid.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    cfg = _lib.Config(d["L"], d["V"], d["K"], d["budget_cap"], d["dtype"], d["mask"], d["flags"], d["t_draft"],
                      tv.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), d["n_ctx"], gp)
    return cfg, (tv, grid)


def _create(lib, cfg):
    h = ctypes.c_void_p()
    st = lib.caddtree_plan_create(ctypes.byref(cfg), ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("kw,status", [
    (dict(L=0), _lib.E_INVALID),
    (dict(L=33), _lib.E_UNSUPPORTED),
    (dict(K=0), _lib.E_INVALID),
    (dict(K=17), _lib.E_UNSUPPORTED),
    (dict(V=3, K=4), _lib.E_INVALID),
    (dict(V=2 ** 31), _lib.E_UNSUPPORTED),
    (dict(budget_cap=-1, tv=np.ones(1)), _lib.E_INVALID),
    (dict(budget_cap=4097), _lib.E_UNSUPPORTED),
    (dict(dtype=7), _lib.E_INVALID),
    (dict(mask=9), _lib.E_INVALID),
    (dict(flags=4), _lib.E_INVALID),
    (dict(t_draft=0.0), _lib.E_COST),
    (dict(t_draft=-1.0), _lib.E_COST),
    (dict(t_draft=float("nan")), _lib.E_COST),
    (dict(budget_cap=3, tv=np.array([1.0, 2.0, 1.5, 3.0])), _lib.E_COST),          # decreasing
    (dict(budget_cap=3, tv=np.array([1.0, 3.0, 4.0, 4.5])), _lib.E_COST),          # concave
    (dict(budget_cap=2, tv=np.array([1.0, np.inf, 5.0])), _lib.E_COST),
    (dict(budget_cap=2, tv=np.array([-2.0, -1.5, -1.0])), _lib.E_COST),            # C_d + C_v <= 0
    # context-length grid (Sec. 4.6)
    (dict(n_ctx=-1), _lib.E_INVALID),
    (dict(n_ctx=65), _lib.E_UNSUPPORTED),
    (dict(n_ctx=2), _lib.E_INVALID),                                               # grid missing
    (dict(n_ctx=3, grid=[0, 1000, 1000]), _lib.E_INVALID),                         # not increasing
    (dict(n_ctx=2, grid=[-1, 1000]), _lib.E_INVALID),
    (dict(n_ctx=2, grid=[0, 2 ** 53 + 1]), _lib.E_INVALID),
    (dict(n_ctx=2, grid=[0, 10], budget_cap=3,
          tv=np.array([[1.0, 1.1, 1.2, 1.3], [1.0, 3.0, 4.0, 4.5]])), _lib.E_COST),   # second table concave
    (dict(n_ctx=2, grid=[0, 10], budget_cap=3,
          tv=np.array([[1.0, 1.1, 1.2, 1.3], [1.0, 0.9, 1.0, 1.1]])), _lib.E_COST),   # second table decreasing
])
def test_plan_validation_before_any_hip_call(lib, kw, status):
    cfg, _tv = _cfg(**kw)
    st, h = _create(lib, cfg)
    assert st == status, (st, lib.caddtree_last_error())
    assert not h.value
    assert lib.caddtree_last_error()


def test_null_arguments(lib):
    cfg, _tv = _cfg()
    assert lib.caddtree_plan_create(ctypes.byref(cfg), None) == _lib.E_INVALID
    h = ctypes.c_void_p()
    assert lib.caddtree_plan_create(None, ctypes.byref(h)) == _lib.E_INVALID
    cfg2 = _lib.Config(4, 1024, 4, 32, 0, 1, 0, 1.0, None, 0, None)
    assert lib.caddtree_plan_create(ctypes.byref(cfg2), ctypes.byref(h)) == _lib.E_INVALID
    assert lib.caddtree_build(None, None, 1, 1024, 0, None, None, None, 0, None) == _lib.E_INVALID
    assert lib.caddtree_reduce_topk(None, None, 1, 1024, None, None, None, None, None) == _lib.E_INVALID
    assert lib.caddtree_expand(None, None, None, None, 1, None, None, None, None, None, None, None, None,
                               None) == _lib.E_INVALID
    assert lib.caddtree_emit(None, None, None, None, 1, 0, None, None, None) == _lib.E_INVALID
    assert lib.caddtree_accept(None, None, None, None, 1, None, None, 8, None, None, None, None, None,
                               None) == _lib.E_INVALID
    assert lib.caddtree_workspace_bytes(None, 10) == 0
    lib.caddtree_plan_destroy(None)


def test_nonconvex_flag_accepts_nondecreasing(lib):
    cfg, _tv = _cfg(budget_cap=3, tv=np.array([1.0, 3.0, 4.0, 4.5]), flags=_lib.ALLOW_NONCONVEX)
    st, h = _create(lib, cfg)
    # validation passes; without a GPU the device query is what fails
    assert st in (_lib.OK, _lib.E_HIP)
    if st == _lib.OK:
        lib.caddtree_plan_destroy(h)


@pytest.mark.parametrize("kw", [
    dict(flags=_lib.FIXED_BUDGET),
    dict(flags=_lib.FIXED_BUDGET | _lib.ALLOW_NONCONVEX),
    dict(n_ctx=9, grid=[1000 * j for j in range(9)]),
    dict(n_ctx=1, grid=None),
])
def test_valid_plans_pass_validation(lib, kw):
    cfg, _keep = _cfg(**kw)
    st, h = _create(lib, cfg)
    # validation passes; without a GPU the device query is what fails
    assert st in (_lib.OK, _lib.E_HIP), lib.caddtree_last_error()
    if st == _lib.OK:
        lib.caddtree_plan_destroy(h)


def test_convexity_slack_accepts_rounding():
    # piecewise-linear table whose differences wobble at the 1e-16 level
    import synth
    tv = synth.cost_table("c3", 1024)
    d2 = np.diff(tv, 2)
    assert d2.min() < 0 and d2.min() > -1e-12
    cfg, _ = _cfg(budget_cap=1024, tv=tv)
    st, h = _create(_lib.lib(), cfg)
    assert st in (_lib.OK, _lib.E_HIP)
    if st == _lib.OK:
        _lib.lib().caddtree_plan_destroy(h)
