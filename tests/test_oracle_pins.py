"""Pins for the CPU oracle: it is checked against what the paper and the mathematics fix.

* a hand-worked round (tests/golden/hand_example.json);
* library routines and closed forms for the log-normaliser;
* brute force over every node on tiny inputs (top-n sets, eq. phistar);
* exhaustive enumeration of every prefix-closed subtree (Prop. 1, Cor. 2);
* unimodality of theta*(n) under convex cost (Thm. 1) and monotone Phi*(n);
* special cases: constant cost grows to the cap (Sec. 5.4, Tab. 2 text), K = 1
  chain, L = 1 sorted top-K, prohibitive cost gives an empty tree, exact ties
  stop (Algorithm 1 uses <=);
* Monte-Carlo: Phi(T) is the expected accepted length under the drafter's
  factorised joint (eq. surrogate);
* mask invariants;
* the decision margins of the hand-worked round (tests/golden/hand_example_margins.json),
  which the input guard uses to pick the rounds the parity tests compare;
* planted mistakes: each mutation of the oracle below fails one of the pins.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import alg1 as oexpand
from oracle import vocab as omarg
from oracle import layout as otree
from tests import _brute as brute

HERE = os.path.dirname(os.path.abspath(__file__))


def _hand():
    with open(os.path.join(HERE, "golden", "hand_example.json")) as f:
        return json.load(f)


def _costs_linear(cap, slope):
    return 1.0 + slope * np.arange(cap + 1, dtype=np.float64)


# ----------------------------------------------------------------- pin checks
# Each check raises AssertionError on a mismatch; the mutation tests reuse them.

def check_hand_example():
    g = _hand()
    logits = np.log(np.array(g["q"], dtype=np.float64)).astype(np.float32)
    # the float32 logits are what both sides see; q is recovered to ~1e-7, far inside the margins
    for case in g["cases"]:
        cap = case["cap"]
        tv = _costs_linear(cap, g["t_verify_slope"])
        r = oracle.build_round(logits, "f32", g["K"], g["t_draft"], tv, cap,
                               pos_offset=case["pos_offset"], mask="u8")
        assert r.n_star == case["n_star"], (cap, r.n_star)
        assert r.tree.token_ids.tolist() == case["token_ids"]
        assert r.tree.parent.tolist() == case["parent"]
        assert r.tree.depth.tolist() == case["depth"]
        assert r.tree.pos_ids.tolist() == case["pos_ids"]
        assert r.mask.tolist() == case["mask"]
        np.testing.assert_allclose(r.tree.path_prob, case["path_prob"], rtol=1e-6)
        assert math.isclose(r.exp.phi, case["phi"], rel_tol=1e-6)
        assert math.isclose(r.exp.theta, case["theta"], rel_tol=1e-6)


def _tiny_round(seed, L, K, V, scale=1.5):
    rng = np.random.default_rng(seed)
    return (scale * rng.standard_normal((L, V))).astype(np.float32)


def check_top_n_bruteforce(seed, L, K, V):
    """Fixed-budget expansion pops exactly the top-n nodes by pi, for every n (eq. phistar)."""
    x = _tiny_round(seed, L, K, V)
    q = brute.softmax_direct(x.astype(np.float64))
    ids = np.stack([brute.topk_by_sort(x[i], K) for i in range(L)])
    nodes = brute.all_nodes(q, ids)
    by_pi = sorted(nodes.items(), key=lambda kv: -kv[1])
    m = omarg.marginals(x, "f32", K)
    assert np.array_equal(m["ids"], ids)
    total = len(nodes)
    for n in range(total + 1):
        ex = oexpand.expand(m["logit"], m["lse"], 1.0, np.ones(total + 1), cap=total, budget=n)
        got = {nd.ranks for nd in ex.selected}
        want = {r for r, _ in by_pi[:n]}
        assert got == want, (n, sorted(got), sorted(want))
        np.testing.assert_allclose(ex.deltas, [p for _, p in by_pi[:n]], rtol=1e-12)


def check_prop1_exhaustive(seed, L, K, V, slope=0.05, quad=0.01, cap=None):
    """Exhaustive subtree enumeration: max Phi at every size equals the greedy Phi*(n)
    (Prop. 1), and the method's theta is the maximum over all valid trees (Cor. 2)."""
    x = _tiny_round(seed, L, K, V)
    q = brute.softmax_direct(x.astype(np.float64))
    ids = np.stack([brute.topk_by_sort(x[i], K) for i in range(L)])
    nodes = brute.all_nodes(q, ids)
    trees = brute.enumerate_trees(nodes, L, K)
    best = brute.best_phi_by_size(trees)
    total = len(nodes)
    cap = total if cap is None else cap
    nn = np.arange(total + 1, dtype=np.float64)
    tv = 1.0 + slope * nn + quad * nn * nn
    m = omarg.marginals(x, "f32", K)
    for n in range(total + 1):
        ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=total, budget=n)
        assert math.isclose(ex.phi, best[n], rel_tol=1e-12, abs_tol=1e-15), (n, ex.phi, best[n])
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=cap)
    th = {n: (1.0 + best[n]) / (1.0 + tv[n]) for n in best if n <= cap}
    tmax = max(th.values())
    n_arg = min(n for n, t in th.items() if t >= tmax * (1 - 1e-13))
    assert ex.n_star == n_arg, (ex.n_star, n_arg)
    assert math.isclose(ex.theta, tmax, rel_tol=1e-12)


def check_unimodal_argmax(seed, L, K, V, slope, quad, cap):
    """theta*(n) from brute-force sorted deltas is unimodal under convex cost (Thm. 1);
    the greedy stop is its first maximiser (Cor. 2); Phi*(n) is non-decreasing."""
    x = _tiny_round(seed, L, K, V)
    q = brute.softmax_direct(x.astype(np.float64))
    ids = np.stack([brute.topk_by_sort(x[i], K) for i in range(L)])
    deltas = brute.sorted_deltas(brute.all_nodes(q, ids))
    nn = np.arange(cap + 1, dtype=np.float64)
    tv = 1.0 + slope * nn + quad * nn * nn
    th = brute.theta_curve(deltas, 1.0, tv, cap)
    assert np.all(np.diff(np.cumsum(deltas)) >= 0)
    k = int(np.argmax(th))
    tol = 1e-13
    assert np.all(np.diff(th[: k + 1]) >= -tol) and np.all(np.diff(th[k:]) <= tol)
    m = omarg.marginals(x, "f32", K)
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=cap)
    assert ex.n_star == k, (ex.n_star, k)
    np.testing.assert_allclose(ex.deltas, deltas[: ex.n_star], rtol=1e-12)


def check_topk_ties():
    x = np.array([1.0, 3.0, 3.0, 2.0, 3.0, 0.0], dtype=np.float32)
    ids, vals = omarg.top_k(x, 4)
    assert ids.tolist() == [1, 2, 4, 3], ids
    assert vals.tolist() == [3.0, 3.0, 3.0, 2.0]
    y = np.array([-1.0, -1.0, -1.0], dtype=np.float32)
    assert omarg.top_k(y, 2)[0].tolist() == [0, 1]


def check_hand_margins():
    """Stop margins and cross-depth gaps of the hand-worked round, with their depth spans."""
    g = _hand()
    with open(os.path.join(HERE, "golden", "hand_example_margins.json")) as f:
        gm = json.load(f)
    logits = np.log(np.array(g["q"], dtype=np.float64)).astype(np.float32)
    for case in gm["cases"]:
        cap = case["cap"]
        r = oracle.build_round(logits, "f32", g["K"], g["t_draft"], _costs_linear(cap, g["t_verify_slope"]), cap)
        m = oracle.decision_margins(r.exp)
        assert [sp for _, sp in m.stop] == [sp for _, sp in case["stop"]], (cap, m.stop)
        np.testing.assert_allclose([v for v, _ in m.stop], [v for v, _ in case["stop"]], rtol=2e-6)
        got = sorted(m.cross)
        want = sorted(tuple(c) for c in case["cross"])
        assert [sp for _, sp in got] == [sp for _, sp in want], (cap, got)
        np.testing.assert_allclose([v for v, _ in got], [v for v, _ in want], rtol=0, atol=1e-6)


def check_tie_stops():
    # V = 2 equal logits: q = 0.5 exactly; C(0) = 2, C(1) = 3 gives theta_new = 1.5 / 3 = theta_prev
    x = np.zeros((1, 2), dtype=np.float32)
    m = omarg.marginals(x, "f32", 2)
    assert math.exp(m["lq"][0, 0]) == 0.5
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, np.array([1.0, 2.0, 3.0]), cap=2)
    assert ex.n_star == 0 and ex.stop == "rule"
    assert ex.theta == 0.5


# ----------------------------------------------------------------- tests

def test_hand_example():
    check_hand_example()


def test_hand_example_bits_mask():
    g = _hand()
    case = g["cases"][0]
    bits = otree.emit_mask(np.array(case["parent"]), "bits", cap=40)
    assert bits.shape == (4, 2)
    want = [sum(1 << j for j, v in enumerate(row) if v) for row in case["mask"]]
    assert bits[:, 0].tolist() == want and not bits[:, 1].any()


@pytest.mark.parametrize("seed", range(5))
def test_lse_matches_scipy(seed):
    from scipy.special import logsumexp
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(5000) * rng.uniform(0.1, 20)).astype(np.float32)
    assert math.isclose(omarg.log_normalizer(x), float(logsumexp(x.astype(np.float64))), rel_tol=1e-14, abs_tol=1e-13)


def test_lse_uniform_closed_form():
    for V in (1, 7, 1024, 151936):
        x = np.full(V, 2.5, dtype=np.float32)
        m = omarg.marginals(x[None, :], "f32", 1)
        assert math.isclose(m["lse"][0], 2.5 + math.log(V), rel_tol=1e-15)
        assert math.isclose(m["lq"][0, 0], -math.log(V), rel_tol=1e-13, abs_tol=1e-15)


def test_lse_rejects_nonfinite():
    with pytest.raises(ValueError):
        omarg.log_normalizer(np.array([0.0, np.inf]))


def test_bf16_widening_exact():
    bits = np.array([[0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x4120, 0x7F7F]], dtype=np.uint16)
    w = omarg.widen(bits, "bf16")
    assert w[0, :6].tolist() == [1.0, -2.0, 1.0078125, 0.0, -0.0, 10.0]
    assert w[0, 6] == float.fromhex("0x1.fep127")


def test_topk_ties():
    check_topk_ties()


@pytest.mark.parametrize("seed", range(4))
def test_topk_against_stable_sort(seed):
    rng = np.random.default_rng(100 + seed)
    x = np.round(rng.standard_normal(3000) * 4) / 4  # heavy ties
    ids, vals = omarg.top_k(x.astype(np.float32), 16)
    assert ids.tolist() == brute.topk_by_sort(x, 16).tolist()
    assert np.all(np.diff(vals) <= 0)


@pytest.mark.parametrize("seed,L,K,V", [(0, 2, 2, 4), (1, 3, 2, 5), (2, 2, 3, 5), (3, 3, 3, 6), (4, 1, 5, 8), (5, 4, 2, 3)])
def test_top_n_bruteforce(seed, L, K, V):
    check_top_n_bruteforce(seed, L, K, V)


@pytest.mark.parametrize("seed,L,K,V", [(10, 3, 2, 4), (11, 3, 2, 6), (12, 2, 3, 5), (13, 2, 4, 6)])
def test_prop1_exhaustive(seed, L, K, V):
    check_prop1_exhaustive(seed, L, K, V)


def test_prop1_exhaustive_with_cap():
    check_prop1_exhaustive(14, 3, 2, 5, slope=0.0, quad=0.0, cap=5)


def test_subtree_counts():
    # g(L) = (1 + g(L - 1))^K counts prefix-closed trees incl. the empty one
    for L, K, want in [(3, 2, 676), (2, 3, 729), (2, 4, 83521)]:
        nodes = {r: 0.0 for d in range(1, L + 1) for r in __import__("itertools").product(range(K), repeat=d)}
        assert len(brute.enumerate_trees(nodes, L, K)) == want


@pytest.mark.parametrize("seed", range(8))
def test_unimodal_argmax(seed):
    rng = np.random.default_rng(seed)
    slope, quad = float(rng.uniform(0.0, 0.1)), float(rng.uniform(0.0, 0.01))
    check_unimodal_argmax(seed, 3, 3, 6, slope, quad, cap=39)


def test_constant_cost_grows_to_cap():
    x = _tiny_round(21, 3, 3, 7)
    m = omarg.marginals(x, "f32", 3)
    total = 3 + 9 + 27
    for cap in (0, 1, 10, total, total + 5):
        ex = oexpand.expand(m["logit"], m["lse"], 1.0, np.ones(cap + 1), cap=cap)
        assert ex.n_star == min(cap, total)
        assert ex.stop == ("cap" if cap < total else "exhausted")


def test_k1_chain():
    x = _tiny_round(22, 5, 1, 9)
    q = brute.softmax_direct(x.astype(np.float64))
    m = omarg.marginals(x, "f32", 1)
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, np.ones(6), cap=5)
    assert [nd.ranks for nd in ex.selected] == [(0,) * d for d in range(1, 6)]
    want = np.cumprod(q.max(axis=1))
    np.testing.assert_allclose(ex.deltas, want, rtol=1e-12)


def test_l1_sorted_topk():
    x = _tiny_round(23, 1, 6, 10)
    q = brute.softmax_direct(x.astype(np.float64))[0]
    m = omarg.marginals(x, "f32", 6)
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, np.ones(7), cap=6)
    assert [nd.ranks for nd in ex.selected] == [(k,) for k in range(6)]
    np.testing.assert_allclose(ex.deltas, np.sort(q)[::-1][:6], rtol=1e-12)


def test_prohibitive_cost_empty_tree():
    x = _tiny_round(24, 3, 3, 7)
    m = omarg.marginals(x, "f32", 3)
    tv = 1.0 + 1e6 * np.arange(11, dtype=np.float64)
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=10)
    assert ex.n_star == 0 and ex.phi == 0.0
    assert ex.theta == 1.0 / 2.0
    r = oracle.build_round(x, "f32", 3, 1.0, tv, 10)
    assert r.mask.shape == (0, 0) and len(r.tree.token_ids) == 0


def test_ties_stop():
    check_tie_stops()


def test_hand_margins():
    check_hand_margins()


def test_guard_threshold_grows_with_depth_span():
    from tests import _guard
    M = oracle.Margins
    assert _guard.required(1) == _guard.TAU
    assert _guard.required(30) == 2 * 30 * _guard.LSE_ATOL > _guard.TAU
    assert _guard.clears(M(stop=[(2e-6, 3)], cross=[(1.5e-6, 2)]))
    # a gap of 3e-6 between depths 1 and 19 may flip under 18 normaliser errors of 1e-7 each
    assert not _guard.clears(M(stop=[], cross=[(3e-6, 18)]))
    assert not _guard.clears(M(stop=[(3e-6, 19)], cross=[]))
    assert not _guard.clears(M(stop=[(9e-7, 1)], cross=[]))


def test_margins_of_deep_rounds_carry_their_depth():
    """Every stop margin's span is at least the tested node's depth, and every cross-depth gap is
    non-negative (a frontier node never precedes a selected one)."""
    x = _tiny_round(27, 6, 2, 5, scale=0.3)
    nn = np.arange(64, dtype=np.float64)
    r = oracle.build_round(x, "f32", 2, 1.0, 1.0 + 0.001 * nn, 63)
    m = oracle.decision_margins(r.exp)
    assert max(sp for _, sp in m.stop) == max(s.depth for s in r.exp.steps) >= 3
    assert all(v >= 0 for v, _ in m.cross) and all(sp >= 1 for _, sp in m.cross)


def test_flat_cost_region_always_expands():
    # zero marginal cost makes theta rise strictly, so the tree reaches the end of the flat region
    x = _tiny_round(25, 4, 3, 8)
    m = omarg.marginals(x, "f32", 3)
    cap = 60
    tv = np.where(np.arange(cap + 1) <= 20, 1.0, 1.0 + 5.0 * (np.arange(cap + 1) - 20))
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=cap)
    assert ex.n_star >= 20


def test_lemma1_weighted_average():
    x = _tiny_round(26, 3, 3, 7)
    m = omarg.marginals(x, "f32", 3)
    nn = np.arange(40, dtype=np.float64)
    tv = 1.0 + 0.03 * nn + 0.002 * nn * nn
    ex = oexpand.expand(m["logit"], m["lse"], 1.0, tv, cap=39, budget=39)
    phi = np.concatenate([[0.0], np.cumsum(ex.deltas)])
    C = 1.0 + tv
    th = (1 + phi) / C[: len(phi)]
    for n in range(len(ex.deltas)):
        w = C[n] / C[n + 1]
        rho = ex.deltas[n] / (C[n + 1] - C[n])
        assert math.isclose(th[n + 1], w * th[n] + (1 - w) * rho, rel_tol=1e-13)
        assert (th[n + 1] > th[n]) == (rho > th[n])


@pytest.mark.parametrize("seed", [30, 31])
def test_phi_is_expected_acceptance(seed):
    """E_Q[alpha] = Phi(T): alpha = length of the longest prefix of y ~ Q lying in T (eq. surrogate)."""
    L, K, V = 3, 3, 6
    x = _tiny_round(seed, L, K, V, scale=1.2)
    nn = np.arange(40, dtype=np.float64)
    r = oracle.build_round(x, "f32", K, 1.0, 1.0 + 0.02 * nn, 39)
    paths = {tuple(int(t) for t in _path_tokens(r.tree, i)) for i in range(r.n_star)}
    q = brute.softmax_direct(x.astype(np.float64))
    rng = np.random.default_rng(seed)
    M = 200_000
    ys = np.stack([rng.choice(V, size=M, p=q[i]) for i in range(L)], axis=1)
    alpha = np.zeros(M)
    alive = np.ones(M, dtype=bool)
    for d in range(1, L + 1):
        hit = np.array([tuple(y[:d]) in paths for y in ys.tolist()]) & alive
        alpha += hit
        alive = hit
    mean, sd = alpha.mean(), alpha.std() / math.sqrt(M)
    assert abs(mean - r.exp.phi) < 4.5 * sd + 1e-12, (mean, r.exp.phi, sd)


def _path_tokens(tree, i):
    out = []
    while i >= 0:
        out.append(tree.token_ids[i])
        i = int(tree.parent[i])
    return out[::-1]


@pytest.mark.parametrize("seed", range(4))
def test_mask_invariants(seed):
    x = _tiny_round(40 + seed, 5, 3, 8, scale=0.8)
    r = oracle.build_round(x, "f32", 3, 1.0, np.ones(101), 100, mask="u8")
    M, par, dep = r.mask, r.tree.parent, r.tree.depth
    n = r.n_star
    assert n == 100
    assert np.all(np.diag(M) == 1)
    assert np.all(np.triu(M, 1) == 0)
    assert np.array_equal(M.sum(axis=1), dep)
    for i in range(n):
        row = np.zeros(n, dtype=np.uint8) if par[i] < 0 else M[par[i]].copy()
        row[i] = 1
        assert np.array_equal(M[i], row)
    bits = otree.emit_mask(par, "bits", cap=100)
    unpacked = np.array([[(bits[i, j // 32] >> (j % 32)) & 1 for j in range(n)] for i in range(n)])
    assert np.array_equal(unpacked, M)
    # canonical order: depth ascending, rank tuples ascending within a depth, parents first
    keys = [(len(rk), rk) for rk in r.tree.ranks]
    assert keys == sorted(keys)
    assert all(par[i] < i for i in range(n))


# ----------------------------------------------------------------- planted mistakes
# Each mutation edits one line of the oracle's own source, loads the edited
# module in place of the original, and expects at least one pin to fail.

def _plant(monkeypatch, modname, old, new):
    import importlib
    import inspect
    import sys
    import types
    mod = importlib.import_module(modname)
    src = inspect.getsource(mod)
    assert src.count(old) == 1, (modname, old)
    mutant = types.ModuleType(modname)
    mutant.__package__ = "oracle"
    mutant.__file__ = mod.__file__
    exec(compile(src.replace(old, new), mod.__file__, "exec"), mutant.__dict__)
    for key in [k for k in list(sys.modules) if k == "oracle" or k.startswith("oracle.")]:
        holder = sys.modules[key]
        for name, val in list(vars(holder).items()):
            if (inspect.isfunction(val) or inspect.isclass(val)) and val.__module__ == modname \
                    and hasattr(mutant, name):
                monkeypatch.setattr(holder, name, getattr(mutant, name))


MUTATIONS = [
    ("oracle.vocab", "np.lexsort((ids, -x))", "np.lexsort((-ids, -x))", check_topk_ties, ()),
    ("oracle.vocab", "return m + float(np.log(np.sum(np.exp(x - m))))",
     "return float(np.log(np.sum(np.exp(x - m))))", check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.vocab", "return {\"ids\": ids, \"logit\": val, \"lq\": val - lse[:, None], \"lse\": lse}",
     "return {\"ids\": ids, \"logit\": val[::-1].copy(), \"lq\": val - lse[:, None], \"lse\": lse}",
     check_top_n_bruteforce, (3, 3, 3, 6)),
    ("oracle.alg1", "kept = not (theta_new <= theta_prev)", "kept = not (theta_new < theta_prev)", check_tie_stops, ()),
    ("oracle.alg1", "A[d] = A[d - 1] + float(lse[d - 1])", "A[d] = A[d - 1] + float(lse[d % len(lse)])",
     check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.alg1", "sig = min(lam - float(self.A[d]), base_sig)", "sig = min(lam + float(self.A[d]), base_sig)",
     check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.alg1", "for r in range(self.K):", "for r in range(self.K - 1):", check_top_n_bruteforce, (2, 2, 3, 5)),
    ("oracle.alg1", "if len(prefix) == self.L:", "if len(prefix) == self.L - 1:", check_top_n_bruteforce, (2, 3, 2, 5)),
    ("oracle.alg1", "lam = base_lam + float(self.logit[d - 1, ranks[-1]])",
     "lam = base_lam + float(self.logit[ranks[-1] % self.L, (d - 1) % self.K])", check_top_n_bruteforce, (3, 3, 3, 6)),
    ("oracle.alg1", "order = sorted(listed, key=Node.key)", "order = sorted(listed, key=lambda nd: (nd.depth, nd.ranks))",
     check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.alg1", "if child.sigma < tau:", "if child.sigma < tau and r > 0:", check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.alg1", "complete = len(listed) == tree.total", "complete = True", check_top_n_bruteforce, (1, 3, 2, 5)),
    ("oracle.alg1", "theta_new = (1.0 + phi + delta) / C(n + 1)", "theta_new = (phi + delta) / C(n + 1)",
     check_hand_example, ()),
    ("oracle.alg1", "theta_new = (1.0 + phi + delta) / C(n + 1)", "theta_new = (1.0 + phi + delta) / C(n)",
     check_hand_example, ()),
    ("oracle.alg1", "if nd.depth < tree.L:", "if nd.depth < tree.L - 1:", check_hand_margins, ()),
    ("oracle.alg1", "if r + 1 < tree.K:", "if r + 1 < tree.K - 1:", check_hand_margins, ()),
    ("oracle.pipeline", "a = s.delta * s.c_n", "a = s.delta * s.c_next", check_hand_margins, ()),
    ("oracle.pipeline", "b = (1.0 + s.phi) * c", "b = s.phi * c", check_hand_margins, ()),
    ("oracle.pipeline", "stop.append((abs(a - b) / (abs(a) + abs(b)), max(s.depth, deepest)))",
     "stop.append((abs(a - b) / (abs(a) + abs(b)), s.depth))", check_hand_margins, ()),
    ("oracle.pipeline", "if d2 != d:", "if True:", check_hand_margins, ()),
    ("oracle.layout", "key=lambda i: (len(ranks[i]), ranks[i])", "key=lambda i: i", check_hand_example, ()),
    ("oracle.layout", "return TreeOut(rk, tok, par, dep, prob, pos_offset + dep)",
     "return TreeOut(rk, tok, par, dep, prob, pos_offset + dep - 1)", check_hand_example, ()),
    ("oracle.layout", "tok[i] = int(topk_ids[d - 1, r[-1]])", "tok[i] = int(topk_ids[r[-1] % topk_ids.shape[0], d - 1])",
     check_hand_example, ()),
]


@pytest.mark.parametrize("i", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(monkeypatch, i):
    modname, old, new, check, args = MUTATIONS[i]
    check(*args)                      # the pin holds on the real oracle
    _plant(monkeypatch, modname, old, new)
    with pytest.raises(Exception):
        check(*args)
