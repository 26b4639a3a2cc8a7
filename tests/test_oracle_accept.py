"""Pins for the oracle's synthetic acceptance (Sec. 3.3 tree verification, eq. surrogate).

* a hand-worked tree and target paths (tests/golden/hand_example_accept.json);
* exact expectation: summing alpha over every cell of the inverse-transform
  partition, weighted by the cell's probability, gives Phi(T) (eq. surrogate);
* Monte-Carlo: the mean accepted length over uniform draws estimates Phi(T);
* throughput: Theta = sum (1 + alpha) / sum C (Sec. 4.2) on a hand case;
* planted mistakes must fail one of these pins.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import accept as oacc
from tests.test_oracle_pins import _plant

HERE = os.path.dirname(os.path.abspath(__file__))


def _hand_round():
    with open(os.path.join(HERE, "golden", "hand_example.json")) as f:
        g = json.load(f)
    logits = np.log(np.array(g["q"], dtype=np.float64)).astype(np.float32)
    tv = 1.0 + g["t_verify_slope"] * np.arange(33, dtype=np.float64)
    return oracle.build_round(logits, "f32", g["K"], g["t_draft"], tv, 32), tv


def check_hand_accept():
    with open(os.path.join(HERE, "golden", "hand_example_accept.json")) as f:
        g = json.load(f)
    r, tv = _hand_round()
    for case in g["cases"]:
        assert oacc.sample_ranks(r.marg["logit"], r.marg["lse"], case["u"]) == case["ranks"], case
        assert oacc.simulate_round(r, case["u"]) == case["alpha"], case
    c = oacc.round_cost(1.0, tv, r.n_star)
    assert abs(oacc.throughput([2, 0], [c, c]) - g["throughput_two_rounds"]) < 1e-9


def _tiny(seed, L, K, V, cap, slope):
    rng = np.random.default_rng(seed)
    x = (1.3 * rng.standard_normal((L, V))).astype(np.float32)
    tv = 1.0 + slope * np.arange(cap + 1, dtype=np.float64)
    return oracle.build_round(x, "f32", K, 1.0, tv, cap)


def check_exact_expectation(seed=0, L=3, K=3, V=7, cap=30, slope=0.01):
    """E[alpha] over the inverse-transform partition equals Phi(T) (eq. surrogate)."""
    r = _tiny(seed, L, K, V, cap, slope)
    m = r.marg
    q = [[math.exp(float(m["logit"][i, k]) - float(m["lse"][i])) for k in range(K)] for i in range(L)]
    # cell j of position i: rank j (width q_i^(j)) for j < K, the outside bucket for j = K;
    # a uniform in the middle of the cell stands for the whole cell
    lows = [[sum(q[i][:j]) for j in range(K + 1)] for i in range(L)]
    highs = [[sum(q[i][:j + 1]) if j < K else 1.0 for j in range(K + 1)] for i in range(L)]
    total = 0.0
    for cells in itertools.product(range(K + 1), repeat=L):
        w = 1.0
        u = []
        for i, j in enumerate(cells):
            w *= highs[i][j] - lows[i][j]
            u.append(0.5 * (lows[i][j] + highs[i][j]))
        total += w * oacc.simulate_round(r, u)
    assert r.n_star > 2
    assert abs(total - r.exp.phi) < 1e-12, (total, r.exp.phi)


def test_hand_accept():
    check_hand_accept()


@pytest.mark.parametrize("seed", range(4))
def test_exact_expectation(seed):
    check_exact_expectation(seed)


def test_exact_expectation_deeper():
    check_exact_expectation(7, L=4, K=2, V=5, cap=40, slope=0.003)


@pytest.mark.parametrize("seed", [50, 51])
def test_monte_carlo_mean_is_phi(seed):
    r = _tiny(seed, 4, 3, 9, 60, 0.005)
    rng = np.random.default_rng(seed)
    M = 40000
    a = np.array([oacc.simulate_round(r, rng.random(4)) for _ in range(M)], dtype=np.float64)
    assert abs(a.mean() - r.exp.phi) < 4.5 * a.std() / math.sqrt(M)


def test_outside_mass_never_accepted():
    r = _tiny(3, 2, 2, 40, 10, 0.01)
    assert oacc.simulate_round(r, [0.999999, 0.1]) == 0


def test_sample_margin():
    r, _ = _hand_round()
    m = r.marg
    assert oacc.sample_margin(m["logit"], m["lse"], [0.1, 0.1]) > 0.5
    assert oacc.sample_margin(m["logit"], m["lse"], [0.6000001, 0.1]) < 1e-6


MUTATIONS = [
    ("oracle.accept", "if float(u[i]) < c:\n                pick = r", "if float(u[i]) < c:\n                pick = r + 1",
     check_hand_accept, ()),
    ("oracle.accept", "c = c + math.exp(float(logit[i, r]) - float(lse[i]))\n            if float(u[i]) < c:\n                pick",
     "c = math.exp(float(logit[i, r]) - float(lse[i]))\n            if float(u[i]) < c:\n                pick",
     check_exact_expectation, ()),
    ("oracle.accept", "        alpha = d\n", "        alpha = d + 1\n", check_hand_accept, ()),
    ("oracle.accept", "return float(sum(1 + a for a in alphas)) / float(sum(costs))",
     "return float(sum(alphas)) / float(sum(costs))", check_hand_accept, ()),
]


@pytest.mark.parametrize("i", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(monkeypatch, i):
    modname, old, new, check, args = MUTATIONS[i]
    check(*args)
    _plant(monkeypatch, modname, old, new)
    with pytest.raises(Exception):
        check(*args)
