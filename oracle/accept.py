"""Synthetic acceptance of a draft tree against a sampled target path (oracle; test infrastructure).

Tree verification (Sec. 3.3) accepts the longest prefix of the target's own
continuation that is a path of the draft tree; the round then emits those
alpha draft tokens plus one token from the target (the next bonus token).
Here the target continuation y = (y_1 .. y_L) is drawn from the drafter's
factorised distribution Q (eq. factorized), the distribution under which the
expected accepted length is Phi(T) (eq. surrogate).  Position i is drawn by
inverse transform from a uniform u_i in [0, 1):

* q_i^(k) = exp(l_i^(k) - LSE_i) for the K kept tokens, in rank order (the
  probabilities Algorithm 1 works with; no renormalisation);
* the cumulative sums c_r = q^(0) + ... + q^(r) are formed left to right in
  fp64;
* y_i is the rank-r token for the smallest r with u_i < c_r, and a token
  outside the top-K (which no tree node carries) when u_i >= c_{K-1}.

alpha is the largest d such that (y_1 .. y_d) is a node of the tree, 0 when
y_1 is not.  A round costs C(n*) = C_d + C_v(n*) (Sec. 4.2), and R rounds
give the throughput Theta_R = sum_t (1 + alpha_t) / sum_t C_t (Sec. 4.2);
its inverse is the time per token the paper's tables report.
"""

from __future__ import annotations

import math
from typing import Sequence

import numpy as np

OUTSIDE = -1


def sample_ranks(logit: np.ndarray, lse: np.ndarray, u: Sequence[float]) -> list:
    """Rank of the target token at every position (OUTSIDE when it is not among the top K)."""
    logit = np.asarray(logit, dtype=np.float64)
    L, K = logit.shape
    ranks = []
    for i in range(L):
        c = 0.0
        pick = OUTSIDE
        for r in range(K):
            c = c + math.exp(float(logit[i, r]) - float(lse[i]))
            if float(u[i]) < c:
                pick = r
                break
        ranks.append(pick)
    return ranks


def accepted_length(tree_ranks: Sequence[tuple], ranks: Sequence[int]) -> int:
    """Length of the longest prefix of the sampled rank path that is a node of the tree."""
    nodes = set(tuple(r) for r in tree_ranks)
    alpha = 0
    for d in range(1, len(ranks) + 1):
        if ranks[d - 1] == OUTSIDE or tuple(ranks[:d]) not in nodes:
            break
        alpha = d
    return alpha


def simulate_round(result, u: Sequence[float]) -> int:
    """alpha of one oracle round (``pipeline.RoundResult``) for the uniforms u [L]."""
    m = result.marg
    return accepted_length(result.tree.ranks, sample_ranks(m["logit"], m["lse"], u))


def round_cost(t_draft: float, t_verify: np.ndarray, n: int) -> float:
    """C(n) = C_d + C_v(n) (Sec. 4.2)."""
    return t_draft + float(t_verify[n])


def throughput(alphas: Sequence[int], costs: Sequence[float]) -> float:
    """Theta_R = sum (1 + alpha_t) / sum C_t over the rounds (Sec. 4.2)."""
    return float(sum(1 + a for a in alphas)) / float(sum(costs))


def sample_margin(logit: np.ndarray, lse: np.ndarray, u: Sequence[float]) -> float:
    """Smallest relative distance between a uniform and a cumulative boundary it is compared with.

    For the input guard: a log-normaliser perturbed by rounding scales every
    q_i^(k) of position i by one factor, so the draw can only change where u_i
    sits within that relative distance of some c_r."""
    logit = np.asarray(logit, dtype=np.float64)
    L, K = logit.shape
    worst = math.inf
    for i in range(L):
        c = 0.0
        for r in range(K):
            c = c + math.exp(float(logit[i, r]) - float(lse[i]))
            worst = min(worst, abs(float(u[i]) - c) / c)
            if float(u[i]) < c:
                break
    return worst
