"""Input guard: redraw rounds whose tree decisions sit within a hair of a tie.

A GPU log-normaliser LSE_i differs from the oracle's fp64 value by at most
``LSE_ATOL`` (the parity tests check it), and the log prefix probability of a
depth-d node carries the sum of d such errors.  So a stop decision or a
selected-versus-frontier comparison between depths d and d' can flip only if
its margin is below span * LSE_ATOL, with span the depth (stop) or |d - d'|
(comparison) that ``oracle.decision_margins`` reports.  The guard keeps every
margin of a round at or above max(TAU, 2 * span * LSE_ATOL): TAU = 1e-6 is
the gap the workloads require, and the factor 2 leaves headroom for the
relative form of the stop margin.  A round that fails is redrawn with the next
attempt of its seed.  Same-depth comparisons are exact on both sides and need
no guard.
"""

from __future__ import annotations

from typing import Dict, Tuple

import numpy as np

import oracle
import synth
from tests._parity import LSE_ATOL

TAU = 1e-6
MAX_ATTEMPTS = 20


def required(span: int, tau: float = TAU) -> float:
    """The margin a decision whose error can reach span normalisers must keep."""
    return max(tau, 2.0 * span * LSE_ATOL)


def clears(m: "oracle.Margins", tau: float = TAU) -> bool:
    return all(v >= required(span, tau) for v, span in m.stop + m.cross)


_CTX_CACHE: Dict[Tuple[str, int], Tuple[np.ndarray, np.ndarray, np.ndarray]] = {}


def ctx_inputs(cfg: synth.Config):
    """(grid, tables, context length of every round of the full batch) of a context-aware workload."""
    key = (cfg.name, cfg.B)
    if key not in _CTX_CACHE:
        grid, tables = synth.ctx_tables(cfg)
        _CTX_CACHE[key] = (grid, tables, synth.ctx_lengths(cfg, cfg.B))
    return _CTX_CACHE[key]


def round_cost(cfg: synth.Config, b: int) -> np.ndarray:
    """C_v(0..cap) of round b: the workload's table, or the oracle's interpolation at the round's context."""
    if not cfg.ctx:
        return synth.cost_table(cfg)
    grid, tables, ell = ctx_inputs(cfg)
    return oracle.context_cost(tables, grid, int(ell[b]))


def oracle_round(cfg: synth.Config, x: np.ndarray, pos_offset: int = 0, mask=None, b: int = 0):
    return oracle.build_round(x, cfg.dtype, cfg.K, cfg.t_draft, round_cost(cfg, b), cfg.cap,
                              pos_offset=pos_offset, mask=mask or cfg.mask,
                              budget=cfg.cap if cfg.fixed else None)


def guarded_round(cfg: synth.Config, b: int, tau: float = TAU, pos_offset: int = 0):
    """(attempt, logits, oracle result) for round b, redrawn until its margins clear tau."""
    for a in range(MAX_ATTEMPTS):
        x = synth.draw_round(cfg, b, a)
        r = oracle_round(cfg, x, pos_offset, b=b)
        if clears(oracle.decision_margins(r.exp), tau):
            return a, x, r
    raise RuntimeError(f"round {b} of {cfg.name} failed the guard {MAX_ATTEMPTS} times")


def guarded_batch(cfg: synth.Config, rounds, tau: float = TAU, pos_offset: int = 0):
    """Returns (attempts {b: a}, logits [n, L, V], [oracle results]) for the given rounds."""
    attempts: Dict[int, int] = {}
    xs, rs = [], []
    for b in rounds:
        a, x, r = guarded_round(cfg, b, tau, pos_offset)
        attempts[b] = a
        xs.append(x)
        rs.append(r)
    return attempts, np.stack(xs), rs


def guarded_uniforms(cfg: synth.Config, rs, rounds, tau: float = TAU, max_draws: int = MAX_ATTEMPTS):
    """Uniforms [len(rounds), L] for the acceptance draw of the given rounds (oracle results rs): each
    round takes the first draw whose uniforms keep a relative distance of at least tau from every
    cumulative boundary they are compared with."""
    draws = [synth.accept_uniforms(cfg, max(rounds) + 1, k) for k in range(max_draws)]
    out = np.empty((len(rounds), cfg.L))
    for j, (b, r) in enumerate(zip(rounds, rs)):
        for k in range(max_draws):
            u = draws[k][b]
            if oracle.accept.sample_margin(r.marg["logit"], r.marg["lse"], u) >= tau:
                out[j] = u
                break
        else:
            raise RuntimeError(f"round {b}: no acceptance draw clears the guard")
    return out
