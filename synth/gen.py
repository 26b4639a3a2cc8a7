"""Per-round logit generators.

Recipes (one round = an ``[L, V]`` block of drafter logits):

``normal``
    l = 3 z with z ~ N(0, 1), stored as fp32.
``peak``
    Gumbel noise g = -ln(-ln u), u ~ U(0, 1) in fp64 (u clipped to
    [2^-53, 1 - 2^-53] so both logarithms stay finite), over all V entries.
    One peak token per position, p_i ~ U{0 .. V-1}, boosted by
    a_i * (L - i + 1) / L with a_i ~ U(2, 12) for i = 1 .. L: the full boost at
    the first position, 1/L of it at the last.  Cast to fp32 (round to
    nearest), then to bf16 (round to nearest even) for bf16 workloads.
``peak_temp``
    ``peak`` divided, in fp32, by a per-position temperature drawn uniformly
    from {0.3, 1, 3} before the bf16 cast, so sharp and flat positions mix in
    one round.
``peak_cold``
    ``peak`` divided by 0.3 at every position (fp32).

Draw order inside a round is fixed: the (L, V) uniforms (or normals), then the
L peak ids, then the L boost amplitudes, then the L temperatures.
"""

from __future__ import annotations

import os
from typing import Dict, Iterable, Optional, Sequence

import numpy as np

from .configs import Config

_TEMPS = np.array([0.3, 1.0, 3.0], dtype=np.float64)


def _rng(seed: int, b: int, attempt: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(b, attempt))))


def bf16_bits_from_f32(x32: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    bits = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    bias = ((bits >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((bits + bias) >> np.uint32(16)).astype(np.uint16)


def _draw_f32(cfg: Config, b: int, attempt: int) -> np.ndarray:
    rng = _rng(cfg.seed, b, attempt)
    L, V = cfg.L, cfg.V
    if cfg.recipe == "normal":
        return (3.0 * rng.standard_normal((L, V))).astype(np.float32)
    u = rng.random((L, V))
    np.clip(u, 2.0 ** -53, 1.0 - 2.0 ** -53, out=u)
    np.log(u, out=u)
    np.negative(u, out=u)
    np.log(u, out=u)
    np.negative(u, out=u)          # u now holds the Gumbel noise g
    peak = rng.integers(0, V, size=L)
    amp = rng.uniform(2.0, 12.0, size=L)
    pos = np.arange(1, L + 1, dtype=np.float64)
    u[np.arange(L), peak] += amp * (L - pos + 1.0) / L
    x32 = u.astype(np.float32)
    if cfg.recipe == "peak_temp":
        temp = rng.choice(_TEMPS, size=L).astype(np.float32)
        x32 = (x32 / temp[:, None]).astype(np.float32)
    elif cfg.recipe == "peak_cold":
        x32 = (x32 / np.float32(0.3)).astype(np.float32)
    elif cfg.recipe != "peak":
        raise ValueError(f"unknown recipe {cfg.recipe!r}")
    return x32


def draw_round(cfg: Config, b: int, attempt: int = 0) -> np.ndarray:
    """Logits of round ``b`` (redraw ``attempt``): float32 or uint16 bf16 bits, shape [L, V]."""
    x32 = _draw_f32(cfg, b, attempt)
    if cfg.dtype == "bf16":
        return bf16_bits_from_f32(x32)
    if cfg.dtype == "f32":
        return x32
    raise ValueError(f"unknown dtype {cfg.dtype!r}")


def np_dtype(cfg: Config):
    return np.uint16 if cfg.dtype == "bf16" else np.float32


# ---------------------------------------------------------------- batches

def draw_batch(cfg: Config, rounds: Optional[Sequence[int]] = None,
               attempts: Optional[Dict[int, int]] = None, workers: int = 1,
               out: Optional[np.ndarray] = None) -> np.ndarray:
    """Logits of a batch, shape [len(rounds), L, V].

    ``rounds`` defaults to ``range(cfg.B)``; ``attempts`` maps a round index to
    its redraw attempt (default 0).  ``workers > 1`` fills the rounds from a
    pool of threads (numpy's generators and ufuncs release the GIL), so no
    child process is started.
    """
    rounds = list(range(cfg.B)) if rounds is None else list(rounds)
    attempts = attempts or {}
    n = len(rounds)
    shape = (n, cfg.L, cfg.V)
    dt = np_dtype(cfg)
    if out is None:
        out = np.empty(shape, dtype=dt)
    assert out.shape == shape and out.dtype == dt

    def fill(i: int) -> None:
        b = rounds[i]
        out[i] = draw_round(cfg, b, attempts.get(b, 0))

    workers = max(1, min(int(workers), n))
    if workers == 1:
        for i in range(n):
            fill(i)
        return out
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(fill, range(n)))
    return out


def default_workers() -> int:
    """Generator threads: every core this process may use, at most 16 (the host share of one GPU)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def iter_rounds(cfg: Config, rounds: Iterable[int]):
    for b in rounds:
        yield b, draw_round(cfg, b)
