"""Workload configurations: shapes, dtypes, generator recipe and cost tables.

The five graded workloads (``c0`` .. ``c4``), two ungraded stress workloads
(``s1``, ``s2``) and variants that exercise the context-aware cost and the
fixed-budget mode.  Costs are in arbitrary units; the drafting cost is 1.0
everywhere.  The verification cost is given as a table ``C_v(0..cap)``, the
form in which the method consumes it (a profiled, convex, non-decreasing
function of the node count; the paper's cost model, Sec. 4.2 and Sec. 4.6).

Context-aware variants carry one table per point of a context-length grid
(Sec. 4.6 profiles at 0, 1k, .., 8k tokens) and a context length per round.
"""

from __future__ import annotations

import dataclasses
from typing import Callable, Dict

import numpy as np

SEED_BASE = 260601813


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    B: int            # rounds per batch
    L: int            # block positions per round
    V: int            # vocabulary size
    dtype: str        # "f32" or "bf16"
    K: int            # top-K per position
    cap: int          # budget cap (maximum number of draft nodes)
    t_draft: float    # C_d
    cost: str         # name of the C_v recipe, see ``cost_table``
    mask: str         # "u8" (dense bytes) or "bits" (packed u32, LSB first)
    recipe: str       # "normal", "peak" or "peak_temp"
    seed: int
    ctx: str = ""     # context-cost recipe (``ctx_tables``); "" = one table
    fixed: bool = False   # fixed-budget mode: the top-``cap`` tree, no stop rule

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def row_bytes(self) -> int:
        return self.V * self.elem_bytes

    @property
    def batch_bytes(self) -> int:
        return self.B * self.L * self.V * self.elem_bytes

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


def _quad(a: float, b: float) -> Callable[[np.ndarray], np.ndarray]:
    return lambda n: 1.0 + a * n + b * n * n


def _piecewise_c3(n: np.ndarray) -> np.ndarray:
    # flat at 1.0 up to n = 64, slope 0.004 up to n = 256, slope 0.012 beyond
    return np.where(n <= 64, 1.0,
                    np.where(n <= 256, 1.0 + 0.004 * (n - 64),
                             1.768 + 0.012 * (n - 256)))


def _flat_then_rise(f: int) -> Callable[[np.ndarray], np.ndarray]:
    # flat at 1.0 up to n = f, then a convex rise (the marginal grows from 0.004)
    return lambda n: np.where(n <= f, 1.0, 1.0 + 0.004 * (n - f) + 0.00002 * (n - f) * (n - f))


_COSTS: Dict[str, Callable[[np.ndarray], np.ndarray]] = {
    "c0": _quad(0.01, 0.0005),
    "c1": _quad(0.002, 0.00002),
    "c3": _piecewise_c3,
    "c4": _quad(0.001, 0.000005),
    "const": lambda n: np.ones_like(n, dtype=np.float64),
    "tiny": lambda n: 1.0 + 1e-6 * n,          # almost flat: trees of hundreds of nodes
    # flat starts of other lengths than c3's 64 (test workloads)
    "flat16": _flat_then_rise(16),
    "flat32": _flat_then_rise(32),
    "flat128": _flat_then_rise(128),
    "flat200": _flat_then_rise(200),
}


def cost_table(cfg_or_name, cap: int | None = None) -> np.ndarray:
    """C_v(0..cap) as float64, length cap + 1."""
    if isinstance(cfg_or_name, Config):
        name, cap = cfg_or_name.cost, cfg_or_name.cap if cap is None else cap
    else:
        name = cfg_or_name
    n = np.arange(cap + 1, dtype=np.float64)
    return np.ascontiguousarray(_COSTS[name](n), dtype=np.float64)


V_FULL = 151936

CONFIGS: Dict[str, Config] = {
    "c0": Config("c0", B=1, L=4, V=1024, dtype="f32", K=4, cap=32, t_draft=1.0,
                 cost="c0", mask="u8", recipe="normal", seed=SEED_BASE + 0),
    "c1": Config("c1", B=64, L=16, V=V_FULL, dtype="bf16", K=8, cap=512, t_draft=1.0,
                 cost="c1", mask="u8", recipe="peak", seed=SEED_BASE + 1),
    "c2": Config("c2", B=1024, L=16, V=V_FULL, dtype="bf16", K=8, cap=512, t_draft=1.0,
                 cost="c1", mask="u8", recipe="peak", seed=SEED_BASE + 2),
    "c3": Config("c3", B=256, L=16, V=V_FULL, dtype="bf16", K=16, cap=1024, t_draft=1.0,
                 cost="c3", mask="bits", recipe="peak_temp", seed=SEED_BASE + 3),
    "c4": Config("c4", B=256, L=32, V=V_FULL, dtype="f32", K=16, cap=4096, t_draft=1.0,
                 cost="c4", mask="bits", recipe="peak", seed=SEED_BASE + 4),
}

# Ungraded stress workloads: constant cost (always grows to the cap) and a
# low-temperature regime that gives deep trees of a few hundred nodes.
STRESS: Dict[str, Config] = {
    "s1": Config("s1", B=256, L=32, V=V_FULL, dtype="f32", K=16, cap=4096, t_draft=1.0,
                 cost="const", mask="bits", recipe="peak", seed=SEED_BASE + 11),
    "s2": Config("s2", B=256, L=32, V=V_FULL, dtype="f32", K=16, cap=4096, t_draft=1.0,
                 cost="c4", mask="bits", recipe="peak_cold", seed=SEED_BASE + 12),
}


# Context grid of the cost profile (Sec. 4.6: 0, 1k, .., 8k tokens).
CTX_GRID = tuple(1000 * j for j in range(9))


def _ctx9(j: int, n: np.ndarray) -> np.ndarray:
    # the base cost and the marginal cost per node both grow with the context
    # (what Sec. 5.3 reports of the measured profiles); convex in n at every j
    return (1.0 + 0.05 * j) + (0.002 + 0.0005 * j) * n + (0.00002 + 0.000002 * j) * n * n


def ctx_tables(cfg: Config):
    """(grid [J] int64, tables [J, cap + 1] float64) of a context-aware workload."""
    if cfg.ctx != "ctx9":
        raise KeyError(f"workload {cfg.name} has no context-cost recipe")
    n = np.arange(cfg.cap + 1, dtype=np.float64)
    return np.array(CTX_GRID, dtype=np.int64), np.stack([_ctx9(j, n) for j in range(len(CTX_GRID))])


def ctx_lengths(cfg: Config, B: int) -> np.ndarray:
    """Context length of each round, int64 [B]: uniform on [-500, 9500] (so both ends of the grid are
    passed), with every 7th round placed exactly on a grid point."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed, spawn_key=(1 << 30,))))
    ell = rng.integers(-500, 9501, size=B).astype(np.int64)
    on = np.arange(B) % 7 == 0
    ell[on] = np.array(CTX_GRID, dtype=np.int64)[(np.arange(B)[on] // 7) % len(CTX_GRID)]
    return ell


def cost_profiles(cfg: Config, N: int = 1024, noise: float = 0.01):
    """Synthetic verification-cost measurements for the offline fit (Sec. 4.6): node counts 1 .. N and, per
    point of the context grid, the workload's context table at those counts times (1 + noise * z),
    z ~ N(0, 1).  Returns (n [N] float64, profiles [J, N] float64)."""
    grid, tables = ctx_tables(cfg.replace(cap=N))
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed, spawn_key=(1 << 28,))))
    n = np.arange(1, N + 1, dtype=np.float64)
    prof = tables[:, 1:] * (1.0 + noise * rng.standard_normal((len(grid), N)))
    return n, prof


def accept_uniforms(cfg: Config, B: int, draw: int = 0) -> np.ndarray:
    """Uniforms in [0, 1), float64 [B, L], for drawing target paths in the acceptance simulation; ``draw``
    selects an independent stream (a redraw, or another sample of the same rounds)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed, spawn_key=(1 << 29, draw))))
    return rng.random((B, cfg.L))


# Variants: c1 / c2 shapes with the context-aware cost, and the fixed-budget
# (DDTree) construction at budgets from its grid {16, .., 1024} (Sec. 5.1).
VARIANTS: Dict[str, Config] = {
    "c1x": CONFIGS["c1"].replace(name="c1x", ctx="ctx9", seed=SEED_BASE + 21),
    "c2x": CONFIGS["c2"].replace(name="c2x", ctx="ctx9", seed=SEED_BASE + 22),
    "c1f16": CONFIGS["c1"].replace(name="c1f16", cap=16, fixed=True, seed=SEED_BASE + 31),
    "c1f128": CONFIGS["c1"].replace(name="c1f128", cap=128, fixed=True, seed=SEED_BASE + 32),
    "c1f1024": CONFIGS["c1"].replace(name="c1f1024", cap=1024, fixed=True, seed=SEED_BASE + 33),
    "c2f128": CONFIGS["c2"].replace(name="c2f128", cap=128, fixed=True, seed=SEED_BASE + 34),
    "c2f1024": CONFIGS["c2"].replace(name="c2f1024", cap=1024, fixed=True, seed=SEED_BASE + 35),
}


def get_config(name: str) -> Config:
    name = name.lower()
    for table in (CONFIGS, STRESS, VARIANTS):
        if name in table:
            return table[name]
    raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS) + sorted(STRESS) + sorted(VARIANTS)}")
