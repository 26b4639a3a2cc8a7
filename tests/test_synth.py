"""Input generators: shapes, dtypes, determinism, per-round independence, bf16 rounding."""

import numpy as np
import pytest

import synth
from synth.gen import draw_round, draw_batch, bf16_bits_from_f32


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, 1.0078125 + 2 ** -9, -2.0, 3.0e38, 1e-40], dtype=np.float32)
    got = bf16_bits_from_f32(x)
    # 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 is a tie -> even (1 + 2^-6 = 0x3F82)
    assert got[0] == 0x3F80 and got[1] == 0x3F80 and got[2] == 0x3F82
    assert got[3] == 0x3F81
    assert got[4] == 0xC000
    assert got[5] == 0x7F62          # 3.0e38 rounds to 0x7F62 (3.0030e38)
    assert got[6] == 0x0000 or got[6] == 0x0001


def test_shapes_and_dtypes():
    for name in ("c0", "c1", "c3", "c4"):
        cfg = synth.get_config(name)
        small = cfg.replace(V=min(cfg.V, 2048))
        x = draw_round(small, 0)
        assert x.shape == (cfg.L, small.V)
        assert x.dtype == (np.uint16 if cfg.dtype == "bf16" else np.float32)


def test_determinism_and_independence():
    cfg = synth.get_config("c1").replace(V=4096, B=6)
    a = draw_batch(cfg)
    b = draw_batch(cfg, rounds=[3, 1])
    assert np.array_equal(a[3], b[0]) and np.array_equal(a[1], b[1])
    c = draw_batch(cfg, attempts={2: 1})
    assert np.array_equal(a[0], c[0]) and not np.array_equal(a[2], c[2])


def test_pool_matches_serial():
    cfg = synth.get_config("c3").replace(V=3000, B=7)
    serial = draw_batch(cfg, workers=1)
    pooled = draw_batch(cfg, workers=3)
    assert np.array_equal(serial, pooled)


def test_peak_recipe_shape_of_distribution():
    cfg = synth.get_config("c1").replace(V=20000)
    x = draw_round(cfg, 5)
    f = (x.astype(np.uint32) << 16).view(np.float32)
    # Gumbel(0,1) noise: mean ~0.577; one boosted peak per position, boost decays with depth
    assert abs(float(np.median(f)) - 0.3665) < 0.05
    assert np.isfinite(f).all()


def test_cost_tables():
    c3 = synth.cost_table("c3", 1024)
    assert c3[0] == 1.0 and c3[64] == 1.0
    assert abs(c3[256] - 1.768) < 1e-12 and abs(c3[1024] - (1.768 + 0.012 * 768)) < 1e-9
    d = np.diff(c3)
    assert np.all(np.diff(d) >= -1e-12)     # convex up to rounding
    c1 = synth.cost_table(synth.get_config("c1"))
    assert len(c1) == 513 and c1[10] == 1.0 + 0.002 * 10 + 0.00002 * 100
    for f in (16, 32, 128, 200):
        t = synth.cost_table(f"flat{f}", 700)
        assert np.all(t[:f + 1] == 1.0) and t[f + 1] > 1.0      # flat up to f, rising after
        assert np.all(np.diff(np.diff(t)) >= -1e-12)            # convex up to rounding


@pytest.mark.parametrize("name", ["c0", "c1", "c2", "c3", "c4"])
def test_config_table(name):
    cfg = synth.get_config(name)
    assert cfg.K <= 16 and cfg.L <= 32 and cfg.cap <= 4096 and cfg.K <= cfg.V


def test_ctx_lengths_prefix_stable():
    """A smaller batch of a context-aware workload sees the same context lengths as the full batch."""
    cfg = synth.get_config("c1x")
    full = synth.ctx_lengths(cfg, cfg.B)
    assert np.array_equal(synth.ctx_lengths(cfg, 21), full[:21])
    grid, tables = synth.ctx_tables(cfg)
    assert tables.shape == (len(grid), cfg.cap + 1)
    assert np.all(np.diff(tables, axis=1) > 0) and np.all(np.diff(tables, 2, axis=1) > 0)
