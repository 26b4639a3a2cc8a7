"""Seeded synthetic workloads for the CaDDTree hot path.

This module holds input recipes only: drafter logits with the shapes and value
distributions of the benchmark configurations, and the verification-cost tables
those configurations define.  It computes no part of the tree construction
(no normaliser, no top-K, no expansion, no stop rule): the GPU library and the
CPU oracle both receive these arrays as plain inputs.

Every round is generated from its own seed, ``SeedSequence(seed, spawn_key=(b,
attempt))`` with the PCG64 bit generator, so any single round of a batch can be
regenerated on its own and a round can be redrawn (``attempt + 1``) without
touching the others.

bf16 logits are carried as ``uint16`` bit patterns (round-to-nearest-even from
fp32); fp32 logits as ``float32``.
"""

from .configs import (CONFIGS, STRESS, VARIANTS, Config, accept_uniforms, cost_profiles, cost_table, ctx_lengths,
                      ctx_tables, get_config)
from .gen import draw_round, draw_batch, bf16_bits_from_f32

__all__ = [
    "CONFIGS", "STRESS", "VARIANTS", "Config", "get_config", "cost_table", "ctx_tables", "ctx_lengths",
    "accept_uniforms", "cost_profiles",
    "draw_round", "draw_batch", "bf16_bits_from_f32",
]
