"""caddtree_build_noalloc (the entry point for callers that cannot allocate) against caddtree_build.

The same kernels run with the top-K table in the library's own device array instead of the
caller's workspace, so every output must be bit-identical to caddtree_build's on the same
inputs: two calls in a row, the second with a smaller batch, then a call on another plan,
and the size limit of the array.
"""

import numpy as np
import pytest

import synth
from paper_2606_01813_amd import CaddtreeError, _lib
from tests._parity import host, make_plan, say, torch_logits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    _lib.lib()
    return torch


def _both(plan, lg, pos_offset=0):
    import torch
    B = lg.shape[0]
    ref = plan.new_outputs(B)
    plan.build(lg, ref, pos_offset=pos_offset, workspace=plan.new_workspace(B))
    got = plan.new_outputs(B)
    plan.build_noalloc(lg, got, pos_offset=pos_offset)
    torch.cuda.synchronize()
    return host(ref), host(got)


def _same(ref, got, what):
    for k, v in ref.items():
        if v is None:
            assert got[k] is None, (what, k)
            continue
        assert np.array_equal(v, got[k]), f"{what}: {k} differs from caddtree_build"


def test_noalloc_matches_build_twice_then_smaller():
    cfg = synth.get_config("c1")                     # 64 rounds x 16 x 151936 bf16, K = 8, cap 512
    plan = make_plan(cfg)
    xs = synth.draw_batch(cfg, workers=synth.gen.default_workers())
    say(f"[noalloc] c1 full batch: {cfg.B} rounds")
    ref, got = _both(plan, torch_logits(cfg, xs), pos_offset=2)
    _same(ref, got, "c1, 64 rounds")
    # a smaller batch of other rounds: the array keeps the first call's table, which must not leak in
    small = synth.draw_batch(cfg, rounds=range(100, 120))
    say("[noalloc] second call: 20 other rounds")
    ref2, got2 = _both(plan, torch_logits(cfg, small))
    _same(ref2, got2, "c1, 20 rounds")
    assert ref2["n_star"].min() > 0


def test_noalloc_on_another_plan():
    cfg = synth.get_config("c4").replace(V=3000, B=12)     # L = 32, K = 16, fp32, packed mask
    plan = make_plan(cfg)
    say("[noalloc] c4-shaped plan, 12 rounds of V = 3000")
    ref, got = _both(plan, torch_logits(cfg, synth.draw_batch(cfg)))
    _same(ref, got, "c4 shape")


def test_noalloc_on_a_wide_kernel_plan():
    cfg = synth.get_config("s1").replace(V=2000, B=6)      # cost flat to cap 4096: 16 wavefronts per round
    plan = make_plan(cfg)
    say("[noalloc] s1-shaped plan, 6 rounds of V = 2000")
    ref, got = _both(plan, torch_logits(cfg, synth.draw_batch(cfg)))
    _same(ref, got, "s1 shape")
    assert ref["n_star"].min() == cfg.cap


def test_noalloc_limit():
    import torch
    cfg = synth.get_config("c1").replace(V=16, cap=8)
    plan = make_plan(cfg)
    per_round = plan.workspace_bytes(1)
    fit = max(b for b in range(7000, 7400) if plan.workspace_bytes(b) <= _lib.NOALLOC_SCRATCH_BYTES)
    assert fit == 7281, (fit, per_round)
    lg = torch.randn((fit + 1, cfg.L, cfg.V), device="cuda", dtype=torch.float32).to(torch.bfloat16)
    say(f"[noalloc] limit: {fit} rounds fit, {fit + 1} do not")
    out = plan.new_outputs(fit + 1)
    with pytest.raises(CaddtreeError) as e:
        plan.build_noalloc(lg, out)
    assert e.value.status == _lib.E_WORKSPACE
    torch.cuda.synchronize()
    assert int(out.n_star.max()) == -1                  # nothing was enqueued
    ref, got = _both(plan, lg[:fit])
    _same(ref, got, f"{fit} rounds")
    # with the top-K table passed in, the array is not used and the batch may be larger
    full = plan.new_outputs(fit + 1, topk=True)
    plan.build_noalloc(lg, full)
    ref_full = plan.new_outputs(fit + 1, topk=True)
    plan.build(lg, ref_full)
    torch.cuda.synchronize()
    _same(host(ref_full), host(full), f"{fit + 1} rounds with the top-K table passed in")
