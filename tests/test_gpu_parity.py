"""GPU parity: the HIP library against the oracle, element by element, on seeded inputs.

Small cases (several tiles, ragged tails, every dtype / mask / special case) and
the full-size workloads (run in the launch configuration the benchmark times)
are compared element by element on every round; only a 70,000-round grid test is
compared on a sample.
Properties that hold at any size are checked on every round.  Rounds are drawn
through the input guard (tests/_guard.py), so every floating-point decision of a
compared round keeps a margin of at least 1e-6, more for deep trees.
"""

import numpy as np
import pytest

import synth
from tests import _fullbatch, _guard
from tests._parity import (check_tree_properties, compare_topk, compare_tree, ctx_tensor, host, make_plan,
                           run_build, say, torch_logits)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2606_01813_amd._lib as L
    L.lib()  # the HIP library must be built and loadable: no fallback
    return torch


def _parity_batch(cfg, rounds, pos_offset=0, pad=0, mask=None):
    attempts, x, rs = _guard.guarded_batch(cfg, rounds, pos_offset=pos_offset)
    say(f"[parity] {cfg.name} L={cfg.L} V={cfg.V} K={cfg.K} cap={cfg.cap} {cfg.dtype} mask={mask or cfg.mask} "
        f"rounds={len(rounds)} pad={pad} redraws={sum(attempts.values())}")
    plan = make_plan(cfg, mask=mask)
    out = run_build(plan, torch_logits(cfg, x, pad=pad), pos_offset=pos_offset, ctx_len=ctx_tensor(cfg, rounds))
    h = host(out)
    worst = compare_topk(h, rs)
    if (mask or cfg.mask) == cfg.mask:
        compare_tree(h, rs, mask or cfg.mask, cfg.cap, pos_offset=pos_offset)
    say(f"[parity]   ok; max |lse - oracle| = {worst:.2e}; n* = {[r.n_star for r in rs][:12]}")
    return h, rs


SMALL = [
    # name, overrides
    ("c0", dict()),
    ("c0", dict(B=48)),
    ("c0", dict(V=1000, L=3, K=3, cap=40, B=16)),                       # ragged tail, short rows
    ("c0", dict(V=17, L=2, K=2, cap=10, B=16)),                         # V below one wave chunk
    ("c0", dict(V=4099, L=5, K=5, cap=64, B=8, dtype="bf16", mask="bits")),
    ("c1", dict(V=20000, B=8)),                                         # full L=16, K=8, cap 512
    ("c1", dict(V=2500, B=8, L=7, K=16, mask="bits")),
    ("c3", dict(V=30011, B=6)),                                         # temperature mix, packed mask
    ("c4", dict(V=3000, B=4)),                                          # L=32, K=16, cap 4096, fp32
    ("c4", dict(V=64, B=4, K=16, L=32)),                                # V = one fp32 chunk
    ("c0", dict(V=5, K=5, L=3, cap=200, B=6)),                          # every token in the top-K
    ("c1", dict(V=16, K=16, L=4, cap=600, B=4, cost="tiny")),           # the same in bf16, trees past 512
    ("c1", dict(V=262144, L=4, B=2)),                                   # a larger vocabulary, whole chunks only
    ("c4", dict(V=131072, L=3, B=2)),                                   # the same in fp32
]


@pytest.mark.parametrize("i", range(len(SMALL)))
def test_small_parity(i):
    name, kw = SMALL[i]
    cfg = synth.get_config(name).replace(**kw)
    _parity_batch(cfg, list(range(cfg.B)), pos_offset=3 * i)


def test_unaligned_rows_use_the_guarded_path():
    cfg = synth.get_config("c1").replace(V=3001, B=4)
    _parity_batch(cfg, list(range(cfg.B)), pad=1)        # row stride V + 1: rows off 16-byte boundaries
    cfg32 = synth.get_config("c0").replace(V=999, B=4)
    _parity_batch(cfg32, list(range(cfg32.B)), pad=3)


def test_dense_and_packed_masks_agree():
    cfg = synth.get_config("c1").replace(V=5000, B=4)
    h8, rs = _parity_batch(cfg, list(range(4)), mask="u8")
    hb, _ = _parity_batch(cfg, list(range(4)), mask="bits")
    for i, r in enumerate(rs):
        n = r.n_star
        words = hb["mask"][i, :n, :(n + 31) // 32].view(np.uint32)
        unpacked = np.array([[(words[a, c // 32] >> (c % 32)) & 1 for c in range(n)] for a in range(n)])
        assert np.array_equal(unpacked, h8["mask"][i, :n, :n])


# ------------------------------------------------------------- stage-by-stage

def _oracle_tables(cfg, rs):
    import torch
    ids = torch.tensor(np.stack([r.marg["ids"] for r in rs]).astype(np.int32), device="cuda")
    logit = torch.tensor(np.stack([r.marg["logit"] for r in rs]).astype(np.float32), device="cuda")
    lse = torch.tensor(np.stack([r.marg["lse"] for r in rs]), dtype=torch.float64, device="cuda")
    return ids, logit, lse


@pytest.mark.parametrize("name,kw", [
    ("c0", dict(B=32)),
    ("c1", dict(V=4000, B=8)),
    ("c3", dict(V=4000, B=8)),
    ("s1", dict(V=1500, B=2)),                         # constant cost: grows to the 4096 cap
    ("s2", dict(V=1500, B=3)),                         # cold marginals: deep trees
    ("c4", dict(V=800, B=4, cost="const", cap=700)),   # heap sizes far past the LDS fast cases
    ("c4", dict(V=900, B=3, cost="tiny", cap=1500)),   # rising cost, trees too large for the batched kernel:
                                                       # the serial form runs in place (its LDS fits)
    ("c4", dict(V=900, B=2, cost="tiny", cap=4096)),   # the same with a 4096 cap: flagged for the serial kernel
])
def test_expand_stage_on_oracle_inputs(name, kw):
    """Algorithm 1 alone, fed the oracle's own top-K table and fp64 normalisers: no guard needed."""
    import torch
    cfg = synth.get_config(name).replace(**kw)
    xs = synth.draw_batch(cfg)
    rs = [_guard.oracle_round(cfg, xs[b]) for b in range(cfg.B)]
    say(f"[expand] {cfg.name} L={cfg.L} K={cfg.K} cap={cfg.cap} n*={[r.n_star for r in rs]}")
    plan = make_plan(cfg)
    out = plan.new_outputs(cfg.B)
    ids, logit, lse = _oracle_tables(cfg, rs)
    plan.expand(ids, logit, lse, out)
    plan.emit(out, pos_offset=0)
    torch.cuda.synchronize()
    h = host(out)
    compare_tree(h, rs, cfg.mask, cfg.cap, prob_rtol=1e-6)
    for i, r in enumerate(rs):
        assert np.array_equal(h["path_prob"][i, :r.n_star], r.tree.path_prob.astype(np.float32))


@pytest.mark.parametrize("name,kw", [
    ("c1", dict(V=3000, B=16)),
    ("c4", dict(V=1200, B=6)),
    ("s2", dict(V=1000, B=4)),
    ("c4", dict(V=900, B=2, cost="tiny", cap=1200)),
    ("s1", dict(V=1000, B=3)),                  # constant cost, trees of 4096 nodes
])
def test_expand_paths_agree(name, kw, monkeypatch):
    """The batched expansion and the serial one give bit-identical trees."""
    import torch
    cfg = synth.get_config(name).replace(**kw)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    outs = {}
    for mode in ("auto", "serial"):
        if mode == "serial":
            monkeypatch.setenv("CADDTREE_EXPAND", "serial")
        else:
            monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
        plan = make_plan(cfg)
        outs[mode] = host(run_build(plan, lg))
    say(f"[paths] {cfg.name} n*={outs['auto']['n_star'].tolist()[:8]}")
    _paths_agree(outs)


@pytest.mark.parametrize("kw", [
    dict(cost="c4", cap=400),                # convex cost
    dict(cost="c3", cap=400),                # flat start: 65 nodes kept before any cost
    dict(cost="tiny", cap=600),              # almost flat: trees of hundreds of nodes
    dict(cost="c4", cap=150, fixed=True),    # fixed budget
])
def test_expand_paths_agree_on_ties(kw, monkeypatch):
    """Logits on a 0.5 grid, one boosted token per position: many nodes tie on sigma (and on
    Lambda), so the batched kernel's sigma-order selection, its cut tie groups and its in-place
    threshold raises all run; its trees must equal the serial kernel's."""
    import torch
    cfg = synth.get_config("c4").replace(V=1500, B=96, L=8, K=16, **kw)
    rng = np.random.default_rng(11)
    x = np.round(rng.standard_normal((cfg.B, cfg.L, cfg.V)) * 2.0) / 2.0
    peak = rng.integers(0, cfg.V, size=(cfg.B, cfg.L))
    x[np.arange(cfg.B)[:, None], np.arange(cfg.L)[None, :], peak] += rng.choice([0.0, 3.0, 6.0], size=(cfg.B, cfg.L))
    lg = torch_logits(cfg, x.astype(np.float32))
    outs = {}
    for mode in ("auto", "serial"):
        if mode == "serial":
            monkeypatch.setenv("CADDTREE_EXPAND", "serial")
        else:
            monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
        plan = make_plan(cfg)
        outs[mode] = host(run_build(plan, lg))
    n = outs["auto"]["n_star"]
    say(f"[paths ties] {kw} n* mean {n.mean():.1f} min {n.min()} max {n.max()}")
    _paths_agree(outs)


def _paths_agree(outs):
    """The two expansion kernels give the same trees; Phi (and theta from it) may differ by the
    rounding of the summation order, far below the fp32 output precision."""
    for k, v in outs["auto"].items():
        if v is None:
            continue
        if k in ("phi", "theta"):
            np.testing.assert_allclose(v, outs["serial"][k], rtol=1e-6, err_msg=k)
        else:
            assert np.array_equal(v, outs["serial"][k]), k


@pytest.mark.parametrize("name,kw", [
    ("c1", dict(V=4000, B=8)),                           # dense mask, batched expansion
    ("c1", dict(V=4000, B=8, mask="bits", L=9)),
    ("c3", dict(V=4000, B=6)),                           # packed mask, flat start (n* >= 64: two row tiles)
    ("s2", dict(V=1500, B=3)),                           # deep trees of 100-200 nodes
    ("c4", dict(V=900, B=3, cost="tiny", cap=1500)),     # the serial form in place, trees past 64 rows
    ("c4", dict(V=900, B=2, cost="tiny", cap=4096)),     # rounds flagged for the serial kernel
    ("c0", dict(B=24, cap=7)),                           # cap below one mask word; trees cut by the cap
])
def test_fused_emit_matches_emit_kernel(name, kw, monkeypatch):
    """caddtree_build's expansion epilogue writes the mask and position ids itself; they equal the
    emission kernel's bit for bit (and the oracle's, on the guarded rounds)."""
    cfg = synth.get_config(name).replace(**kw)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    outs = {}
    for mode in ("fused", "separate"):
        if mode == "separate":
            monkeypatch.setenv("CADDTREE_EMIT", "separate")
        plan = make_plan(cfg)
        outs[mode] = host(run_build(plan, lg, pos_offset=5))
        plan.close()
    a, b = outs["fused"], outs["separate"]
    say(f"[emit] {cfg.name} L={cfg.L} K={cfg.K} cap={cfg.cap} mask={cfg.mask} n*={a['n_star'].tolist()[:8]}")
    assert a["n_star"].max() > 0
    for k in ("n_star", "token_ids", "parent", "depth", "pos_ids", "mask", "path_prob", "phi", "theta"):
        assert np.array_equal(a[k], b[k]), f"{k} differs between the fused and the separate emission"


def test_emit_stage_on_oracle_trees():
    import torch
    cfg = synth.get_config("s2").replace(V=1200, B=3)
    xs = synth.draw_batch(cfg)
    rs = [_guard.oracle_round(cfg, xs[b], pos_offset=11) for b in range(cfg.B)]
    for mask in ("u8", "bits"):
        plan = make_plan(cfg, mask=mask)
        out = plan.new_outputs(cfg.B)
        for i, r in enumerate(rs):
            n = r.n_star
            out.parent[i, :n] = torch.tensor(r.tree.parent, dtype=torch.int32)
            out.depth[i, :n] = torch.tensor(r.tree.depth, dtype=torch.int32)
            out.n_star[i] = n
        say(f"[emit] mask={mask} n*={[r.n_star for r in rs]}")
        plan.emit(out, pos_offset=11)
        torch.cuda.synchronize()
        h = host(out)
        for i, r in enumerate(rs):
            n = r.n_star
            assert np.array_equal(h["pos_ids"][i, :n], r.tree.pos_ids)
            ref = _guard.oracle.emit_mask(r.tree.parent, mask, cfg.cap)
            if mask == "u8":
                assert np.array_equal(h["mask"][i, :n, :n], ref)
            else:
                w = (n + 31) // 32
                assert np.array_equal(h["mask"][i, :n, :w].view(np.uint32), ref[:, :w])


# ------------------------------------------------------------- special cases

def test_special_costs():
    import torch
    base = synth.get_config("c1").replace(V=3000, B=4, cap=64)
    xs = synth.draw_batch(base)
    lg = torch_logits(base, xs)
    cases = {
        "steep": (1.0 + 1e6 * np.arange(65.0), lambda n: n == 0),
        "constant": (np.ones(65), lambda n: n == 64),
    }
    for name, (tv, expect) in cases.items():
        plan = make_plan(base, t_verify=tv)
        out = run_build(plan, lg)
        h = host(out)
        say(f"[special] {name} n*={h['n_star'].tolist()}")
        assert all(expect(int(n)) for n in h["n_star"])
        for i in range(base.B):
            r = _guard.oracle.build_round(xs[i], base.dtype, base.K, base.t_draft, tv, base.cap, mask=base.mask)
            compare_tree(h, [r], base.mask, base.cap, rounds=[i])


def test_cap_zero_and_empty_batch():
    import torch
    cfg = synth.get_config("c0").replace(cap=0, B=2)
    plan = make_plan(cfg)
    xs = synth.draw_batch(cfg)
    out = run_build(plan, torch_logits(cfg, xs))
    assert out.n_star.cpu().tolist() == [0, 0]
    th = out.theta.cpu().numpy()
    assert np.allclose(th, 1.0 / (1.0 + synth.cost_table(cfg)[0]))
    empty = torch.zeros((0, cfg.L, cfg.V), dtype=torch.float32, device="cuda")
    out0 = plan.new_outputs(0)
    plan.build(empty, out0, workspace=None)
    torch.cuda.synchronize()


def test_k1_chain_and_l1():
    cfg = synth.get_config("c0").replace(K=1, cap=16, B=6, V=700)
    _parity_batch(cfg, list(range(cfg.B)))
    cfg = synth.get_config("c0").replace(L=1, K=16, cap=16, B=6, V=5000)
    _parity_batch(cfg, list(range(cfg.B)))


def test_bf16_ties():
    """Heavily tied bf16 logits: top-K and expansion tie-breaks must match exactly."""
    import torch
    cfg = synth.get_config("c1").replace(V=6000, B=4, L=4, K=16, cap=200)
    rng = np.random.default_rng(7)
    x32 = (np.round(rng.standard_normal((cfg.B, cfg.L, cfg.V)) * 2) / 2).astype(np.float32)
    xs = synth.bf16_bits_from_f32(x32)
    rs = [_guard.oracle_round(cfg, xs[b]) for b in range(cfg.B)]
    plan = make_plan(cfg)
    out = run_build(plan, torch_logits(cfg, xs))
    h = host(out)
    compare_topk(h, rs)
    # expansion on the oracle's normalisers is exact even with equal-probability nodes
    out2 = plan.new_outputs(cfg.B)
    ids, logit, lse = _oracle_tables(cfg, rs)
    plan.expand(ids, logit, lse, out2)
    plan.emit(out2)
    torch.cuda.synchronize()
    compare_tree(host(out2), rs, cfg.mask, cfg.cap)


@pytest.mark.parametrize("waves", [1, 4, 16])
def test_k1_signed_zero_ties(waves, monkeypatch):
    """Rows whose K-th largest logit is a zero shared by +0 and -0 entries: the two compare equal, so the
    ids decide, in every wavefront's list and in the merge of the lists."""
    import oracle
    import torch
    monkeypatch.setenv("CADDTREE_K1_WAVES", str(waves))
    for dtype in ("f32", "bf16"):
        cfg = synth.get_config("c1").replace(V=9000, B=3, L=4, K=8, dtype=dtype)
        rng = np.random.default_rng(11)
        x32 = (-1.0 - rng.random((cfg.B, cfg.L, cfg.V))).astype(np.float32)   # all below -1
        for b in range(cfg.B):
            for i in range(cfg.L):
                top = rng.choice(cfg.V, 3, replace=False)
                x32[b, i, top] = 1.0 + rng.random(3).astype(np.float32)           # three above 0
                zeros = rng.choice(np.setdiff1d(np.arange(cfg.V), top), 12, replace=False)
                x32[b, i, zeros[:6]] = 0.0
                x32[b, i, zeros[6:]] = -0.0                                      # twelve zeros of both signs
        xs = synth.bf16_bits_from_f32(x32) if dtype == "bf16" else x32
        plan = make_plan(cfg)
        out = plan.new_outputs(cfg.B, topk=True)
        plan.reduce_topk(torch_logits(cfg, xs), out.topk_ids, out.topk_logit, out.lse, out.topk_lq)
        torch.cuda.synchronize()
        h = host(out)
        for b in range(cfg.B):
            m = oracle.marginals(xs[b], dtype, cfg.K)
            assert np.array_equal(h["topk_ids"][b], m["ids"]), (dtype, b)
            assert np.array_equal(h["topk_logit"][b].astype(np.float64), m["logit"]), (dtype, b)
            assert np.abs(h["lse"][b] - m["lse"]).max() <= 1e-7


def test_determinism():
    cfg = synth.get_config("c1").replace(V=40000, B=12)
    xs = synth.draw_batch(cfg)
    plan = make_plan(cfg)
    lg = torch_logits(cfg, xs)
    a = host(run_build(plan, lg))
    b = host(run_build(plan, lg))
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k]), k


# ------------------------------------------------------------- process set-up

def test_plan_before_torch_in_a_fresh_process():
    """PyTorch-ROCm bundles its own HIP runtime under the soname the library links; the binding
    imports torch before loading the library so that both use that one runtime.  A fresh process
    that creates a plan first and touches torch afterwards must still see the GPU and build."""
    import os
    import subprocess
    import sys
    import textwrap
    code = textwrap.dedent('''
        import numpy as np
        from paper_2606_01813_amd import Plan
        plan = Plan(L=4, V=1024, K=4, cap=32, t_draft=1.0, t_verify=1.0 + 0.01 * np.arange(33), dtype="f32")
        import torch
        assert torch.cuda.is_available(), "torch lost the GPU"
        x = torch.randn(2, 4, 1024, device="cuda")
        out = plan.new_outputs(2)
        plan.build(x, out, workspace=plan.new_workspace(2))
        torch.cuda.synchronize()
        n = out.n_star.tolist()
        assert all(1 <= v <= 32 for v in n), n
        print("n_star", n)
    ''')
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    say(f"[process] {r.stdout.strip()}")
    assert r.returncode == 0, r.stderr[-3000:]


# ------------------------------------------------------------- degenerate logits

@pytest.mark.parametrize("kw", [
    dict(cost="const", cap=100, fixed=False),   # grows to the cap through a tie group of 256
    dict(cost="c4", cap=100, fixed=True),       # fixed budget through the same ties
    dict(cost="const", cap=340, fixed=False),   # the whole tree (4 + 16 + 64 + 256 nodes)
    # a flat start to 64 whose first set (16 + 256 nodes) passes the early-raise limit, where no
    # threshold keeps between 65 and 89 nodes: the raise fails, the limit is dropped, and the stop
    # cuts the tie group of depth 2 at 64
    dict(cost="c3", cap=300, fixed=False, K=16, V=20),
])
def test_constant_logits(kw):
    """Every logit equal: all nodes of a depth tie on sigma and Lambda, so the pop order inside a
    depth is the rank tuple alone, and the cap (or the stop) cuts a group of equal nodes.  No
    decision depends on the normaliser's rounding (depths differ by ln V in sigma; a flat cost or a
    fixed budget never stops before the cap, and the flat start's stop after 64 nodes has a margin
    of about one half), so the oracle's tree is compared without the input guard."""
    shape = dict(B=3, L=4, V=1000, K=4, dtype="f32", mask="bits")
    shape.update(kw)
    cfg = synth.get_config("c0").replace(**shape)
    x = np.zeros((cfg.B, cfg.L, cfg.V), dtype=np.float32)
    x[1] += 2.5                                   # a constant shift changes nothing
    x[2] -= 7.0
    rs = [_guard.oracle_round(cfg, x[b], b=b) for b in range(cfg.B)]
    plan = make_plan(cfg)
    h = host(run_build(plan, torch_logits(cfg, x)))
    compare_topk(h, rs)
    compare_tree(h, rs, cfg.mask, cfg.cap)
    say(f"[constant] {kw}: n* {[r.n_star for r in rs]}")


def test_certain_tokens():
    """One token per position 100 nats above the rest: its log q rounds to 0, so the chain of those
    tokens has sigma = 0 at every depth (the clamp of the prefix probability) and the chain pops in
    depth order.  The stage gets the oracle's own tables (exact); the whole path, whose normaliser
    may differ from the oracle's by a few ulps, must give the same tree."""
    import torch
    cfg = synth.get_config("c1").replace(B=4, V=3000, dtype="f32", mask="u8")
    rng = np.random.default_rng(9)
    x = (rng.standard_normal((cfg.B, cfg.L, cfg.V)) * 0.5).astype(np.float32)
    peak = rng.integers(0, cfg.V, size=(cfg.B, cfg.L))
    x[np.arange(cfg.B)[:, None], np.arange(cfg.L)[None, :], peak] = 100.0
    rs = [_guard.oracle_round(cfg, x[b], b=b) for b in range(cfg.B)]
    for r in rs:
        assert r.n_star >= cfg.L and np.all(r.tree.depth[:cfg.L] == np.arange(1, cfg.L + 1))
    plan = make_plan(cfg)
    out = plan.new_outputs(cfg.B)
    ids, logit, lse = _oracle_tables(cfg, rs)
    plan.expand(ids, logit, lse, out)
    plan.emit(out, pos_offset=0)
    torch.cuda.synchronize()
    compare_tree(host(out), rs, cfg.mask, cfg.cap, prob_rtol=1e-6)
    h = host(run_build(plan, torch_logits(cfg, x)))
    compare_tree(h, rs, cfg.mask, cfg.cap)
    say(f"[certain] n* {[r.n_star for r in rs]}")


# ------------------------------------------------------------- optional outputs

def test_workspace_topk_and_no_mask():
    """Without top-K outputs the table lives in the workspace, and a plan may emit no mask: the
    tree is the same as with every output requested."""
    cfg = synth.get_config("c3").replace(V=7000, B=6)
    lg = torch_logits(cfg, synth.draw_batch(cfg))
    full = host(run_build(make_plan(cfg), lg, topk=True))
    bare = host(run_build(make_plan(cfg, mask="none"), lg, topk=False))
    assert bare["mask"] is None and bare["topk_ids"] is None
    assert np.array_equal(bare["n_star"], full["n_star"])
    for i, n in enumerate(full["n_star"]):
        for k in ("token_ids", "parent", "depth", "pos_ids", "path_prob"):
            assert np.array_equal(bare[k][i, :n], full[k][i, :n]), f"round {i} {k}"
    assert np.array_equal(bare["phi"], full["phi"]) and np.array_equal(bare["theta"], full["theta"])


# ------------------------------------------------------------- concurrency

def test_concurrent_builds_on_two_streams():
    """One plan, two host threads, each building on its own stream into its own outputs and
    workspace, with no synchronisation between them: every result equals the build done alone
    (a plan is immutable; the last-error string is per thread)."""
    import threading
    import torch
    cfg = synth.get_config("c1").replace(V=6000, B=6)
    plan = make_plan(cfg)
    inputs = [torch_logits(cfg, synth.draw_batch(cfg.replace(seed=cfg.seed + k))) for k in range(2)]
    refs = [host(run_build(plan, lg)) for lg in inputs]
    outs = [plan.new_outputs(cfg.B) for _ in range(2)]
    wss = [plan.new_workspace(cfg.B) for _ in range(2)]
    streams = [torch.cuda.Stream() for _ in range(2)]
    torch.cuda.synchronize()
    errors = []

    def worker(k):
        try:
            with torch.cuda.stream(streams[k]):
                for _ in range(20):
                    plan.build(inputs[k], outs[k], workspace=wss[k], stream=streams[k])
        except Exception as e:   # noqa: BLE001 (reported below)
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k in range(2):
        h = host(outs[k])
        assert np.array_equal(h["n_star"], refs[k]["n_star"]), f"stream {k}: n_star"
        for i, n in enumerate(refs[k]["n_star"]):
            for key in ("token_ids", "parent", "depth", "pos_ids"):
                assert np.array_equal(h[key][i, :n], refs[k][key][i, :n]), f"stream {k}: round {i} {key}"
            assert np.array_equal(h["mask"][i, :n, :n], refs[k]["mask"][i, :n, :n]), f"stream {k}: round {i} mask"
    say(f"[streams] two threads x 20 builds: equal to the single builds; n* {refs[0]['n_star'].tolist()} "
        f"{refs[1]['n_star'].tolist()}")


# ------------------------------------------------------------- HIP graph capture

def test_build_under_graph_capture():
    """caddtree_build enqueues kernels only (no allocation, memset or synchronisation), so a caller
    can capture it in a HIP graph; every replay must equal the eager build, with eager work and
    synchronisations between the replays."""
    import torch
    cfg = synth.get_config("c1").replace(V=5000, B=8, mask="bits")
    xs = synth.draw_batch(cfg)
    plan = make_plan(cfg)
    lg = torch_logits(cfg, xs)
    ref = host(run_build(plan, lg))
    out = plan.new_outputs(cfg.B)
    ws = plan.new_workspace(cfg.B)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                # warm-up outside the capture
        plan.build(lg, out, workspace=ws, stream=torch.cuda.current_stream())
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.build(lg, out, workspace=ws, stream=torch.cuda.current_stream())
    for rep in range(3):
        for t in (out.n_star, out.token_ids, out.parent, out.depth, out.mask):
            t.fill_(-9)
        run_build(plan, lg)                      # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        h = host(out)
        assert np.array_equal(h["n_star"], ref["n_star"]), f"replay {rep}: n_star"
        for i, n in enumerate(ref["n_star"]):
            for k in ("token_ids", "parent", "depth", "pos_ids", "path_prob"):
                assert np.array_equal(h[k][i, :n], ref[k][i, :n]), f"replay {rep}: round {i} {k}"
            w = (n + 31) // 32
            assert np.array_equal(h["mask"][i, :n, :w], ref["mask"][i, :n, :w]), f"replay {rep}: round {i} mask"
        say(f"[graph] replay {rep}: equal to the eager build; n* = {h['n_star'].tolist()}")


# ------------------------------------------------------------- seeded random shapes

def random_case(i):
    """A seeded random small workload: any L, K, V, cap, dtype, mask and cost family the plan accepts,
    a fixed budget now and then, padded rows and a position offset."""
    rng = np.random.default_rng(7000 + i)
    base = synth.get_config(("c0", "c1", "c3", "s2")[i % 4])
    K = int(rng.integers(1, 17))
    cfg = base.replace(
        name=f"rand{i}", B=int(rng.integers(1, 7)), L=int(rng.integers(1, 33)), K=K,
        V=int(rng.integers(max(K, 2), 6001)), cap=int(rng.integers(0, 701)),
        dtype=("f32", "bf16")[int(rng.integers(0, 2))], mask=("u8", "bits")[int(rng.integers(0, 2))],
        cost=str(rng.choice(["c0", "c1", "c3", "c4", "const", "tiny"])), fixed=bool(rng.random() < 0.2),
        seed=synth.configs.SEED_BASE + 7000 + i)
    return cfg, int(rng.integers(0, 100)), int(rng.choice([0, 0, 1, 3, 8]))


@pytest.mark.parametrize("i", range(48))
def test_random_shapes(i):
    cfg, pos_offset, pad = random_case(i)
    _parity_batch(cfg, list(range(cfg.B)), pos_offset=pos_offset, pad=pad)


def random_flat_case(i):
    """A seeded random workload with a flat cost start of 16 to 200 nodes (every tree keeps that many
    before any stop test), so the batched expansion's early raise and its restarts run under many
    shapes: any L, K, V, dtype and mask, sharp (deep) or temperature-mixed rows."""
    rng = np.random.default_rng(9300 + i)
    base = synth.get_config(("c3", "s2")[i % 2])
    K = int(rng.integers(2, 17))
    cost = str(rng.choice(["flat16", "flat32", "flat128", "flat200"]))
    flat = int(cost[4:])
    cfg = base.replace(
        name=f"flat{i}", B=int(rng.integers(2, 7)), L=int(rng.integers(3, 33)), K=K,
        V=int(rng.integers(max(K, 64), 6001)), cap=int(rng.integers(flat + 1, 701)),
        dtype=("f32", "bf16")[int(rng.integers(0, 2))], mask=("u8", "bits")[int(rng.integers(0, 2))],
        cost=cost, fixed=False, seed=synth.configs.SEED_BASE + 9300 + i)
    return cfg, int(rng.integers(0, 100))


@pytest.mark.parametrize("i", range(16))
def test_random_flat_starts(i):
    cfg, pos_offset = random_flat_case(i)
    _parity_batch(cfg, list(range(cfg.B)), pos_offset=pos_offset)


def random_wide_case(i):
    """A seeded random workload for the several-wavefront expansion: a fixed budget or a cost flat to
    the cap, of 512 to 1600 nodes, with any L, K, V, dtype and mask."""
    rng = np.random.default_rng(9100 + i)
    K = int(rng.integers(2, 17))
    fixed = bool(rng.random() < 0.5)
    cfg = synth.get_config("c1").replace(
        name=f"wide{i}", B=int(rng.integers(1, 5)), L=int(rng.integers(4, 33)), K=K,
        V=int(rng.integers(max(K, 64), 3001)), cap=int(rng.integers(512, 1601)),
        dtype=("f32", "bf16")[int(rng.integers(0, 2))], mask=("u8", "bits")[int(rng.integers(0, 2))],
        cost="c4" if fixed else "const", fixed=fixed, seed=synth.configs.SEED_BASE + 9100 + i)
    return cfg, int(rng.integers(0, 100)), int(rng.choice([0, 0, 1, 3]))


@pytest.mark.parametrize("i", range(12))
def test_random_wide_shapes(i):
    cfg, pos_offset, pad = random_wide_case(i)
    _parity_batch(cfg, list(range(cfg.B)), pos_offset=pos_offset, pad=pad)


# ------------------------------------------------------------- full-size workloads

def _full_size(name, sample=None, workers=16):
    """One build over the whole batch in the benchmark's launch configuration, compared with the oracle
    element by element on every round (or on ``sample`` only, for the largest trees), with any-size
    properties checked on every round."""
    cfg = synth.get_config(name) if isinstance(name, str) else name
    name = cfg.name
    if sample is None:
        say(f"[full] {name}: B={cfg.B} L={cfg.L} V={cfg.V} {cfg.dtype}; guard + oracle on every round")
        attempts, lg, rs = _fullbatch.guarded_batch(cfg, say=say, consume=lambda x: torch_logits(cfg, x))
        rounds = list(range(cfg.B))
    else:
        attempts, _, rs = _guard.guarded_batch(cfg, sample)
        say(f"[full] {name}: B={cfg.B} L={cfg.L} V={cfg.V} {cfg.dtype}; guarded sample of {len(sample)} rounds")
        xs = synth.draw_batch(cfg, attempts=attempts, workers=workers)
        rounds = list(sample)
        lg = torch_logits(cfg, xs)
        del xs
    redrawn = sorted(b for b, a in attempts.items() if a > 0)
    say(f"[full] {name}: redraws {sum(attempts.values())} over {len(redrawn)} rounds {redrawn[:16]}")
    plan = make_plan(cfg)
    out = run_build(plan, lg, ctx_len=ctx_tensor(cfg, range(cfg.B)))
    h = host(out)
    worst = compare_topk(h, rs, rounds=rounds)
    compare_tree(h, rs, cfg.mask, cfg.cap, rounds=rounds)
    for i in range(cfg.B):
        check_tree_properties(h, cfg, i)
    ns = h["n_star"]
    say(f"[full] {name}: {len(rounds)} of {cfg.B} rounds identical to the oracle; max |lse diff| {worst:.2e}; "
        f"n* mean {ns.mean():.1f} min {ns.min()} max {ns.max()}")


def test_full_c1():
    _full_size("c1")


def test_full_c2():
    _full_size("c2")


def test_full_c3():
    _full_size("c3")


def test_full_c4():
    _full_size("c4")


def test_many_rounds():
    # more rounds than a grid dimension of 65535 blocks: the expansion and emission grids run
    # one block per round along x
    cfg = synth.get_config("c0").replace(name="many", B=70000, L=2, V=40, K=2, cap=6)
    rng = np.random.default_rng(6)
    _full_size(cfg, sorted({0, 65535, 65536, 69999} | set(rng.choice(70000, 60, replace=False).tolist())))


def test_full_s2():
    # the paper's tree sizes (n* in the hundreds, depth up to ~19): batched selection by histogram
    _full_size("s2")


def test_full_s1():
    # a constant cost keeps every node up to the cap: 4096-node trees in the lean layout, every round
    _full_size("s1")


# ------------------------------------------------------------- context-aware cost (Sec. 4.6)

def test_ctx_parity_small():
    """Per-round context lengths inside, on and outside the grid, interpolated per eq. cv-interp."""
    cfg = synth.get_config("c1x").replace(V=20000, B=21)
    h, rs = _parity_batch(cfg, list(range(cfg.B)))
    ell = _guard.ctx_inputs(cfg)[2][: cfg.B]
    say(f"[ctx] ell={ell.tolist()}")
    assert (ell < 0).any() and (ell > 8000).any() and np.isin(ell, synth.configs.CTX_GRID).any()


def test_ctx_on_grid_point_equals_single_table():
    """A round sitting on grid point L_j uses exactly the table C_v(.; L_j)."""
    import torch
    cfg = synth.get_config("c1x").replace(V=5000, B=6)
    grid, tables = synth.ctx_tables(cfg)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    plan = make_plan(cfg)
    for j in (0, 3, 8):
        ctx = torch.full((cfg.B,), int(grid[j]), dtype=torch.int64, device="cuda")
        a = host(run_build(plan, lg, ctx_len=ctx))
        single = make_plan(cfg.replace(ctx=""), t_verify=tables[j])
        b = host(run_build(single, lg))
        say(f"[ctx] grid point {grid[j]}: n*={a['n_star'].tolist()}")
        for k in a:
            if a[k] is not None:
                assert np.array_equal(a[k], b[k]), (j, k)


def test_ctx_budget_shrinks_with_context():
    """Costs that grow with the context give budgets that do not grow with it, on the same round
    (the behaviour Sec. 5.3 reports; here each step of the grid raises C_v(n) for every n > 0 and the
    marginal costs too)."""
    import torch
    cfg = synth.get_config("c1x").replace(V=8000, B=8)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    plan = make_plan(cfg)
    prev = None
    for ell in (0, 1500, 4000, 6500, 8000):
        ctx = torch.full((cfg.B,), ell, dtype=torch.int64, device="cuda")
        ns = host(run_build(plan, lg, ctx_len=ctx))["n_star"]
        say(f"[ctx] ell={ell} n*={ns.tolist()}")
        if prev is not None:
            assert np.all(ns <= prev)
        prev = ns


def test_ctx_len_required():
    import torch
    from paper_2606_01813_amd import CaddtreeError
    cfg = synth.get_config("c1x").replace(V=3000, B=2)
    plan = make_plan(cfg)
    lg = torch_logits(cfg, synth.draw_batch(cfg))
    out = plan.new_outputs(cfg.B)
    with pytest.raises(CaddtreeError):
        plan.build(lg, out, workspace=plan.new_workspace(cfg.B))
    torch.cuda.synchronize()


def test_ctx_expand_paths_agree(monkeypatch):
    cfg = synth.get_config("c1x").replace(V=3000, B=21)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    ctx = ctx_tensor(cfg, range(cfg.B))
    outs = {}
    for mode in ("auto", "serial"):
        if mode == "serial":
            monkeypatch.setenv("CADDTREE_EXPAND", "serial")
        else:
            monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
        outs[mode] = host(run_build(make_plan(cfg), lg, ctx_len=ctx))
    _paths_agree(outs)


def test_full_c1x():
    _full_size("c1x")


def test_full_c2x():
    _full_size("c2x")


# ------------------------------------------------------------- fixed budget (DDTree, Sec. 3.4)

@pytest.mark.parametrize("name,kw", [
    ("c1f16", dict(V=6000, B=8)),
    ("c1f128", dict(V=6000, B=8)),              # the batched kernel's range
    ("c1f1024", dict(V=3000, B=3)),             # batched kernel, set read from LDS
    ("c1", dict(V=2000, B=2, cap=2048, fixed=True)),   # the largest set with a cost table
    ("c1", dict(V=2000, B=2, cap=3000, fixed=True)),   # lean set (no cost table) of 5120 nodes
    ("c1", dict(V=2000, B=2, cap=4096, fixed=True)),   # the largest budget
    ("c0", dict(fixed=True, cap=32, B=8)),      # fp32, L=4, K=4: 32 of 340 nodes
    ("c0", dict(fixed=True, L=2, K=3, cap=20, B=4, V=50)),   # 12 nodes < cap: the whole tree
])
def test_fixed_budget_parity(name, kw):
    cfg = synth.get_config(name).replace(**kw)
    h, rs = _parity_batch(cfg, list(range(cfg.B)))
    for i in range(cfg.B):
        check_tree_properties(h, cfg, i)


def test_fixed_budget_paths_agree(monkeypatch):
    cfg = synth.get_config("c1f128").replace(V=3000, B=16)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    outs = {}
    for mode in ("auto", "serial"):
        if mode == "serial":
            monkeypatch.setenv("CADDTREE_EXPAND", "serial")
        else:
            monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
        outs[mode] = host(run_build(make_plan(cfg), lg))
    _paths_agree(outs)


@pytest.mark.parametrize("name,kw", [
    ("c1f1024", dict(V=3000, B=12)),                          # fixed budget, 2048-node set
    ("c1", dict(V=2000, B=8, cap=512, fixed=True)),           # the smallest budget on eight wavefronts
    ("c1", dict(V=2000, B=6, cap=4096, fixed=True)),          # the largest budget, 5120-node set
    ("s1", dict(V=2000, B=6)),                                # cost flat to the cap 4096
    ("s1", dict(V=2000, B=8, L=12, cap=700)),                 # flat cost, shorter trees
    ("c1", dict(V=1000, B=300, cap=600, fixed=True)),         # more rounds than CUs: eight wavefronts
])
def test_wide_and_one_wave_kernels_agree(name, kw, monkeypatch):
    """Large trees of a known size run on 8 or 16 wavefronts per round (16 while every round has a
    CU of its own); the one-wavefront kernel (CADDTREE_EXPAND=level) and the serial kernel give
    the same trees."""
    cfg = synth.get_config(name).replace(**kw)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    outs = {}
    for mode in ("auto", "level", "serial"):
        if mode == "auto":
            monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
        else:
            monkeypatch.setenv("CADDTREE_EXPAND", mode)
        outs[mode] = host(run_build(make_plan(cfg), lg))
    n = outs["auto"]["n_star"]
    say(f"[wide] {cfg.name} cap {cfg.cap} B {cfg.B} n* min {n.min()} max {n.max()}")
    _paths_agree({"auto": outs["auto"], "serial": outs["level"]})
    _paths_agree({"auto": outs["auto"], "serial": outs["serial"]})


def test_wide_kernel_on_ties(monkeypatch):
    """Logits on a 0.5 grid (many nodes tie on sigma and on Lambda): the eight-wavefront kernel's
    raises, histogram splits and cut tie groups give the one-wavefront kernel's trees."""
    import torch
    cfg = synth.get_config("c4").replace(V=1500, B=48, L=8, K=16, cost="c4", cap=600, fixed=True)
    rng = np.random.default_rng(12)
    x = np.round(rng.standard_normal((cfg.B, cfg.L, cfg.V)) * 2.0) / 2.0
    peak = rng.integers(0, cfg.V, size=(cfg.B, cfg.L))
    x[np.arange(cfg.B)[:, None], np.arange(cfg.L)[None, :], peak] += rng.choice([0.0, 3.0, 6.0], size=(cfg.B, cfg.L))
    lg = torch_logits(cfg, x.astype(np.float32))
    for c in (cfg, cfg.replace(cost="const", fixed=False)):
        outs = {}
        for mode in ("auto", "level"):
            if mode == "auto":
                monkeypatch.delenv("CADDTREE_EXPAND", raising=False)
            else:
                monkeypatch.setenv("CADDTREE_EXPAND", mode)
            outs[mode] = host(run_build(make_plan(c), lg))
        n = outs["auto"]["n_star"]
        say(f"[wide ties] {c.cost} fixed={c.fixed} n* mean {n.mean():.1f} min {n.min()} max {n.max()}")
        _paths_agree({"auto": outs["auto"], "serial": outs["level"]})


def test_fixed_budget_is_top_n_of_the_greedy_tree():
    """The fixed-budget tree at n* of the greedy stop is the greedy tree itself (Prop. 1: T*_n nest)."""
    cfg = synth.get_config("c1").replace(V=6000, B=8)
    xs = synth.draw_batch(cfg)
    lg = torch_logits(cfg, xs)
    g = host(run_build(make_plan(cfg), lg))
    for i in range(cfg.B):
        n = int(g["n_star"][i])
        f = host(run_build(make_plan(cfg.replace(cap=max(n, 1), fixed=True)), lg[i:i + 1]))
        if n == 0:
            continue
        for k in ("token_ids", "parent", "depth"):
            assert np.array_equal(f[k][0, :n], g[k][i, :n]), (i, k)


def test_full_c2f128():
    _full_size("c2f128")


def test_full_c1f1024():
    _full_size("c1f1024")


# ------------------------------------------------------------- synthetic acceptance (Sec. 3.3, eq. surrogate)

def _accept(plan, topk, tree, u, ctx=None):
    import torch
    B = int(tree.token_ids.shape[0])
    al = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    rc = torch.full((B,), -7.0, dtype=torch.float64, device="cuda")
    plan.accept(topk, tree, torch.tensor(np.ascontiguousarray(u), dtype=torch.float64, device="cuda"), al, rc,
                ctx_len=ctx)
    torch.cuda.synchronize()
    return al.cpu().numpy(), rc.cpu().numpy()


def test_accept_stage_on_oracle_inputs():
    """The oracle's own top-K tables and trees: the draw and the walk alone."""
    import torch
    cfg = synth.get_config("s2").replace(V=1500, B=6)
    xs = synth.draw_batch(cfg)
    rs = [_guard.oracle_round(cfg, xs[b]) for b in range(cfg.B)]
    u = _guard.guarded_uniforms(cfg, rs, list(range(cfg.B)), tau=1e-9)
    plan = make_plan(cfg)
    topk = plan.new_outputs(cfg.B, topk=True)
    ids, logit, lse = _oracle_tables(cfg, rs)
    topk.topk_ids, topk.topk_logit, topk.lse = ids, logit, lse
    tree = plan.new_outputs(cfg.B)
    for i, r in enumerate(rs):
        n = r.n_star
        tree.token_ids[i, :n] = torch.tensor(r.tree.token_ids, dtype=torch.int32)
        tree.parent[i, :n] = torch.tensor(r.tree.parent, dtype=torch.int32)
        tree.n_star[i] = n
    al, rc = _accept(plan, topk, tree, u)
    want = [_guard.oracle.accept.simulate_round(r, u[i]) for i, r in enumerate(rs)]
    say(f"[accept] s2 n*={[r.n_star for r in rs]} alpha={al.tolist()}")
    assert al.tolist() == want
    tv = synth.cost_table(cfg)
    assert rc.tolist() == [_guard.oracle.accept.round_cost(cfg.t_draft, tv, r.n_star) for r in rs]


@pytest.mark.parametrize("name,kw", [
    ("c1", dict(V=20000, B=16)),
    ("c1x", dict(V=8000, B=14)),
    ("c0", dict(B=40)),
    ("c1f128", dict(V=5000, B=6)),
])
def test_accept_end_to_end(name, kw):
    """Build on the GPU, then accept: alpha and the round cost equal the oracle's on guarded draws."""
    cfg = synth.get_config(name).replace(**kw)
    rounds = list(range(cfg.B))
    attempts, x, rs = _guard.guarded_batch(cfg, rounds)
    u = _guard.guarded_uniforms(cfg, rs, rounds)
    plan = make_plan(cfg)
    ctx = ctx_tensor(cfg, rounds)
    out = run_build(plan, torch_logits(cfg, x), ctx_len=ctx)
    al, rc = _accept(plan, out, out, u, ctx=ctx)
    want = [_guard.oracle.accept.simulate_round(r, u[i]) for i, r in enumerate(rs)]
    say(f"[accept] {name} alpha={al.tolist()[:16]}")
    assert al.tolist() == want
    costs = [_guard.oracle.accept.round_cost(cfg.t_draft, _guard.round_cost(cfg, b), r.n_star)
             for b, r in zip(rounds, rs)]
    assert rc.tolist() == costs


def test_accept_mean_is_phi_full_c2():
    """At full size: over 1024 rounds and 8 draws each, the mean accepted length matches the mean Phi
    (eq. surrogate) within 4.5 standard errors."""
    import torch
    cfg = synth.get_config("c2")
    xs = synth.draw_batch(cfg, workers=16)
    lg = torch_logits(cfg, xs)
    del xs
    plan = make_plan(cfg)
    out = run_build(plan, lg)
    phi = out.phi.cpu().numpy().astype(np.float64)
    alphas = []
    for k in range(8):
        al, rc = _accept(plan, out, out, synth.accept_uniforms(cfg, cfg.B, k))
        assert np.all((al >= 0) & (al <= cfg.L))
        alphas.append(al)
    a = np.stack(alphas).astype(np.float64)
    # per round: E[alpha] = Phi; the rounds' draws are independent
    se = np.sqrt(a.var(axis=0, ddof=0).mean() / a.size + 1e-12)
    say(f"[accept] c2 mean alpha {a.mean():.4f} mean phi {phi.mean():.4f} se {se:.4f}")
    assert abs(a.mean() - phi.mean()) < 4.5 * max(se, 1e-3)


# ------------------------------------------------------------- fitted cost profiles (Sec. 4.6, eq. convex-reg)

def test_plan_from_fitted_profiles():
    """Noisy cost profiles at 9 context lengths, fitted by the library on the host, drive a context-aware
    plan; the oracle fits the same profiles and builds the same trees."""
    from paper_2606_01813_amd import fit_cost
    cfg = synth.get_config("c1x").replace(V=8000, B=14)
    grid, _ = synth.ctx_tables(cfg)
    n, prof = synth.cost_profiles(cfg, N=1024)
    lib_tables = np.stack([fit_cost(n, prof[j], cap=cfg.cap)[1] for j in range(len(grid))])
    ora_tables = np.stack([_guard.oracle.costfit.cost_table(n, _guard.oracle.costfit.fit_convex(n, prof[j]),
                                                              cfg.cap) for j in range(len(grid))])
    assert np.max(np.abs(lib_tables - ora_tables)) <= 1e-9 * np.max(np.abs(ora_tables))
    ell = _guard.ctx_inputs(cfg)[2]
    rounds = list(range(cfg.B))
    rs, xs = [], []
    for b in rounds:
        for a in range(_guard.MAX_ATTEMPTS):
            x = synth.draw_round(cfg, b, a)
            tv = _guard.oracle.context_cost(ora_tables, grid, int(ell[b]))
            r = _guard.oracle.build_round(x, cfg.dtype, cfg.K, cfg.t_draft, tv, cfg.cap, mask=cfg.mask)
            if _guard.clears(_guard.oracle.decision_margins(r.exp)):
                break
        rs.append(r)
        xs.append(x)
    plan = make_plan(cfg, t_verify=lib_tables, ctx_grid=grid)
    out = run_build(plan, torch_logits(cfg, np.stack(xs)), ctx_len=ctx_tensor(cfg, rounds))
    h = host(out)
    say(f"[fit] n*={h['n_star'].tolist()}")
    compare_tree(h, rs, cfg.mask, cfg.cap)


@pytest.mark.parametrize("waves", [2, 4, 8, 16])
def test_k1_merge_with_short_segments(waves, monkeypatch):
    """Rows split over more wavefronts than they have chunks: some segments are empty or hold fewer than K
    elements, so their lists end part empty and the merge ranks padding entries among the real ones."""
    monkeypatch.setenv("CADDTREE_K1_WAVES", str(waves))
    for kw in (dict(V=40, K=16, L=4, cap=64, B=4), dict(V=16, K=16, L=4, cap=600, B=3, cost="tiny"),
               dict(V=1100, K=8, L=5, cap=64, B=4)):
        _parity_batch(synth.get_config("c1").replace(**kw), list(range(kw["B"])))


@pytest.mark.parametrize("waves", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("unroll", [4, 8])
def test_k1_launch_shapes(waves, unroll, monkeypatch):
    """Every split of a row over 1 .. 16 wavefronts and both load depths give the oracle's top-K table
    and trees (the shape only changes the order of the fp64 partial sums)."""
    monkeypatch.setenv("CADDTREE_K1_WAVES", str(waves))
    monkeypatch.setenv("CADDTREE_K1_UNROLL", str(unroll))
    cfg = synth.get_config("c1").replace(V=70001, B=3)
    _parity_batch(cfg, list(range(cfg.B)))
    cfg32 = synth.get_config("c4").replace(V=30011, B=2, L=8)
    _parity_batch(cfg32, list(range(cfg32.B)))
