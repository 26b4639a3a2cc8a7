"""Helpers for the GPU parity tests: run the library through the binding and compare
element by element with the oracle."""

from __future__ import annotations

import sys

import numpy as np

import synth

# Tolerances.  The kernel's log-normaliser differs from the oracle's fp64 value
# by fp32 exp2 rounding on the terms outside the top-K (the top-K terms are
# summed in fp64), which is below 1e-8 on these workloads; 1e-7 leaves margin.
LSE_ATOL = 1e-7
PROB_RTOL = 1e-5        # probabilities and theta, relative, in fp32 (the required bound)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_logits(cfg: synth.Config, x: np.ndarray, device="cuda", pad: int = 0):
    """Host logits [n, L, V] (uint16 bf16 bits or float32) -> device tensor [n, L, V + pad]."""
    import torch
    n, L, V = x.shape
    if cfg.dtype == "bf16":
        src = torch.from_numpy(np.ascontiguousarray(x).view(np.int16))
        dt = torch.bfloat16
    else:
        src = torch.from_numpy(np.ascontiguousarray(x))
        dt = torch.float32
    if pad:
        full = torch.zeros((n, L, V + pad), dtype=src.dtype)
        full[:, :, :V] = src
        src = full
    t = src.to(device)
    if cfg.dtype == "bf16":
        t = t.view(torch.bfloat16)
    assert t.dtype == dt
    return t[:, :, :V] if pad else t


def make_plan(cfg: synth.Config, mask=None, **kw):
    """A plan for the workload: its cost table (or context tables and grid) and its budget mode."""
    from paper_2606_01813_amd import Plan
    if cfg.ctx and "t_verify" not in kw:
        grid, tables = synth.ctx_tables(cfg)
        kw.update(t_verify=tables, ctx_grid=grid)
    kw.setdefault("fixed_budget", cfg.fixed)
    return Plan(L=cfg.L, V=cfg.V, K=cfg.K, cap=cfg.cap, t_draft=cfg.t_draft,
                t_verify=kw.pop("t_verify", synth.cost_table(cfg)), dtype=cfg.dtype,
                mask=mask or cfg.mask, **kw)


def ctx_tensor(cfg: synth.Config, rounds, device="cuda"):
    """Device int64 context lengths of the given rounds of a context-aware workload (None otherwise)."""
    if not cfg.ctx:
        return None
    import torch
    from tests._guard import ctx_inputs
    ell = ctx_inputs(cfg)[2]
    return torch.tensor(np.asarray(ell)[list(rounds)], dtype=torch.int64, device=device)


def run_build(plan, logits, pos_offset=0, topk=True, ctx_len=None):
    import torch
    B = logits.shape[0]
    out = plan.new_outputs(B, device=logits.device, topk=topk)
    ws = plan.new_workspace(B, device=logits.device)
    plan.build(logits, out, pos_offset=pos_offset, workspace=ws, ctx_len=ctx_len)
    torch.cuda.synchronize()
    return out


def host(out):
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.__dict__.items()}


def compare_topk(h, rs, rounds=None, lse_atol=LSE_ATOL):
    """Top-K table of GPU outputs h (host dict) against oracle results rs (one per round)."""
    worst = 0.0
    for j, r in enumerate(rs):
        i = j if rounds is None else rounds[j]
        m = r.marg
        assert np.array_equal(h["topk_ids"][i], m["ids"]), f"round {i}: top-K ids differ"
        assert np.array_equal(h["topk_logit"][i].astype(np.float64), m["logit"]), f"round {i}: top-K logits differ"
        d = np.abs(h["lse"][i] - m["lse"])
        worst = max(worst, float(d.max()))
        assert d.max() <= lse_atol, f"round {i}: |lse diff| {d.max():.3e}"
        lq_ref = m["lq"].astype(np.float32).astype(np.float64)
        np.testing.assert_allclose(h["topk_lq"][i], lq_ref, rtol=2e-6, atol=1e-6, err_msg=f"round {i}: lq")
    return worst


def compare_tree(h, rs, cfg_mask, cap, rounds=None, pos_offset=0, prob_rtol=PROB_RTOL):
    for j, r in enumerate(rs):
        i = j if rounds is None else rounds[j]
        n = r.n_star
        assert h["n_star"][i] == n, f"round {i}: n_star {h['n_star'][i]} != {n}"
        t = r.tree
        assert np.array_equal(h["token_ids"][i, :n], t.token_ids), f"round {i}: token ids"
        assert np.array_equal(h["parent"][i, :n], t.parent), f"round {i}: parents"
        assert np.array_equal(h["depth"][i, :n], t.depth), f"round {i}: depths"
        assert np.array_equal(h["pos_ids"][i, :n], t.pos_ids), f"round {i}: pos ids"
        np.testing.assert_allclose(h["path_prob"][i, :n], t.path_prob.astype(np.float32), rtol=prob_rtol,
                                   err_msg=f"round {i}: path_prob")
        np.testing.assert_allclose(h["phi"][i], np.float32(r.exp.phi), rtol=prob_rtol, err_msg=f"round {i}: phi")
        np.testing.assert_allclose(h["theta"][i], np.float32(r.exp.theta), rtol=prob_rtol,
                                   err_msg=f"round {i}: theta")
        # untouched beyond n*
        assert np.all(h["token_ids"][i, n:] == -1) and np.all(h["parent"][i, n:] == -2)
        if cfg_mask == "u8":
            assert np.array_equal(h["mask"][i, :n, :n], r.mask), f"round {i}: dense mask"
            assert not h["mask"][i, n:, :].any() and not h["mask"][i, :, n:].any()
        elif cfg_mask == "bits":
            words = (n + 31) // 32
            got = h["mask"][i, :n, :words].view(np.uint32)
            assert np.array_equal(got, r.mask[:, :words]), f"round {i}: packed mask"
            assert not h["mask"][i, n:, :].any() and not h["mask"][i, :, words:].any()


def check_tree_properties(h, cfg: synth.Config, i: int, t_verify=None):
    """Properties every output round satisfies, whatever its inputs (any size)."""
    n = int(h["n_star"][i])
    assert 0 <= n <= cfg.cap
    if cfg.fixed:
        total = sum(cfg.K ** d for d in range(1, cfg.L + 1))
        assert n == min(cfg.cap, total)
    if t_verify is None:
        from tests._guard import round_cost
        t_verify = round_cost(cfg, i)
    tv = t_verify
    par, dep, tok = h["parent"][i, :n], h["depth"][i, :n], h["token_ids"][i, :n]
    assert np.all(par < np.arange(n))
    assert np.all((dep >= 1) & (dep <= cfg.L))
    assert np.all(dep[par >= 0] == dep[par[par >= 0]] + 1) if n else True
    assert np.all(dep[par < 0] == 1)
    assert np.all(np.diff(dep) >= 0)
    ids = h["topk_ids"][i] if h.get("topk_ids") is not None else None
    if ids is not None and n:
        assert np.all(np.isin(tok, ids.reshape(-1)))
    pp = h["path_prob"][i, :n].astype(np.float64)
    if n:
        assert np.all(pp[par >= 0] <= pp[par[par >= 0]] * (1 + 1e-6))
    phi = float(h["phi"][i])
    assert abs(phi - pp.sum()) <= 1e-5 * max(1.0, phi)
    theta = (1.0 + phi) / (cfg.t_draft + tv[n])
    assert abs(float(h["theta"][i]) - theta) <= 1e-5 * theta
