#!/usr/bin/env python3
"""Benchmark: CaDDTree draft-tree construction throughput on one MI355X.

One step = one ``caddtree_build`` over a whole batch of rounds (vocabulary
reduction + top-K, best-first expansion with the greedy stop, mask and position
ids), with the logits already resident in HBM.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--workload c2]

Other workloads (``--workload``): c1, c3, c4, the stress cases s1, s2, the
context-aware cost variants c1x, c2x (one context length per round, nine cost
tables, Sec. 4.6) and the fixed-budget (DDTree) variants c1f16, c1f128,
c1f1024, c2f128, c2f1024.

``--simulate`` runs the synthetic analogue of the paper's comparisons
(Tab. 1-3) instead: trees from CaDDTree, from the fixed-budget construction
at every budget of the DDTree grid {16, .., 1024}, from a constant C_v and
from perturbed cost parameters, each verified against target paths drawn from
the drafter's marginals (``caddtree_accept``) and charged under the nominal
cost model; prints one JSON line with time per token (sum C / sum (1 +
alpha), in units of C_d), mean accepted length and mean budget per variant.

Timing: the read-bandwidth probe runs first (its sweep brings the GPU to its working clocks), then
W warm-up steps, then K steps back to back with HIP events on the launch stream before the first and
after the last: ``value`` = B K / that time.  (An event between two steps leaves the GPU idle for
several microseconds, so per-step events, recorded in a second pass, give only the distribution.)
The roofline's kernel time is the average of K back-to-back launches of the vocabulary reduction
between two events; a stage-by-stage pass gives the split between the three stages.

Default workload c2: 1024 rounds x L=16 x V=151936 bf16 logits, K=8, cap 512,
C_d = 1, C_v(n) = 1 + 0.002 n + 0.00002 n^2 (the HBM-saturating batch of the
L=16 / V=151936 / bf16 rounds/sec metric).  Inputs are the seeded synthetic
generator of that workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
METRIC = "rounds/sec, L=16 V=151936 bf16 marginals→CaDDTree; % of HBM peak"
K1_SOURCE = os.path.join(ROOT, "paper_2606_01813_amd", "csrc", "reduce_topk.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def k1_source_hash() -> str:
    with open(K1_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per K1 launch from committed rocprofv3 counter runs, if they match this kernel source."""
    path = os.path.join(ROOT, "profiles", f"k1_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("k1_source_sha256_16") != k1_source_hash():
        return None
    return rec.get("bytes_per_launch")


_POOL_XS = None     # the batch, shared with forked workers (copy-on-write)
_POOL_CFG = None


def _oracle_round(cfg, x, b: int, tv_plain, ctx) -> bool:
    """One round through the oracle; True if its decision margins clear the parity tests' input guard."""
    import oracle
    from tests._guard import clears
    tv = tv_plain if ctx is None else oracle.context_cost(ctx[1], ctx[0], int(ctx[2][b]))
    r = oracle.build_round(x, cfg.dtype, cfg.K, cfg.t_draft, tv, cfg.cap, mask=cfg.mask,
                           budget=cfg.cap if cfg.fixed else None)
    return clears(oracle.decision_margins(r.exp))


def _pool_worker(args):
    start, stride, deadline = args
    cfg, xs = _POOL_CFG, _POOL_XS
    tv = synth.cost_table(cfg)
    ctx = None
    if cfg.ctx:
        grid, tables = synth.ctx_tables(cfg)
        ctx = (grid, tables, synth.ctx_lengths(cfg, cfg.B))
    n = near = 0
    b = start
    while b < xs.shape[0] and time.time() < deadline:
        near += not _oracle_round(cfg, xs[b], b, tv, ctx)
        n += 1
        b += stride
    return n, near


def cpu_baseline(cfg, xs, target_s: float, max_rounds: int):
    """The oracle (test infrastructure) on the host's cores: a fork pool over the rounds of the same batch
    for about target_s seconds (the rounds a worker has started are finished), plus one core alone."""
    import multiprocessing as mp
    global _POOL_XS, _POOL_CFG
    tv = synth.cost_table(cfg)
    ctx = None
    if cfg.ctx:
        grid, tables = synth.ctx_tables(cfg)
        ctx = (grid, tables, synth.ctx_lengths(cfg, cfg.B))
    # one core
    t0 = time.perf_counter()
    n1 = 0
    while n1 < min(max_rounds, xs.shape[0]):
        _oracle_round(cfg, xs[n1], n1, tv, ctx)
        n1 += 1
        if time.perf_counter() - t0 >= target_s / 4:
            break
    one = n1 / (time.perf_counter() - t0)
    # every core the process may use (at most 16: the host share of one GPU)
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    workers = max(1, min(16, avail))
    _POOL_XS, _POOL_CFG = xs, cfg
    t0 = time.perf_counter()
    deadline = time.time() + target_s
    pool = mp.get_context("fork").Pool(workers)
    try:
        counts = pool.map(_pool_worker, [(w, workers, deadline) for w in range(workers)])
    finally:
        pool.close()
        pool.join()
    dt = time.perf_counter() - t0
    _POOL_XS = None
    n = sum(c[0] for c in counts)
    near = sum(c[1] for c in counts)
    return {"value": n / dt, "unit": "rounds/s", "cores": workers, "kind": "oracle",
            "single_core_value": one,
            "guard": {"rounds": n, "near_a_tie": near,
                      "rule": "a round is near a tie when a stop margin or cross-depth gap is below "
                              "max(1e-6, 2 * depth span * 1e-7); the parity tests redraw such rounds"},
            "sample": f"{n} rounds of {cfg.name} on a fork pool of {workers} workers ({dt:.1f} s; "
                      f"{avail} cores available), and {n1} rounds on one core; single-process fp64 numpy oracle "
                      f"(LSE + top-K + Algorithm 1 + mask per round); input generation excluded"}


def copy_probe(mib: int) -> None:
    """A plain device copy of known size (y = x * 1, fp32) for counter calibration: one launch reads and
    writes mib MiB.  The source is never written and a larger buffer is written after allocating it, so
    none of it sits in a cache when the copy runs."""
    import torch
    n = mib * (1 << 20) // 4
    x = torch.empty(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    evict = torch.zeros(max(n // 2, 1 << 28), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    del evict
    torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "launches": 1}), flush=True)


PROBE_LIB = os.path.join(ROOT, "paper_2606_01813_amd", "libcaddtree_probe.so")


def read_probe(logits, cfg, stream, reps: int = 10):
    """Best pure-read time over the logits batch (same rows, same 16-byte non-temporal loads as the
    reduction kernel, no arithmetic), over every wave split and load depth: the bandwidth a read of this
    shape reaches on this GPU.  None when the rows are not whole 16-byte units."""
    import ctypes
    import torch
    es = cfg.elem_bytes
    row_bytes = cfg.V * es
    stride = int(logits.stride(1)) * es
    if row_bytes % 16 or stride % 16 or logits.data_ptr() % 16:
        return None
    lib = ctypes.CDLL(PROBE_LIB)
    lib.caddtree_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.caddtree_probe_read.restype = ctypes.c_int
    sink = torch.zeros(1, dtype=torch.int32, device=logits.device)
    rows = cfg.B * cfg.L
    best = None
    for waves in (1, 2, 4, 8, 16):
        for unroll in (4, 8):
            def launch():
                rc = lib.caddtree_probe_read(logits.data_ptr(), rows, stride, row_bytes, waves, unroll,
                                             sink.data_ptr(), stream.cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"read probe launch failed: hipError {rc}")
            for _ in range(2):
                launch()
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for a, b in ev:
                a.record(stream)
                launch()
                b.record(stream)
            torch.cuda.synchronize()
            us = float(np.median([a.elapsed_time(b) for a, b in ev])) * 1e3
            if best is None or us < best["us"]:
                best = {"us": us, "waves_per_row": waves, "unroll": unroll}
    best["bytes"] = rows * row_bytes
    best["gbs"] = best["bytes"] / (best["us"] * 1e-6) / 1e9
    return best


def nstar_histogram(ns):
    """Counts of n* in power-of-two bins [0, 1), [1, 2), [2, 4), .. (the last bin ends past the largest n*)."""
    edges = [0, 1]
    while edges[-1] <= int(ns.max()):
        edges.append(edges[-1] * 2)
    counts, _ = np.histogram(ns, bins=edges)
    return {"edges": edges, "counts": counts.tolist()}


DDTREE_GRID = (16, 32, 64, 128, 256, 512, 1024)


def simulate(args) -> None:
    """Simulated time per token of CaDDTree against the fixed-budget construction and cost ablations."""
    import torch
    from paper_2606_01813_amd import Plan
    cfg = synth.get_config(args.workload or "s2")
    assert not cfg.ctx and not cfg.fixed, "simulate takes a plain workload"
    log(f"[simulate] generating {cfg.name}: {cfg.B} x {cfg.L} x {cfg.V} {cfg.dtype}")
    xs = synth.draw_batch(cfg, workers=args.workers)
    dev = torch.device("cuda:0")
    if cfg.dtype == "bf16":
        logits = torch.from_numpy(xs.view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        logits = torch.from_numpy(xs).to(dev)
    del xs
    B = cfg.B
    tv = synth.cost_table(cfg)
    big = max(cfg.cap, max(DDTREE_GRID))
    nominal = Plan(L=cfg.L, V=cfg.V, K=cfg.K, cap=big, t_draft=cfg.t_draft,
                   t_verify=synth.cost_table(cfg.cost, big), dtype=cfg.dtype, mask="none")
    us = [torch.from_numpy(synth.accept_uniforms(cfg, B, k)).to(dev) for k in range(args.draws)]

    variants = [("caddtree", dict(cap=cfg.cap, t_draft=cfg.t_draft, t_verify=tv))]
    variants += [(f"fixed_{n}", dict(cap=n, t_draft=cfg.t_draft, t_verify=synth.cost_table(cfg.cost, n),
                                    fixed_budget=True)) for n in DDTREE_GRID]
    flat = np.full(min(cfg.cap, 1024) + 1, tv[0])
    variants += [("constant_cv", dict(cap=min(cfg.cap, 1024), t_draft=cfg.t_draft, t_verify=flat))]
    variants += [("cd_x0.5", dict(cap=cfg.cap, t_draft=0.5 * cfg.t_draft, t_verify=tv)),
                 ("cd_x2", dict(cap=cfg.cap, t_draft=2.0 * cfg.t_draft, t_verify=tv)),
                 ("cv_x0.5", dict(cap=cfg.cap, t_draft=cfg.t_draft, t_verify=0.5 * tv)),
                 ("cv_x2", dict(cap=cfg.cap, t_draft=cfg.t_draft, t_verify=2.0 * tv))]
    rows = {}
    for vname, kw in variants:
        plan = Plan(L=cfg.L, V=cfg.V, K=cfg.K, dtype=cfg.dtype, mask="none", **kw)
        out = plan.new_outputs(B, topk=True)
        plan.build(logits, out, workspace=plan.new_workspace(B))
        al = torch.empty(B, dtype=torch.int32, device=dev)
        rc = torch.empty(B, dtype=torch.float64, device=dev)
        tot_c = tot_t = tot_a = 0.0
        for u in us:
            nominal.accept(out, out, u, al, rc)
            tot_c += float(rc.sum())
            tot_t += float((al.to(torch.float64) + 1.0).sum())
            tot_a += float(al.to(torch.float64).sum())
        ns = out.n_star.to(torch.float64)
        rows[vname] = {"time_per_token": tot_c / tot_t, "mean_accept": tot_a / (B * len(us)),
                       "mean_n_star": float(ns.mean()), "std_n_star": float(ns.std()),
                       "mean_phi": float(out.phi.to(torch.float64).mean())}
        log(f"[simulate] {vname:12s} time/token {rows[vname]['time_per_token']:.4f} "
            f"accept {rows[vname]['mean_accept']:.3f} n* {rows[vname]['mean_n_star']:.1f}")
        plan.close()
    best = min(DDTREE_GRID, key=lambda n: rows[f"fixed_{n}"]["time_per_token"])
    line = {"simulate": cfg.name, "rounds": B, "draws": len(us),
            "workload": f"{cfg.name}: {B} rounds x L={cfg.L} x V={cfg.V} {cfg.dtype}, K={cfg.K}, cap {cfg.cap}",
            "cost_units": "C_d = 1", "variants": rows, "ddtree_oracle_budget": best,
            "caddtree_over_ddtree_oracle": rows["caddtree"]["time_per_token"] / rows[f"fixed_{best}"]["time_per_token"]}
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None, help="default c2 (s2 with --simulate)")
    ap.add_argument("--workers", type=int, default=synth.gen.default_workers())
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", action="store_true", help="skip the read-bandwidth probe (counter runs)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain elementwise copy of this many MiB (counter calibration)")
    ap.add_argument("--simulate", action="store_true",
                    help="synthetic analogue of the paper's comparisons (default workload s2)")
    ap.add_argument("--draws", type=int, default=16, help="target-path draws per round for --simulate")
    args = ap.parse_args()
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    if args.simulate:
        simulate(args)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the rounds are independent and this "
              f"build has no multi-GPU path; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    cfg = synth.get_config(args.workload or "c2")
    log(f"[bench] generating {cfg.name}: {cfg.B} x {cfg.L} x {cfg.V} {cfg.dtype} ({cfg.batch_bytes / 1e9:.2f} GB) "
        f"with {args.workers} workers")
    t = time.perf_counter()
    xs = synth.draw_batch(cfg, workers=args.workers)
    log(f"[bench] generated in {time.perf_counter() - t:.1f} s")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] cpu baseline: oracle on up to {args.cpu_seconds:.0f} s of rounds")
        cpu = cpu_baseline(cfg, xs, args.cpu_seconds, max_rounds=cfg.B)
        log(f"[bench] cpu baseline {cpu['value']:.3f} rounds/s")

    import torch
    from paper_2606_01813_amd import Plan
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if cfg.dtype == "bf16":
        logits = torch.from_numpy(xs.view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        logits = torch.from_numpy(xs).to(dev)
    del xs
    cost_kw = dict(t_verify=synth.cost_table(cfg))
    ctx = None
    if cfg.ctx:
        grid, tables = synth.ctx_tables(cfg)
        cost_kw = dict(t_verify=tables, ctx_grid=grid)
        ctx = torch.from_numpy(synth.ctx_lengths(cfg, cfg.B)).to(dev)
    plan = Plan(L=cfg.L, V=cfg.V, K=cfg.K, cap=cfg.cap, t_draft=cfg.t_draft, dtype=cfg.dtype, mask=cfg.mask,
                fixed_budget=cfg.fixed, **cost_kw)
    B = cfg.B
    out = plan.new_outputs(B)
    ws = plan.new_workspace(B)
    stream = torch.cuda.current_stream()

    def step():
        plan.build(logits, out, pos_offset=0, workspace=ws, stream=stream, ctx_len=ctx)

    # the read probe first: its sweep streams the logits about a hundred times, so the GPU is at its
    # working clocks when the warm-up steps start
    probe = None if args.no_probe else read_probe(logits, cfg, stream)
    if probe:
        log(f"[bench] read probe {probe['us']:.1f} us = {probe['gbs']:.0f} GB/s "
            f"({probe['waves_per_row']} waves per row, {probe['unroll']} loads in flight)")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K whole-path steps back to back, HIP events on the launch stream before the first and
    # after the last only (an event between steps leaves the GPU idle for several microseconds)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gpu_step_us = ev0.elapsed_time(ev1) * 1e3 / args.steps
    log(f"[bench] {args.steps} steps in {elapsed * 1e3:.2f} ms (wall); {gpu_step_us:.1f} us per step on the GPU")

    # the same steps once more, each bracketed by its own events: the distribution of step times (each
    # step then also carries the events' idle time)
    step_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
    for a, b in step_ev:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    step_us = np.array([a.elapsed_time(b) for a, b in step_ev]) * 1e3

    # the vocabulary reduction alone, K launches back to back between two HIP events on the launch stream:
    # their average duration is the roofline's
    topk = plan.new_outputs(B, topk=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        plan.reduce_topk(logits, topk.topk_ids, topk.topk_logit, topk.lse, topk.topk_lq, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    k1_avg = e0.elapsed_time(e1) * 1e3 / args.steps   # us

    # per-stage durations (the same work through the three stage entry points, interleaved)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for s in range(args.steps):
        e = ev[s]
        e[0].record(stream)
        plan.reduce_topk(logits, topk.topk_ids, topk.topk_logit, topk.lse, topk.topk_lq, stream=stream)
        e[1].record(stream)
        plan.expand(topk.topk_ids, topk.topk_logit, topk.lse, topk, stream=stream, ctx_len=ctx)
        e[2].record(stream)
        plan.emit(topk, pos_offset=0, stream=stream)
        e[3].record(stream)
    torch.cuda.synchronize()
    k1s = np.array([e[0].elapsed_time(e[1]) for e in ev]) * 1e3   # us
    k2 = np.array([e[1].elapsed_time(e[2]) for e in ev]) * 1e3
    k3 = np.array([e[2].elapsed_time(e[3]) for e in ev]) * 1e3
    ns = out.n_star.cpu().numpy()
    same = bool(torch.equal(out.n_star, topk.n_star) and torch.equal(out.token_ids, topk.token_ids))

    rows = B * cfg.L
    k1_bytes = rows * cfg.V * cfg.elem_bytes + rows * (cfg.K * 12 + 8)
    achieved = k1_bytes / (k1_avg * 1e-6) / 1e9
    med_step = float(np.median(step_us))
    value = B / (gpu_step_us * 1e-6)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": gpu_step_us * 1e-3,
        "wall_ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {B} rounds x L={cfg.L} x V={cfg.V} {cfg.dtype} logits, K={cfg.K}, "
                               f"cap {cfg.cap}, mask {cfg.mask}"
                               + (", context-aware cost (9 tables)" if cfg.ctx else "")
                               + (", fixed budget" if cfg.fixed else ""),
                   "rounds": B, "L": cfg.L, "V": cfg.V, "logits_dtype": cfg.dtype, "K": cfg.K, "cap": cfg.cap,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(cfg.name),
                     "kernel": "reduce_topk_kernel", "bytes_per_launch": k1_bytes,
                     "avg_launch_us": k1_avg,
                     "probe_gbs": probe["gbs"] if probe else None,
                     "pct_of_probe": achieved / probe["gbs"] if probe else None},
        "read_probe": probe,
        "cpu_baseline": cpu,
        "stages_us": {"reduce_topk": float(k1s.mean()), "expand": float(k2.mean()), "emit": float(k3.mean())},
        "stages_median_us": {"reduce_topk": float(np.median(k1s)), "expand": float(np.median(k2)),
                             "emit": float(np.median(k3))},
        # the expansion is a dependent chain per round, with no bandwidth or flop roofline: its batch time,
        # that time per round, and the nodes the batch keeps per second of it
        "expand": {"median_us_per_batch": float(np.median(k2)), "us_per_round": float(np.median(k2)) / B,
                   "nodes_kept": int(ns.sum()), "nodes_kept_per_s": float(ns.sum()) / (float(np.median(k2)) * 1e-6)},
        "step_us": {"gpu_mean": gpu_step_us,
                    "with_per_step_events": {"median": med_step, "min": float(step_us.min()),
                                             "max": float(step_us.max()), "rounds_per_s_at_median": B / (med_step * 1e-6),
                                             "all": [round(float(x), 1) for x in step_us]}},
        "end_to_end_hbm_frac": cfg.batch_bytes / (gpu_step_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "n_star": {"mean": float(ns.mean()), "std": float(ns.std()), "min": int(ns.min()), "max": int(ns.max()),
                   "histogram": nstar_histogram(ns)},
        "stage_path_matches_build": same,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
