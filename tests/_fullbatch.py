"""Full-size batches for the GPU parity tests, with the oracle's result for every round.

Every round of the batch goes through the input guard (tests/_guard.py): it is
drawn, built by the oracle and redrawn with its next seed attempt until its
decision margins clear the guard.  The work runs in a pool of *spawned* worker
processes that import only numpy, the input generators and the oracle, so
they never touch the GPU; each writes its rounds' logits into one shared-memory
batch and returns their oracle results.  The pool is closed and joined (not
terminated), so its workers exit on their own.
"""

from __future__ import annotations

import multiprocessing as mp
import time
from multiprocessing import shared_memory
from typing import Any, Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth
from synth.gen import default_workers, np_dtype

_SHM = None


def _init(name: str) -> None:
    global _SHM
    _SHM = shared_memory.SharedMemory(name=name)


def _work(args):
    from tests import _guard
    cfg, n, chunk = args
    out = np.ndarray((n, cfg.L, cfg.V), dtype=np_dtype(cfg), buffer=_SHM.buf)
    res = []
    for slot, b in chunk:
        a, x, r = _guard.guarded_round(cfg, b)
        out[slot] = x
        res.append((slot, a, r))
    del out
    return res


def guarded_batch(cfg: synth.Config, rounds: Optional[Sequence[int]] = None, workers: Optional[int] = None,
                  chunk: int = 8, say=print, consume: Optional[Callable[[np.ndarray], Any]] = None
                  ) -> Tuple[Dict[int, int], Any, List]:
    """(attempts {b: a}, logits, oracle results) for the given rounds (default: all B).

    The logits [n, L, V] are a copy of the shared batch, or, with ``consume``, whatever
    ``consume(batch)`` returns (for example a device copy), taken before the shared memory is released.
    """
    rounds = list(range(cfg.B)) if rounds is None else list(rounds)
    n = len(rounds)
    workers = default_workers() if workers is None else max(1, int(workers))
    shape = (n, cfg.L, cfg.V)
    dt = np_dtype(cfg)
    nbytes = int(np.prod(shape)) * np.dtype(dt).itemsize
    shm = shared_memory.SharedMemory(create=True, size=max(1, nbytes))
    attempts: Dict[int, int] = {}
    results: List = [None] * n
    t0 = time.perf_counter()
    try:
        jobs = [(cfg, n, [(s, rounds[s]) for s in range(k, min(k + chunk, n))]) for k in range(0, n, chunk)]
        pool = mp.get_context("spawn").Pool(workers, initializer=_init, initargs=(shm.name,))
        try:
            done, step = 0, max(1, n // 4)
            for res in pool.imap_unordered(_work, jobs):
                for slot, a, r in res:
                    attempts[rounds[slot]] = a
                    results[slot] = r
                before, done = done, done + len(res)
                if done // step != before // step or done == n:
                    say(f"[full] {cfg.name}: oracle {done}/{n} rounds ({time.perf_counter() - t0:.1f} s)")
        finally:
            pool.close()
            pool.join()
        t1 = time.perf_counter()
        view = np.ndarray(shape, dtype=dt, buffer=shm.buf)
        xs = view.copy() if consume is None else consume(view)
        del view
        say(f"[full] {cfg.name}: workers joined after {t1 - t0:.1f} s, batch taken in {time.perf_counter() - t1:.1f} s")
    finally:
        shm.close()
        shm.unlink()
    return attempts, xs, results
