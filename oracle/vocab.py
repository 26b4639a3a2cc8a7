"""Per-position marginals: log-normaliser and top-K (oracle; test infrastructure).

The drafter's marginal at block position i is q_i = softmax(l_i) over the full
vocabulary (Sec. 3.2, eq. marginals).  Algorithm 1 consumes, per position, the
top-K tokens and their log-probabilities log q_i^(k) = l_i^(k) - LSE_i, where
LSE_i = log sum_v exp(l_i,v) is the full-vocabulary log-normaliser (no
renormalisation over the K kept tokens).
"""

from __future__ import annotations

import numpy as np


def widen(logits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored logits to float64.

    ``dtype == "bf16"``: ``logits`` holds uint16 bf16 bit patterns; a bf16 value
    is the fp32 value whose upper 16 bits are those bits.  ``"f32"``: float32.
    """
    if dtype == "bf16":
        bits = np.asarray(logits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(logits, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def log_normalizer(x: np.ndarray) -> float:
    """LSE of one row: m + log(sum_v exp(x_v - m)), m = max_v x_v (eq. marginals)."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("logits must be finite")
    m = float(np.max(x))
    return m + float(np.log(np.sum(np.exp(x - m))))


def top_k(x: np.ndarray, K: int):
    """The K largest entries of one row, ordered by value descending, then token id ascending.

    Returns (ids int64 [K], values float64 [K]).
    """
    x = np.asarray(x, dtype=np.float64)
    ids = np.arange(x.shape[0], dtype=np.int64)
    # np.lexsort sorts by the last key first: primary -x (value desc), secondary id (asc)
    order = np.lexsort((ids, -x))[:K]
    return ids[order], x[order]


def marginals(logits: np.ndarray, dtype: str, K: int):
    """Top-K table of one round.

    ``logits``: [L, V] stored logits.  Returns a dict with
    ``ids`` int64 [L, K], ``logit`` float64 [L, K] (the raw logits, exact),
    ``lq`` float64 [L, K] (log q_i^(k)), ``lse`` float64 [L].
    """
    x = widen(logits, dtype)
    L, V = x.shape
    if not 1 <= K <= V:
        raise ValueError("need 1 <= K <= V")
    ids = np.empty((L, K), dtype=np.int64)
    val = np.empty((L, K), dtype=np.float64)
    lse = np.empty(L, dtype=np.float64)
    for i in range(L):
        ids[i], val[i] = top_k(x[i], K)
        lse[i] = log_normalizer(x[i])
    return {"ids": ids, "logit": val, "lq": val - lse[:, None], "lse": lse}
