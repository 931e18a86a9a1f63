"""fp64 target epilogue (test infrastructure): from per-query-head future masses to
the per-KV-head target score of KVpop.

App. D.4 step 5 finishes the target computation: aggregate the G query heads that
share a KV head and normalise by the number of future queries. This follows the
order of App. B.1-B.2:

* aggregation over g (App. B.1): max, eq. max_group_aggregation_app (the default),
  or the probability-space mean, eq. mean_group_aggregation_app;
* r_bar = log(m_agg + eps);
* count normalisation (App. B.2, eqs. future_count_app, normalized_target_app):
  r = r_bar - log N_t with N_t = max(1, T - (t + w)), clipped to N_t <= L + 1 for a
  finite lookahead L. With the band convention d in [t + window, t + horizon],
  N_t = max(1, number of admissible d).

eps is a free parameter in the paper (Sec. 3.1 only requires eps > 0).
"""
from __future__ import annotations

import numpy as np

__all__ = ["future_count", "target_scores"]


def future_count(T: int, window: int, horizon: int) -> np.ndarray:
    """N_t for t = 0..T-1: the number of admissible query positions, at least 1."""
    t = np.arange(T)
    n = T - (t + window)
    if horizon >= 0:
        n = np.minimum(n, horizon - window + 1)
    return np.maximum(1, n)


def target_scores(m_bar, n_kv_heads: int, window: int, horizon: int, agg: str = "max", eps: float = 1e-8,
                  normalize: bool = True) -> np.ndarray:
    """r[b, h, t] from m_bar[b, qh, t] (query head qh belongs to KV head qh // G)."""
    m = np.asarray(m_bar, dtype=np.float64)
    B, Hq, T = m.shape
    if Hq % n_kv_heads:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // n_kv_heads
    grouped = m.reshape(B, n_kv_heads, G, T)
    if agg == "max":
        m_agg = grouped.max(axis=2)
    elif agg == "mean":
        m_agg = grouped.mean(axis=2)
    else:
        raise ValueError("agg must be 'max' or 'mean'")
    with np.errstate(divide="ignore"):  # eps = 0 and an empty band give log(0) = -inf
        r = np.log(m_agg + eps)
    if normalize:
        r = r - np.log(future_count(T, window, horizon))[None, None, :]
    return r
