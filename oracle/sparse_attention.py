"""fp64 oracle of KVpop's running top-k sparse attention forward (test infrastructure).

The student's attention keeps, for each query q, the keys of the running top-k mask
(Sec. 3.2, App. C.1 eq. running_topk_mask_app) and attends over them with an
ordinary causal softmax (App. C.3): with logits l(q, t) = scale <q_q, k_t> + bias_t,

  LSE~_q = log sum_t M[q, t] exp l(q, t)          (Sec. 3.2 eq. sparse_lse_main)
  O_q    = sum_t M[q, t] exp(l(q, t) - LSE~_q) v_t

The LSE is the one the paper hands to its transposed target pass (App. D.3).

Token lifetimes. Once the eligible set holds k tokens its cutoff can only fall
(each query adds one eligible token, and the k-th smallest rank of a growing set
does not grow), and before that every eligible token is kept. So a token that
leaves the mask never returns: the queries keeping token t form one interval
[t, e_t). ``eviction_times_bruteforce`` reads e_t off the mask row by row (and
checks that the interval property holds); ``eviction_times`` gets it from the
cutoffs: e_t = T for sinks, otherwise the later of t + w (leaving the protected
window) and the first query whose cutoff drops below rank(t), capped at T.
"""
from __future__ import annotations

import numpy as np

from .future_mass import _as_f64

__all__ = ["eviction_times", "eviction_times_bruteforce", "running_topk_mask_rows", "sparse_attention",
           "lifetime_mask"]


def eviction_times_bruteforce(rank, tau, s: int, w: int) -> np.ndarray:
    """e_t = the first query q >= t with M[q, t] = 0 (T if none), from the mask of
    eq. running_topk_mask_app evaluated one entry at a time. Raises if a token is
    kept again after it was dropped (the interval property fails)."""
    rank = np.asarray(rank)
    tau = np.asarray(tau)
    T = rank.shape[0]
    e = np.full(T, T, dtype=np.int64)
    for t in range(T):
        dropped = None
        for q in range(t, T):
            kept = t < s or (q - t) < w or (s <= t <= q - w and rank[t] <= tau[q])
            if not kept and dropped is None:
                dropped = q
            elif kept and dropped is not None:
                raise AssertionError("token %d is kept again at query %d after leaving at %d" % (t, q, dropped))
        if dropped is not None:
            e[t] = dropped
    return e


def eviction_times(rank, tau, s: int, w: int) -> np.ndarray:
    """e_t from non-increasing cutoffs: T for t < s, else min(T, max(t + w, f_t)) with
    f_t the first query whose cutoff is below rank(t) (T if none)."""
    rank = np.asarray(rank, dtype=np.int64)
    tau = np.asarray(tau, dtype=np.int64)
    T = rank.shape[0]
    if T > 1 and np.any(np.diff(tau) > 0):
        raise ValueError("cutoffs must be non-increasing")
    # first q with tau[q] < r: tau is non-increasing, so -tau is non-decreasing and
    # the count of q with -tau[q] <= -r is the count of q with tau[q] >= r.
    f = np.searchsorted(-tau, -rank, side="right")
    t = np.arange(T, dtype=np.int64)
    e = np.minimum(T, np.maximum(t + w, f))
    e[t < s] = T
    return e


def lifetime_mask(evict, rows=None) -> np.ndarray:
    """Boolean mask [len(rows), T] with M[q, t] = [t <= q < e_t]."""
    e = np.asarray(evict, dtype=np.int64)
    T = e.shape[0]
    q = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    t = np.arange(T)
    return (t[None, :] <= q[:, None]) & (q[:, None] < e[None, :])


def running_topk_mask_rows(rank, tau, s: int, w: int, rows) -> np.ndarray:
    """Rows `rows` of the mask of eq. running_topk_mask_app (causal), [len(rows), T]."""
    rank = np.asarray(rank)
    tau = np.asarray(tau)
    T = rank.shape[0]
    q = np.asarray(rows, dtype=np.int64)[:, None]
    t = np.arange(T)[None, :]
    sink = t < s
    recent = (q - t) < w
    eligible = (t >= s) & (t <= q - w)
    selected = rank[None, :] <= tau[np.asarray(rows)][:, None]
    return (t <= q) & (sink | recent | (eligible & selected))


def sparse_attention(q, k, v, scale: float, mask, bias=None):
    """Masked softmax attention of one head in fp64.

    q: [R, D] query rows (bf16 bits or floats), k, v: [T, D], mask: bool [R, T] with
    at least one kept key per row, bias: optional [T] added to every logit of key t.
    Returns (O [R, D], LSE [R], A [R, D]) where A = sum_t p_t |v_t| bounds how far a
    rounding of the probabilities can move O (used by the tests' tolerance)."""
    qv = _as_f64(q)
    kv = _as_f64(k)
    vv = _as_f64(v)
    M = np.asarray(mask, dtype=bool)
    if not np.all(M.any(axis=1)):
        raise ValueError("every query row must keep at least one key")
    L = float(scale) * (qv @ kv.T)
    if bias is not None:
        L = L + _as_f64(bias)[None, :]
    L = np.where(M, L, -np.inf)
    mx = L.max(axis=1)
    lse = mx + np.log(np.sum(np.exp(L - mx[:, None]), axis=1))
    P = np.exp(L - lse[:, None])
    return P @ vv, lse, P @ np.abs(vv)
