"""Plain fp64 evaluation of the dense future-attention target (test infrastructure).

Notation follows the paper (App. D.1): query positions d, key positions t, logit
l(d, t), causal log-normaliser LSE_d, probability p_{d->t}, unnormalised future
mass m_bar_t summed over query positions d from t + w onwards (eq. future_mass_app,
with the paper's protected window w). The finite lookahead of App. B.2 is expressed
as ``horizon`` = largest admissible d - t (so the paper's lookahead L is
horizon = w + L); ``horizon < 0`` means no lookahead limit.

Grouped-query attention: query head ``qh`` reads KV head ``qh // G`` with
``G = Hq // Hkv`` (the paper's g index runs over the G query heads of KV head h).

Inputs are numpy arrays: either uint16 bf16 bit patterns (decoded exactly here) or
float arrays (widened to float64). ``scale`` is taken as given (callers pass the
float32 value the GPU uses). ``bias`` is an optional per-key additive logit term of
length T.
"""
from __future__ import annotations

import concurrent.futures as _cf

import numpy as np

__all__ = [
    "bf16_bits_to_f64", "causal_logits", "row_lse", "future_mass", "future_mass_transposed",
    "row_lse_blocked", "future_mass_blocked", "row_lse_rows", "future_mass_columns",
]


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bfloat16 bit patterns: a bf16 value is the top half of an fp32."""
    b = np.asarray(bits)
    if b.dtype != np.uint16:
        raise TypeError("expected uint16 bf16 bit patterns")
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _as_f64(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64)


def _upper_d(T: int, t: int, horizon: int) -> int:
    """Largest admissible query position for key t (inclusive)."""
    return T - 1 if horizon < 0 else min(T - 1, t + horizon)


def causal_logits(q: np.ndarray, k: np.ndarray, scale: float, bias=None) -> np.ndarray:
    """Dense logit matrix l[d, t] for one head, -inf above the diagonal (t > d).

    Eq. dense_logit_app (App. D.1): l(d, t) = <q_d, k_t> / sqrt(d_k); here the
    1/sqrt(d_k) factor is the explicit ``scale`` and an optional per-key ``bias_t``
    is added (the sink bias of the synthetic workloads).
    """
    q = _as_f64(q)
    k = _as_f64(k)
    T = q.shape[0]
    L = float(scale) * (q @ k.T)
    if bias is not None:
        L = L + _as_f64(bias)[None, :]
    L[np.triu_indices(T, k=1)] = -np.inf
    return L


def _lse_rows_of(L: np.ndarray) -> np.ndarray:
    """log sum_t exp L[d, t] per row, stabilised by the row maximum."""
    mx = np.max(L, axis=1)
    return mx + np.log(np.sum(np.exp(L - mx[:, None]), axis=1))


def _heads(Q, K):
    Q = np.asarray(Q)
    K = np.asarray(K)
    if Q.ndim != 4 or K.ndim != 4:
        raise ValueError("Q must be [B,Hq,T,D] and K [B,Hkv,T,D]")
    B, Hq, T, D = Q.shape
    if K.shape[0] != B or K.shape[2] != T or K.shape[3] != D or Hq % K.shape[1]:
        raise ValueError("shape mismatch between Q and K")
    return B, Hq, K.shape[1], T, D, Hq // K.shape[1]


def row_lse(Q, K, scale: float, bias=None) -> np.ndarray:
    """Dense causal log-normaliser LSE_d for every (b, qh, d); returns [B, Hq, T].

    Eq. dense_lse_app (App. D.1): LSE_d = log sum_{t' <= d} exp l(d, t').
    Materialises the T x T logit matrix per head (small T only).
    """
    B, Hq, Hkv, T, D, G = _heads(Q, K)
    out = np.empty((B, Hq, T), dtype=np.float64)
    for b in range(B):
        for qh in range(Hq):
            L = causal_logits(Q[b, qh], K[b, qh // G], scale, bias)
            out[b, qh] = _lse_rows_of(L)
    return out


def future_mass(Q, K, scale: float, bias=None, window: int = 0, horizon: int = -1,
                lse=None) -> np.ndarray:
    """Unnormalised future mass m_bar_t per (b, qh, t); returns [B, Hq, T].

    Eqs. causal_prob_app and future_mass_app (App. D.1): p_{d->t} = exp(l(d,t) - LSE_d)
    and m_bar_t = sum over d in [t + window, min(T-1, t + horizon)] of p_{d->t}.
    ``lse`` optionally supplies the normaliser (default: the dense one of ``row_lse``);
    keys whose query range is empty get 0.
    """
    B, Hq, Hkv, T, D, G = _heads(Q, K)
    _check_band(window, horizon)
    out = np.zeros((B, Hq, T), dtype=np.float64)
    d_idx = np.arange(T)[:, None]
    t_idx = np.arange(T)[None, :]
    band = d_idx >= t_idx + window
    if horizon >= 0:
        band &= d_idx <= t_idx + horizon
    for b in range(B):
        for qh in range(Hq):
            L = causal_logits(Q[b, qh], K[b, qh // G], scale, bias)
            l_d = _lse_rows_of(L) if lse is None else np.asarray(lse, dtype=np.float64)[b, qh]
            P = np.exp(L - l_d[:, None])          # p_{d->t}; exactly 0 above the diagonal
            out[b, qh] = np.sum(np.where(band, P, 0.0), axis=0)
    return out


def future_mass_transposed(Q, K, scale: float, bias=None, window: int = 0, horizon: int = -1) -> np.ndarray:
    """The same m_bar_t computed the transposed way of App. D.2.

    Keys become queries and queries become keys (eq. transposed_inputs_app); the
    score of transposed pair (t, d) is l(d, t) - LSE_d (eq.
    transposed_score_modifier_app); the row log-sum-exp of the transposed scores over
    the admissible d gives log m_bar_t (eq. future_mass_lse_app). Returns linear
    m_bar (exp of that log-sum-exp), 0 where the admissible range is empty.
    """
    B, Hq, Hkv, T, D, G = _heads(Q, K)
    _check_band(window, horizon)
    out = np.zeros((B, Hq, T), dtype=np.float64)
    for b in range(B):
        for qh in range(Hq):
            q = _as_f64(Q[b, qh])
            k = _as_f64(K[b, qh // G])
            L = causal_logits(q, k, scale, bias)
            lse_d = _lse_rows_of(L)
            # transposed scores: row t (original key), column d (original query)
            St = float(scale) * (k @ q.T)
            if bias is not None:
                St = St + _as_f64(bias)[:, None]
            St = St - lse_d[None, :]
            t_idx = np.arange(T)[:, None]
            d_idx = np.arange(T)[None, :]
            ok = d_idx >= t_idx + window
            if horizon >= 0:
                ok &= d_idx <= t_idx + horizon
            St = np.where(ok, St, -np.inf)
            mx = np.max(St, axis=1)
            nonempty = np.isfinite(mx)
            res = np.zeros(T)
            m = mx[nonempty]
            res[nonempty] = np.exp(m + np.log(np.sum(np.exp(St[nonempty] - m[:, None]), axis=1)))
            out[b, qh] = res
    return out


def _check_band(window: int, horizon: int) -> None:
    if window < 0:
        raise ValueError("window must be >= 0")
    if horizon >= 0 and horizon < window:
        raise ValueError("horizon must be < 0 (unbounded) or >= window")


# ---------------------------------------------------------------------------
# Blocked forms for long sequences: the same definitions, evaluated one block of
# query rows at a time so the T x T matrix is never held whole. Used on single
# (b, KV head) slices at the benchmark sizes.
# ---------------------------------------------------------------------------

def _block_logits(q_blk: np.ndarray, d0: int, k: np.ndarray, scale: float, bias, t0: int = 0) -> np.ndarray:
    """Logits for query rows d0..d0+n-1 against keys t0..d0+n-1 (causally masked)."""
    n = q_blk.shape[0]
    kk = k[t0: d0 + n]
    L = float(scale) * (q_blk @ kk.T)
    if bias is not None:
        L = L + bias[None, t0: d0 + n]
    d = d0 + np.arange(n)[:, None]
    t = t0 + np.arange(d0 + n - t0)[None, :]
    L[t > d] = -np.inf
    return L


def _map_blocks(fn, starts, threads: int):
    """fn over row-block starts, in order; on ``threads`` host threads when > 1
    (NumPy's elementwise ufuncs and BLAS release the GIL; BLAS is then held to one
    thread per block so the two levels of threading do not multiply)."""
    if threads <= 1 or len(starts) <= 1:
        return [fn(d0) for d0 in starts]
    from threadpoolctl import threadpool_limits
    with threadpool_limits(1, user_api="blas"), _cf.ThreadPoolExecutor(threads) as ex:
        return list(ex.map(fn, starts))


def row_lse_blocked(q, k, scale: float, bias=None, block: int = 1024, threads: int = 1) -> np.ndarray:
    """LSE_d for one head (q [T,D], k [T,D]), one block of query rows at a time
    (blocks are independent; ``threads`` > 1 evaluates them on that many host threads)."""
    q = _as_f64(q)
    k = _as_f64(k)
    bias = None if bias is None else _as_f64(bias)
    T = q.shape[0]
    out = np.empty(T)

    def one(d0):
        out[d0:d0 + block] = _lse_rows_of(_block_logits(q[d0:d0 + block], d0, k, scale, bias))

    _map_blocks(one, list(range(0, T, block)), threads)
    return out


def row_lse_rows(q, k, scale: float, rows, bias=None) -> np.ndarray:
    """LSE_d for selected query rows ``rows`` of one head (each O(d * D))."""
    q = _as_f64(q)
    k = _as_f64(k)
    bias = None if bias is None else _as_f64(bias)
    out = np.empty(len(rows))
    for n, d in enumerate(rows):
        l = float(scale) * (k[: d + 1] @ q[d])
        if bias is not None:
            l = l + bias[: d + 1]
        mx = np.max(l)
        out[n] = mx + np.log(np.sum(np.exp(l - mx)))
    return out


def future_mass_blocked(q, k, scale: float, bias=None, window: int = 0, horizon: int = -1,
                        lse=None, block: int = 1024, threads: int = 1) -> np.ndarray:
    """m_bar_t for one head, accumulating column sums one block of query rows at a time.

    Same definition as ``future_mass`` (eq. future_mass_app). ``lse`` (length T)
    defaults to ``row_lse_blocked``. With a finite horizon a block of rows d0.. only
    reaches keys t >= d0 - horizon, so earlier keys are not evaluated. The blocks'
    column sums are added in block order; ``threads`` > 1 evaluates the blocks on
    that many host threads.
    """
    _check_band(window, horizon)
    q = _as_f64(q)
    k = _as_f64(k)
    bias = None if bias is None else _as_f64(bias)
    T = q.shape[0]
    lse_d = row_lse_blocked(q, k, scale, bias, block, threads) if lse is None else np.asarray(lse, np.float64)

    def one(d0):
        n = min(block, T - d0)
        t0 = 0 if horizon < 0 else max(0, d0 - horizon)
        L = _block_logits(q[d0:d0 + n], d0, k, scale, bias, t0)
        P = np.exp(L - lse_d[d0:d0 + n, None])
        d = d0 + np.arange(n)[:, None]
        t = t0 + np.arange(d0 + n - t0)[None, :]
        ok = d >= t + window
        if horizon >= 0:
            ok &= d <= t + horizon
        return t0, np.sum(np.where(ok, P, 0.0), axis=0)

    out = np.zeros(T)
    starts = list(range(0, T, block))
    for d0, (t0, part) in zip(starts, _map_blocks(one, starts, threads)):
        out[t0: t0 + part.shape[0]] += part
    return out


def future_mass_columns(q, k, scale: float, cols, bias=None, window: int = 0, horizon: int = -1,
                        lse=None) -> np.ndarray:
    """m_bar_t for selected key columns ``cols`` of one head.

    Needs LSE_d for every d in each column's query range; pass ``lse`` (length T) if
    it is already known, else the needed rows are computed with ``row_lse_rows``.
    """
    _check_band(window, horizon)
    q = _as_f64(q)
    k = _as_f64(k)
    bias = None if bias is None else _as_f64(bias)
    T = q.shape[0]
    cols = [int(c) for c in cols]
    if lse is None:
        need = sorted({d for t in cols for d in range(t + window, _upper_d(T, t, horizon) + 1)})
        vals = row_lse_rows(q, k, scale, need, bias)
        lse_map = dict(zip(need, vals))
    out = np.zeros(len(cols))
    for n, t in enumerate(cols):
        lo, hi = t + window, _upper_d(T, t, horizon)
        if lo > hi:
            continue
        d = np.arange(lo, hi + 1)
        l = float(scale) * (q[d] @ k[t])
        if bias is not None:
            l = l + bias[t]
        l_d = np.asarray(lse, np.float64)[d] if lse is not None else np.array([lse_map[x] for x in d])
        out[n] = np.sum(np.exp(l - l_d))
    return out
