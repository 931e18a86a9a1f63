"""fp64 / integer oracle of KVpop's running top-k policy pieces (test infrastructure).

* static priority (App. B.3, eq. static_priority_app, decay step n = 1):
  r_bar_t = r_t - t log(gamma)
* ranks: tokens sorted once by static priority, rank 0 = highest priority; ties go to
  the earlier position (the paper does not say how ties break).
* running cutoff (App. C.2, Alg. fenwick_topk): at query q the eligible set is
  E(q) = {t : s <= t <= q - w} (Sec. 3.1 eq. eligible_set); tau_q is the rank of the
  k-th best eligible token. While |E(q)| < k every eligible token is kept; this is
  represented as tau_q = T (larger than any rank). The printed initialisation
  tau_q = -1 would instead drop them all, which contradicts the fixed budget
  B = s + w + k of Sec. 3 and App. C.1; the reading is recorded with the other
  readings of the paper.
* running top-k mask (App. C.1, eq. running_topk_mask_app):
  M[q, t] = [t < s] or [q - t < w] or ([t in E(q)] and [rank(t) <= tau_q]), t <= q.
* sparse log-normaliser (Sec. 3.2 eq. sparse_lse_main, App. D.3 eq. sparse_lse_app):
  LSE~_d = log sum_t M[d, t] exp(l(d, t)).

Two independent routes compute the cutoffs: a brute-force sort per query and a
Fenwick tree over ranks with binary lifting, written from the description of
App. C.2. Tests pin each against the other and against the budget property.
"""
from __future__ import annotations

import numpy as np

from .future_mass import _as_f64

__all__ = ["static_priority", "static_priority_f32", "ranks_from_priority", "running_cutoff_bruteforce",
           "running_cutoff_fenwick", "running_topk_mask", "sparse_row_lse", "teacher_labels"]


def static_priority(r, log_gamma: float) -> np.ndarray:
    """r_bar_t = r_t - t * log(gamma) for decay step 1 (eq. static_priority_app)."""
    r = np.asarray(r, dtype=np.float64)
    return r - np.arange(r.shape[-1], dtype=np.float64) * float(log_gamma)


def static_priority_f32(r, log_gamma: float) -> np.ndarray:
    """The same static priority evaluated in float32, one rounding per operation:
    fl(r_t - fl(t * log_gamma)). The paper computes decay and top-k ranking in
    float32 (App. F), and the ranking is an integer decided by these values, so the
    oracle takes that decision in the same precision as the GPU."""
    r32 = np.asarray(r, dtype=np.float32)
    t32 = np.arange(r32.shape[-1], dtype=np.float32)
    return r32 - t32 * np.float32(log_gamma)


def ranks_from_priority(prio) -> np.ndarray:
    """rank[t] = position of t when sorted by descending priority, ties by position."""
    prio = np.asarray(prio, dtype=np.float64)
    T = prio.shape[0]
    order = sorted(range(T), key=lambda t: (-prio[t], t))
    rank = np.empty(T, dtype=np.int64)
    for r, t in enumerate(order):
        rank[t] = r
    return rank


def running_cutoff_bruteforce(rank, s: int, w: int, k: int) -> np.ndarray:
    """tau_q by sorting the eligible ranks at every query (O(T^2 log T))."""
    rank = np.asarray(rank)
    T = rank.shape[0]
    tau = np.full(T, T, dtype=np.int64)
    for q in range(T):
        hi = q - w
        if hi < s:
            continue
        elig = np.sort(rank[s:hi + 1])
        if elig.shape[0] >= k:
            tau[q] = elig[k - 1]
    return tau


class _Fenwick:
    """Counts over ranks 0..n-1 with prefix sums and k-th-element search."""

    def __init__(self, n: int):
        self.n = n
        self.tree = [0] * (n + 1)
        self.top = 1
        while self.top * 2 <= n:
            self.top *= 2

    def add(self, i: int) -> None:
        i += 1
        while i <= self.n:
            self.tree[i] += 1
            i += i & (-i)

    def kth(self, k: int) -> int:
        """Smallest rank whose prefix count reaches k (binary lifting)."""
        pos, rem, step = 0, k, self.top
        while step:
            nxt = pos + step
            if nxt <= self.n and self.tree[nxt] < rem:
                pos = nxt
                rem -= self.tree[nxt]
            step //= 2
        return pos  # 0-based rank


def running_cutoff_fenwick(rank, s: int, w: int, k: int) -> np.ndarray:
    """tau_q by one left-to-right scan: insert rank(q - w) when it becomes eligible,
    then read the k-th smallest inserted rank (App. C.2)."""
    rank = np.asarray(rank)
    T = rank.shape[0]
    fw = _Fenwick(T)
    tau = np.full(T, T, dtype=np.int64)
    count = 0
    for q in range(T):
        t = q - w
        if t >= s:
            fw.add(int(rank[t]))
            count += 1
        if count >= k and k > 0:
            tau[q] = fw.kth(k)
    return tau


def running_topk_mask(rank, tau, s: int, w: int) -> np.ndarray:
    """Boolean [T, T] mask of eq. running_topk_mask_app (causal: t <= q)."""
    rank = np.asarray(rank)
    tau = np.asarray(tau)
    T = rank.shape[0]
    q = np.arange(T)[:, None]
    t = np.arange(T)[None, :]
    sink = t < s
    recent = (q - t) < w
    eligible = (t >= s) & (t <= q - w)
    selected = rank[None, :] <= tau[:, None]
    return (t <= q) & (sink | recent | (eligible & selected))


def sparse_row_lse(q, k, scale: float, mask, bias=None) -> np.ndarray:
    """LSE~_d = log sum_t mask[d, t] exp(l(d, t)) for one head (eq. sparse_lse_app)."""
    qv = _as_f64(q)
    kv = _as_f64(k)
    L = float(scale) * (qv @ kv.T)
    if bias is not None:
        L = L + _as_f64(bias)[None, :]
    L = np.where(np.asarray(mask, dtype=bool), L, -np.inf)
    mx = L.max(axis=1)
    return mx + np.log(np.sum(np.exp(L - mx[:, None]), axis=1))


def teacher_labels(rank, tau, s: int, w: int, queries=None):
    """Teacher label and boundary token per query (Sec. 3.1 eq. teacher_label).

    t_new = q - w is the newly eligible token; the teacher keeps the eligible tokens
    with rank <= tau_q (all of them while |E(q)| < k). y_q = +1 if t_new is kept,
    -1 otherwise; t_bnd is the kept eligible token with the largest rank (the
    boundary of the kept set). Queries with an empty eligible set get y = 0 and
    t_bnd = -1. `queries` (optional) restricts the work to those query positions;
    the others are left at y = 0, t_bnd = -1."""
    rank = np.asarray(rank)
    tau = np.asarray(tau)
    T = rank.shape[0]
    y = np.zeros(T, dtype=np.int64)
    t_bnd = np.full(T, -1, dtype=np.int64)
    for q in (range(T) if queries is None else queries):
        hi = q - w
        if hi < s:
            continue
        elig = np.arange(s, hi + 1)
        kept = elig[rank[elig] <= tau[q]]
        t_bnd[q] = kept[np.argmax(rank[kept])]
        y[q] = 1 if rank[hi] <= tau[q] else -1
    return y, t_bnd
