"""Pins of the running top-k oracle (App. B.3, App. C, App. D.3)."""
import math

import numpy as np
import pytest

import oracle


def test_static_priority_and_ranks_by_hand():
    r = np.array([1.0, 3.0, 2.0, 3.0])
    prio = oracle.static_priority(r, math.log(0.5))   # r_t + t log 2
    np.testing.assert_allclose(prio, [1.0, 3.0 + math.log(2), 2.0 + 2 * math.log(2), 3.0 + 3 * math.log(2)])
    # priorities: 1, 3.693, 3.386, 5.079 -> order t=3, 1, 2, 0
    np.testing.assert_array_equal(oracle.ranks_from_priority(prio), [3, 1, 2, 0])
    # ties go to the earlier position
    np.testing.assert_array_equal(oracle.ranks_from_priority([2.0, 5.0, 5.0, 1.0]), [2, 0, 1, 3])


def test_cutoff_hand_case():
    """s=1, w=1, k=2, ranks (0, 3, 1, 4, 2): eligible sets grow as {1}, {1,2}, ..."""
    rank = np.array([0, 3, 1, 4, 2])
    T = 5
    tau = oracle.running_cutoff_bruteforce(rank, 1, 1, 2)
    # q=0,1: E empty or {1} (size < 2) -> keep all (tau = T); q=2: E={1}: size 1 -> T
    # q=3: E={1,2} ranks {3,1} -> 2nd smallest 3; q=4: E={1,2,3} ranks {3,1,4} -> 3
    np.testing.assert_array_equal(tau, [T, T, T, 3, 3])


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("s,w,k", [(0, 1, 1), (4, 16, 8), (2, 5, 30), (1, 0, 3), (4, 64, 1)])
def test_fenwick_matches_bruteforce(seed, s, w, k):
    T = 300
    rank = np.random.default_rng(seed).permutation(T)
    np.testing.assert_array_equal(oracle.running_cutoff_fenwick(rank, s, w, k),
                                  oracle.running_cutoff_bruteforce(rank, s, w, k))


def test_cutoff_monotone_once_saturated():
    """Adding eligible tokens can only lower the k-th smallest rank."""
    T, s, w, k = 500, 4, 32, 40
    rank = np.random.default_rng(5).permutation(T)
    tau = oracle.running_cutoff_fenwick(rank, s, w, k)
    sat = tau < T
    assert np.all(np.diff(tau[sat]) <= 0)
    assert np.argmax(sat) == s + w + k - 1  # first saturated query


@pytest.mark.parametrize("s,w,k", [(4, 16, 20), (1, 8, 5), (0, 4, 12)])
def test_mask_enforces_fixed_budget(s, w, k):
    """Once q >= s + w + k - 1 every query keeps exactly B = s + w + k keys (Sec. 3
    eq. kv_budget, App. C.1); before that it keeps every key."""
    T = 200
    rank = np.random.default_rng(7).permutation(T)
    tau = oracle.running_cutoff_fenwick(rank, s, w, k)
    M = oracle.running_topk_mask(rank, tau, s, w)
    counts = M.sum(axis=1)
    q = np.arange(T)
    np.testing.assert_array_equal(counts[q >= s + w + k - 1], s + w + k)
    np.testing.assert_array_equal(counts[q < s + w + k - 1], q[q < s + w + k - 1] + 1)
    assert not np.any(np.triu(M, 1))


def test_selected_tokens_are_top_k_by_rank():
    T, s, w, k = 150, 3, 10, 7
    rank = np.random.default_rng(8).permutation(T)
    tau = oracle.running_cutoff_fenwick(rank, s, w, k)
    M = oracle.running_topk_mask(rank, tau, s, w)
    for q in range(s + w + k - 1, T):
        elig = np.arange(s, q - w + 1)
        kept = elig[M[q, elig]]
        assert len(kept) == k
        assert set(kept) == set(elig[np.argsort(rank[elig])[:k]])


def test_sparse_lse_all_ones_equals_dense_and_bounds():
    """An all-ones causal mask gives the dense LSE (App. D.3); any sub-mask gives a
    smaller normaliser, never larger."""
    rng = np.random.default_rng(9)
    T, D = 80, 16
    Q = rng.standard_normal((1, 1, T, D))
    K = rng.standard_normal((1, 1, T, D))
    full = np.tril(np.ones((T, T), dtype=bool))
    dense = oracle.row_lse(Q, K, 0.4)[0, 0]
    np.testing.assert_allclose(oracle.sparse_row_lse(Q[0, 0], K[0, 0], 0.4, full), dense, rtol=1e-14, atol=1e-14)
    rank = rng.permutation(T)
    tau = oracle.running_cutoff_fenwick(rank, 2, 8, 6)
    M = oracle.running_topk_mask(rank, tau, 2, 8)
    sp = oracle.sparse_row_lse(Q[0, 0], K[0, 0], 0.4, M)
    assert np.all(sp <= dense + 1e-12)
    # rows that keep everything match exactly
    keep_all = M.sum(axis=1) == np.arange(T) + 1
    np.testing.assert_allclose(sp[keep_all], dense[keep_all], rtol=1e-14, atol=1e-14)


def test_sparse_lse_brute_force():
    rng = np.random.default_rng(10)
    T, D = 6, 3
    q = rng.standard_normal((T, D))
    k = rng.standard_normal((T, D))
    M = np.tril(rng.random((T, T)) < 0.6)
    M[np.arange(T), np.arange(T)] = True
    got = oracle.sparse_row_lse(q, k, 0.7, M)
    for d in range(T):
        want = math.log(sum(math.exp(0.7 * float(q[d] @ k[t])) for t in range(T) if M[d, t]))
        assert got[d] == pytest.approx(want, rel=1e-13)


def test_teacher_labels_hand_case():
    """ranks (0, 3, 1, 4, 2), s=1, w=1, k=2: cutoffs (T, T, T, 3, 3).
    q=2: E={1}, kept all, t_new=1 kept (+1), boundary 1.
    q=3: E={1,2} ranks {3,1}, tau=3: both kept; t_new=2 (+1); boundary = rank 3 -> t=1.
    q=4: E={1,2,3} ranks {3,1,4}, tau=3: t_new=3 has rank 4 > 3 (-1); boundary t=1."""
    rank = np.array([0, 3, 1, 4, 2])
    tau = oracle.running_cutoff_bruteforce(rank, 1, 1, 2)
    y, tb = oracle.teacher_labels(rank, tau, 1, 1)
    np.testing.assert_array_equal(y, [0, 0, 1, 1, -1])
    np.testing.assert_array_equal(tb, [-1, -1, 1, 1, 1])


def test_teacher_labels_properties():
    T, s, w, k = 400, 4, 20, 30
    rank = np.random.default_rng(11).permutation(T)
    tau = oracle.running_cutoff_fenwick(rank, s, w, k)
    y, tb = oracle.teacher_labels(rank, tau, s, w)
    q = np.arange(T)
    assert np.all(y[q - w < s] == 0) and np.all(tb[q - w < s] == -1)
    sat = tau < T
    np.testing.assert_array_equal(rank[tb[sat]], tau[sat])          # boundary has the cutoff rank
    assert np.all(y[(q - w >= s) & ~sat] == 1)                       # budget not yet saturated
    m = (q - w >= s) & sat
    np.testing.assert_array_equal(y[m] == 1, rank[q[m] - w] <= tau[m])


def test_f32_priority_rounding_is_per_operation():
    r = np.array([1.0, 1.0, 1.0], dtype=np.float32)
    p = oracle.static_priority_f32(r, -1e-3)
    want = [np.float32(1.0) - np.float32(np.float32(t) * np.float32(-1e-3)) for t in range(3)]
    np.testing.assert_array_equal(p, np.array(want, dtype=np.float32))


def test_teacher_labels_query_subset_matches_full():
    rng = np.random.default_rng(11)
    T, s, w, k = 120, 2, 5, 9
    rank = oracle.ranks_from_priority(rng.standard_normal(T))
    tau = oracle.running_cutoff_bruteforce(rank, s, w, k)
    y, tb = oracle.teacher_labels(rank, tau, s, w)
    qs = [0, 6, 7, 30, 119]
    ys, tbs = oracle.teacher_labels(rank, tau, s, w, queries=qs)
    np.testing.assert_array_equal(ys[qs], y[qs])
    np.testing.assert_array_equal(tbs[qs], tb[qs])
    rest = np.setdiff1d(np.arange(T), qs)
    assert np.all(ys[rest] == 0) and np.all(tbs[rest] == -1)
