"""Pins of the sparse attention oracle and of token lifetimes (App. C.1, C.3; Sec. 3.2).

The masked forward is checked against a library routine (PyTorch's fp64 causal
scaled-dot-product attention) when the mask is the full causal one, against
pure-Python brute force on tiny inputs, and against closed forms (constant values,
one-hot values). Lifetimes are checked by hand, against a per-entry scan of the
mask, and by rebuilding the mask from them."""
import math

import numpy as np
import pytest

import oracle


def _ranked(rng, T, s, w, k):
    rank = oracle.ranks_from_priority(rng.standard_normal(T))
    tau = oracle.running_cutoff_fenwick(rank, s, w, k)
    return rank, tau


def test_eviction_hand_case():
    """ranks (0, 3, 1, 4, 2), s=1, w=1, k=2, cutoffs (5, 5, 5, 3, 3): token 3 leaves the
    window at q=4 and its rank 4 is above the cutoff 3 there; every other token is a
    sink, stays in the top 2, or is still in the window at the last query."""
    rank = [0, 3, 1, 4, 2]
    tau = [5, 5, 5, 3, 3]
    np.testing.assert_array_equal(oracle.eviction_times(rank, tau, 1, 1), [5, 5, 5, 4, 5])
    np.testing.assert_array_equal(oracle.eviction_times_bruteforce(rank, tau, 1, 1), [5, 5, 5, 4, 5])


@pytest.mark.parametrize("seed,T,s,w,k", [(0, 40, 2, 3, 5), (1, 64, 0, 0, 1), (2, 90, 4, 8, 12), (3, 70, 5, 1, 80),
                                          (4, 50, 60, 2, 3), (5, 120, 1, 0, 7), (6, 33, 3, 40, 2)])
def test_eviction_matches_mask(seed, T, s, w, k):
    """Lifetimes from the cutoffs equal the per-entry scan of the mask, and the mask
    [t <= q < e_t] they define is the running top-k mask, entry for entry."""
    rank, tau = _ranked(np.random.default_rng(seed), T, s, w, k)
    e = oracle.eviction_times(rank, tau, s, w)
    np.testing.assert_array_equal(e, oracle.eviction_times_bruteforce(rank, tau, s, w))
    np.testing.assert_array_equal(oracle.lifetime_mask(e), oracle.running_topk_mask(rank, tau, s, w))
    rows = [0, T // 3, T - 1]
    np.testing.assert_array_equal(oracle.running_topk_mask_rows(rank, tau, s, w, rows),
                                  oracle.running_topk_mask(rank, tau, s, w)[rows])


def test_eviction_rejects_increasing_cutoffs():
    with pytest.raises(ValueError):
        oracle.eviction_times([0, 1, 2], [1, 2, 2], 0, 0)


def _f64_bits(x):
    """float64 values that are exactly representable in bf16, as bf16 bit patterns."""
    f32 = np.asarray(x, dtype=np.float32)
    return (f32.view(np.uint32) >> 16).astype(np.uint16)


def _bf16_data(rng, T, D, scale=1.0):
    return _f64_bits(np.round(rng.standard_normal((T, D)) * 8 * scale) / 8)


def test_full_causal_mask_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    T, D = 37, 16
    q, k, v = (_bf16_data(rng, T, D) for _ in range(3))
    scale = 1.0 / math.sqrt(D)
    M = np.tril(np.ones((T, T), dtype=bool))
    O, lse, A = oracle.sparse_attention(q, k, v, scale, M)
    tq, tk, tv = (torch.from_numpy(oracle.bf16_bits_to_f64(x)) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq[None], tk[None], tv[None], is_causal=True,
                                                           scale=scale)[0].numpy()
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)
    logits = (tq @ tk.T * scale).masked_fill(~torch.from_numpy(M), float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(logits, dim=1).numpy(), rtol=1e-13, atol=1e-13)
    assert np.all(A >= np.abs(O) - 1e-12)


def test_brute_force_tiny():
    """Pure-Python loops over a running top-k mask with a key bias."""
    rng = np.random.default_rng(8)
    T, D, s, w, k = 7, 3, 1, 2, 2
    q, kk, v = (_bf16_data(rng, T, D) for _ in range(3))
    bias = np.array([3.0, 0, 0.5, 0, 0, -1.0, 0])
    rank, tau = _ranked(rng, T, s, w, k)
    M = oracle.running_topk_mask(rank, tau, s, w)
    O, lse, _ = oracle.sparse_attention(q, kk, v, 0.5, M, bias)
    qf, kf, vf = (oracle.bf16_bits_to_f64(x) for x in (q, kk, v))
    for i in range(T):
        kept = [t for t in range(T) if M[i, t]]
        logit = {t: 0.5 * sum(qf[i, d] * kf[t, d] for d in range(D)) + bias[t] for t in kept}
        z = sum(math.exp(x) for x in logit.values())
        assert abs(lse[i] - math.log(z)) < 1e-12
        for d in range(D):
            o = sum(math.exp(logit[t]) / z * vf[t, d] for t in kept)
            assert abs(O[i, d] - o) < 1e-12


def test_constant_values_and_one_hot_values():
    rng = np.random.default_rng(9)
    T, D, s, w, k = 24, 32, 2, 3, 4
    q, kk = (_bf16_data(rng, T, D) for _ in range(2))
    rank, tau = _ranked(rng, T, s, w, k)
    M = oracle.running_topk_mask(rank, tau, s, w)
    # constant value rows: the output is that row for every query
    c = _f64_bits(np.tile(np.round(rng.standard_normal(D) * 4) / 4, (T, 1)))
    O, _, _ = oracle.sparse_attention(q, kk, c, 0.3, M)
    np.testing.assert_allclose(O, np.broadcast_to(oracle.bf16_bits_to_f64(c[0]), (T, D)), rtol=1e-13, atol=1e-13)
    # one-hot value rows (T <= D): the output row is the probability row itself
    eye = _f64_bits(np.eye(T, D))
    P, lse, _ = oracle.sparse_attention(q, kk, eye, 0.3, M)
    P = P[:, :T]
    np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=1e-13)
    assert np.all(P[~M] == 0) and np.all(P[M] > 0)
    qf, kf = oracle.bf16_bits_to_f64(q), oracle.bf16_bits_to_f64(kk)
    i = T - 1
    t0, t1 = np.flatnonzero(M[i])[:2]
    np.testing.assert_allclose(P[i, t0] / P[i, t1], math.exp(0.3 * (qf[i] @ kf[t0] - qf[i] @ kf[t1])), rtol=1e-12)


def test_uniform_bias_shifts_lse_only():
    rng = np.random.default_rng(10)
    T, D = 20, 8
    q, kk, v = (_bf16_data(rng, T, D) for _ in range(3))
    M = np.tril(np.ones((T, T), dtype=bool)) & (rng.random((T, T)) < 0.6)
    M[np.arange(T), np.arange(T)] = True
    O0, l0, _ = oracle.sparse_attention(q, kk, v, 0.25, M)
    O1, l1, _ = oracle.sparse_attention(q, kk, v, 0.25, M, np.full(T, 2.5))
    np.testing.assert_allclose(O1, O0, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l1, l0 + 2.5, rtol=1e-13)


def test_sparse_lse_agrees_with_sparse_row_lse():
    rng = np.random.default_rng(11)
    T, D, s, w, k = 60, 16, 3, 5, 9
    q, kk, v = (_bf16_data(rng, T, D) for _ in range(3))
    rank, tau = _ranked(rng, T, s, w, k)
    M = oracle.running_topk_mask(rank, tau, s, w)
    _, lse, _ = oracle.sparse_attention(q, kk, v, 0.25, M)
    np.testing.assert_allclose(lse, oracle.sparse_row_lse(q, kk, 0.25, M), rtol=1e-13)


def test_rejects_empty_rows():
    M = np.zeros((2, 2), dtype=bool)
    M[0, 0] = True
    with pytest.raises(ValueError):
        oracle.sparse_attention(np.zeros((2, 4)), np.zeros((2, 4)), np.zeros((2, 4)), 1.0, M)
