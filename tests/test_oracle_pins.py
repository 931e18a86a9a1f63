"""Pins of the fp64 oracle against facts fixed by the paper's definitions.

None of these checks re-evaluates the oracle's own formula: each compares it with
something computed another way -- exact fractions enumerated by hand, closed forms
(harmonic numbers, prefix sums), pure-Python brute force written from the
definitions, invariants (rows of a softmax sum to 1), or a library routine.
Definitions: KVpop App. D.1 (eqs. dense_logit_app, dense_lse_app, causal_prob_app,
future_mass_app), App. D.2 (transposed form), App. B.2 (lookahead clip).
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
BANDS = [(0, -1), (1, -1), (1, 1), (1, 5), (0, 0), (3, 7), (0, 4), (2, 2)]


def _frac(s):
    if s == "ln2":
        return math.log(2.0)
    if s == "ln3":
        return math.log(3.0)
    if s == "ln4":
        return math.log(4.0)
    return float(Fraction(s))


def _harm(n):
    """H_n = sum_{k=1}^n 1/k with exact rationals, converted once (n small)."""
    return float(sum((Fraction(1, k) for k in range(1, n + 1)), Fraction(0)))


def _harm_vec(n_max):
    h = np.zeros(n_max + 1)
    acc = Fraction(0)
    for k in range(1, n_max + 1):
        acc += Fraction(1, k)
        h[k] = float(acc)
    return h


def _qk(B, Hq, Hkv, T, D, seed, q_zero=False):
    rng = np.random.default_rng(seed)
    Q = np.zeros((B, Hq, T, D)) if q_zero else rng.standard_normal((B, Hq, T, D))
    K = rng.standard_normal((B, Hkv, T, D))
    return Q, K


# ---------------------------------------------------------------------------
# bf16 decoding
# ---------------------------------------------------------------------------

def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x7F80, 0xFF80, 0x3F81, 0x0001, 0x4049],
                    dtype=np.uint16)
    want = [1.0, -2.0, 0.0, -0.0, math.inf, -math.inf, 1.0 + 2.0 ** -7, 2.0 ** -133, 3.140625]
    got = oracle.bf16_bits_to_f64(bits)
    for g, w in zip(got, want):
        assert g == w
    assert math.copysign(1.0, got[3]) == -1.0


def test_bf16_decode_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 0x7F80, size=4096, dtype=np.uint16)  # finite positives
    bits = np.concatenate([bits, bits | np.uint16(0x8000)])
    t = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.bf16_bits_to_f64(bits), t)


# ---------------------------------------------------------------------------
# hand enumeration (T = 3) -- tests/golden/t3_hand.json
# ---------------------------------------------------------------------------

def _t3_inputs():
    with open(os.path.join(GOLDEN, "t3_hand.json")) as f:
        g = json.load(f)
    T, D = g["T"], g["D"]
    Q = np.zeros((1, 1, T, D))
    K = np.random.default_rng(0).standard_normal((1, 1, T, D))
    bias = np.array([_frac(s) for s in g["bias"]])
    return g, Q, K, bias


def test_hand_t3_lse():
    g, Q, K, bias = _t3_inputs()
    lse = oracle.row_lse(Q, K, 0.5, bias)[0, 0]
    np.testing.assert_allclose(lse, [_frac(s) for s in g["lse"]], rtol=0, atol=1e-14)


@pytest.mark.parametrize("fn", ["future_mass", "future_mass_transposed", "blocked", "columns"])
def test_hand_t3_future_mass(fn):
    g, Q, K, bias = _t3_inputs()
    for case in g["cases"]:
        w, h = case["window"], case["horizon"]
        want = np.array([_frac(s) for s in case["out"]])
        if fn == "future_mass":
            got = oracle.future_mass(Q, K, 0.5, bias, w, h)[0, 0]
        elif fn == "future_mass_transposed":
            got = oracle.future_mass_transposed(Q, K, 0.5, bias, w, h)[0, 0]
        elif fn == "blocked":
            got = oracle.future_mass_blocked(Q[0, 0], K[0, 0], 0.5, bias, w, h, block=2)
        else:
            got = oracle.future_mass_columns(Q[0, 0], K[0, 0], 0.5, [0, 1, 2], bias, w, h)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-14, err_msg=f"{fn} band {(w, h)}")


def test_t1_single_token():
    Q = np.random.default_rng(1).standard_normal((1, 1, 1, 8))
    K = np.random.default_rng(2).standard_normal((1, 1, 1, 8))
    b = np.array([0.75])
    assert oracle.future_mass(Q, K, 0.3, b)[0, 0, 0] == pytest.approx(1.0, abs=1e-15)
    lse = oracle.row_lse(Q, K, 0.3, b)[0, 0, 0]
    assert lse == pytest.approx(0.3 * float(Q[0, 0, 0] @ K[0, 0, 0]) + 0.75, abs=1e-14)
    assert oracle.future_mass(Q, K, 0.3, b, window=1)[0, 0, 0] == 0.0


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("w,h", BANDS)
def test_harmonic_closed_form_q_zero(w, h):
    """Q = 0: every row is uniform, p_{d->t} = 1/(d+1), so
    m_t = H_{min(T, t+h+1)} - H_{t+w} (H_n the harmonic numbers)."""
    T = 97
    Q, K = _qk(1, 2, 1, T, 16, 3, q_zero=True)
    H = _harm_vec(T + 1)
    t = np.arange(T)
    hi = np.full(T, T) if h < 0 else np.minimum(T, t + h + 1)
    lo = t + w
    want = np.where(lo < hi, H[np.minimum(hi, T)] - H[np.minimum(lo, T)], 0.0)
    got = oracle.future_mass(Q, K, 0.125, None, w, h)
    np.testing.assert_allclose(got[0, 0], want, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(got[0, 1], want, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(oracle.row_lse(Q, K, 0.125)[0, 0], np.log(t + 1.0), rtol=0, atol=1e-13)


def test_harmonic_spot_values_t512():
    """Full future at T = 512 with Q = 0: m_0 = H_512 and m_511 = 1/512."""
    T = 512
    Q, K = _qk(1, 1, 1, T, 8, 4, q_zero=True)
    got = oracle.future_mass_blocked(Q[0, 0], K[0, 0], 0.125, block=100)
    assert got[0] == pytest.approx(_harm(512), rel=1e-13)
    assert got[0] == pytest.approx(6.816516534549, rel=1e-11)
    assert got[511] == pytest.approx(1.0 / 512.0, rel=1e-13)


def test_constant_keys_reduce_to_harmonic():
    """All keys equal: each row's logits are constant, rows uniform whatever Q is."""
    T = 64
    rng = np.random.default_rng(5)
    Q = rng.standard_normal((1, 1, T, 16)) * 3.0
    K = np.broadcast_to(rng.standard_normal(16), (1, 1, T, 16)).copy()
    H = _harm_vec(T)
    got = oracle.future_mass(Q, K, 0.7)[0, 0]
    np.testing.assert_allclose(got, H[T] - H[np.arange(T)], rtol=1e-12)


@pytest.mark.parametrize("w,h", BANDS)
@pytest.mark.parametrize("with_bias", [False, True])
def test_constant_query_prefix_closed_form(w, h, with_bias):
    """All queries equal (q_d = q): logits a_t = scale <q, k_t> + bias_t do not depend
    on d, so p_{d->t} = e^{a_t} / Z_d with Z_d = sum_{t' <= d} e^{a_t'}, and
    m_t = e^{a_t} * sum_{d in band(t)} 1 / Z_d -- evaluated with prefix sums."""
    T, D, scale = 150, 32, 0.3
    rng = np.random.default_rng(11)
    q = rng.standard_normal(D)
    K = rng.standard_normal((1, 1, T, D))
    Q = np.broadcast_to(q, (1, 1, T, D)).copy()
    bias = rng.standard_normal(T) * 2.0 if with_bias else None
    a = scale * (K[0, 0] @ q) + (bias if with_bias else 0.0)
    Z = np.cumsum(np.exp(a))
    invZ_prefix = np.concatenate([[0.0], np.cumsum(1.0 / Z)])  # sum_{d < n} 1/Z_d
    t = np.arange(T)
    lo = t + w
    hi = np.full(T, T - 1) if h < 0 else np.minimum(T - 1, t + h)
    want = np.where(lo <= hi, np.exp(a) * (invZ_prefix[np.minimum(hi + 1, T)] - invZ_prefix[np.minimum(lo, T)]), 0)
    got = oracle.future_mass(Q, K, scale, bias, w, h)[0, 0]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(oracle.row_lse(Q, K, scale, bias)[0, 0], np.log(Z), rtol=1e-13)


def test_sink_bias_closed_form():
    """Q = 0 and bias = 3 on key 0 only: m_0 = sum_d e^3 / (e^3 + d)."""
    T = 300
    Q, K = _qk(1, 1, 1, T, 8, 6, q_zero=True)
    bias = np.zeros(T)
    bias[0] = 3.0
    e3 = math.exp(3.0)
    want0 = sum(e3 / (e3 + d) for d in range(T))
    got = oracle.future_mass(Q, K, 0.1, bias)[0, 0]
    assert got[0] == pytest.approx(want0, rel=1e-13)
    # any other key t: sum_{d >= t} 1 / (e^3 + d)
    assert got[5] == pytest.approx(sum(1.0 / (e3 + d) for d in range(5, T)), rel=1e-13)


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def test_row_sums_give_query_count():
    """Each query row's probabilities sum to 1, so summing the full-future mass
    (window 0, no horizon) over all keys gives T (App. D.1 eq. causal_prob_app)."""
    T = 200
    Q, K = _qk(2, 4, 2, T, 32, 8)
    bias = np.random.default_rng(9).standard_normal(T)
    got = oracle.future_mass(Q * 2.0, K, 0.25, bias)
    np.testing.assert_allclose(got.sum(axis=-1), T, rtol=1e-12)


def test_band_additivity():
    """Bands split the query range: (w, -1) = (w, h) + (h + 1, -1)."""
    T = 120
    Q, K = _qk(1, 2, 1, T, 16, 10)
    f = lambda w, h: oracle.future_mass(Q, K, 0.4, None, w, h)
    for w, h in [(0, 0), (0, 7), (1, 1), (3, 40), (1, 1024)]:
        np.testing.assert_allclose(f(w, -1), f(w, h) + f(h + 1, -1), rtol=1e-12, atol=1e-300)


def test_gqa_head_mapping_contiguous_groups():
    """Query head qh reads KV head qh // G: give KV head 0 constant keys (uniform
    rows, harmonic masses) and KV head 1 random keys; with G = 2 the query heads
    0 and 1 must show the harmonic masses and heads 2 and 3 must not."""
    T, D = 64, 16
    rng = np.random.default_rng(12)
    Q = rng.standard_normal((1, 4, T, D)) * 2
    K = np.empty((1, 2, T, D))
    K[0, 0] = rng.standard_normal(D)
    K[0, 1] = rng.standard_normal((T, D)) * 2
    H = _harm_vec(T)
    want = H[T] - H[np.arange(T)]
    got = oracle.future_mass(Q, K, 0.5)
    for qh in (0, 1):
        np.testing.assert_allclose(got[0, qh], want, rtol=1e-12)
    for qh in (2, 3):
        assert np.max(np.abs(got[0, qh] - want)) > 0.1


def test_batch_rows_independent_and_head_permutation():
    T = 40
    Q, K = _qk(2, 4, 2, T, 16, 13)
    full = oracle.future_mass(Q, K, 0.5)
    one = oracle.future_mass(Q[1:], K[1:], 0.5)
    np.testing.assert_array_equal(full[1:], one)
    perm = [1, 0, 3, 2]
    np.testing.assert_array_equal(oracle.future_mass(Q[:, perm], K, 0.5), full[:, perm])


def test_diagonal_dominant_limit():
    """q_d = k_d = c e_{d mod D} with large c: each query attends (almost) only to
    itself, so m_t -> 1 for window 0 and -> 0 for window 1."""
    T, D, c = 32, 64, 12.0
    E = np.zeros((1, 1, T, D))
    E[0, 0, np.arange(T), np.arange(T) % D] = c
    m0 = oracle.future_mass(E, E, 1.0, None, 0, -1)[0, 0]
    m1 = oracle.future_mass(E, E, 1.0, None, 1, -1)[0, 0]
    assert np.all(np.abs(m0 - 1.0) < 1e-40 + T * math.exp(-c * c))
    assert np.all(m1 < T * math.exp(-c * c))


# ---------------------------------------------------------------------------
# brute force from the definitions (pure Python, tiny T)
# ---------------------------------------------------------------------------

def _brute(q, k, scale, bias, w, h):
    T = len(q)
    logit = lambda d, t: scale * sum(a * b for a, b in zip(q[d], k[t])) + (bias[t] if bias is not None else 0.0)
    lse = [math.log(sum(math.exp(logit(d, t)) for t in range(d + 1))) for d in range(T)]
    out = []
    for t in range(T):
        s = 0.0
        for d in range(T):
            if d >= t + w and (h < 0 or d <= t + h) and t <= d:
                s += math.exp(logit(d, t) - lse[d])
        out.append(s)
    return lse, out


@pytest.mark.parametrize("T", [1, 2, 5, 8])
@pytest.mark.parametrize("w,h", [(0, -1), (1, -1), (1, 1), (0, 2), (2, 3)])
def test_brute_force_tiny(T, w, h):
    rng = np.random.default_rng(100 + T)
    D = 4
    Q = rng.standard_normal((1, 2, T, D)) * 1.5
    K = rng.standard_normal((1, 1, T, D)) * 1.5
    bias = rng.standard_normal(T)
    for qh in range(2):
        lse_b, out_b = _brute(Q[0, qh].tolist(), K[0, 0].tolist(), 0.6, bias.tolist(), w, h)
        np.testing.assert_allclose(oracle.row_lse(Q, K, 0.6, bias)[0, qh], lse_b, rtol=1e-13)
        np.testing.assert_allclose(oracle.future_mass(Q, K, 0.6, bias, w, h)[0, qh], out_b, rtol=1e-12, atol=1e-300)


# ---------------------------------------------------------------------------
# the oracle's alternative evaluation routes agree
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("w,h", BANDS)
def test_transposed_blocked_columns_agree(w, h):
    T = 203
    Q, K = _qk(1, 1, 1, T, 32, 14)
    bias = np.random.default_rng(15).standard_normal(T)
    ref = oracle.future_mass(Q, K, 0.35, bias, w, h)[0, 0]
    np.testing.assert_allclose(oracle.future_mass_transposed(Q, K, 0.35, bias, w, h)[0, 0], ref, rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(oracle.future_mass_blocked(Q[0, 0], K[0, 0], 0.35, bias, w, h, block=64), ref,
                               rtol=1e-12, atol=1e-300)
    cols = [0, 1, 63, 64, 100, 201, 202]
    np.testing.assert_allclose(oracle.future_mass_columns(Q[0, 0], K[0, 0], 0.35, cols, bias, w, h), ref[cols],
                               rtol=1e-12, atol=1e-300)
    lse_b = oracle.row_lse_blocked(Q[0, 0], K[0, 0], 0.35, bias, block=50)
    np.testing.assert_allclose(lse_b, oracle.row_lse(Q, K, 0.35, bias)[0, 0], rtol=1e-13, atol=1e-14)
    # the same blocks on several host threads
    np.testing.assert_allclose(oracle.row_lse_blocked(Q[0, 0], K[0, 0], 0.35, bias, block=50, threads=3), lse_b,
                               rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(oracle.future_mass_blocked(Q[0, 0], K[0, 0], 0.35, bias, w, h, block=32, threads=4),
                               ref, rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(oracle.row_lse_rows(Q[0, 0], K[0, 0], 0.35, [0, 7, 202], bias), lse_b[[0, 7, 202]],
                               rtol=1e-13, atol=1e-14)


def test_external_lse_is_used():
    """Supplying a shifted normaliser scales every summand by exp(-shift)."""
    T = 50
    Q, K = _qk(1, 1, 1, T, 8, 16)
    lse = oracle.row_lse(Q, K, 0.5)
    a = oracle.future_mass(Q, K, 0.5, None, 0, -1, lse=lse)
    b = oracle.future_mass(Q, K, 0.5, None, 0, -1, lse=lse + 0.5)
    np.testing.assert_allclose(b, a * math.exp(-0.5), rtol=1e-13)


def test_invalid_bands_rejected():
    Q, K = _qk(1, 1, 1, 4, 4, 17)
    with pytest.raises(ValueError):
        oracle.future_mass(Q, K, 1.0, None, -1, -1)
    with pytest.raises(ValueError):
        oracle.future_mass(Q, K, 1.0, None, 3, 2)
