"""Pins of the oracle's target epilogue (App. B.1-B.2, App. D.4 step 5)."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load():
    with open(os.path.join(GOLDEN, "target_hand.json")) as f:
        return json.load(f)


def test_future_count_closed_forms():
    np.testing.assert_array_equal(oracle.future_count(5, 0, -1), [5, 4, 3, 2, 1])
    np.testing.assert_array_equal(oracle.future_count(5, 2, -1), [3, 2, 1, 1, 1])
    # lookahead L = horizon - window: at most L + 1 admissible queries
    np.testing.assert_array_equal(oracle.future_count(6, 1, 2), [2, 2, 2, 2, 1, 1])
    np.testing.assert_array_equal(oracle.future_count(4, 0, 0), [1, 1, 1, 1])


@pytest.mark.parametrize("agg", ["max", "mean"])
def test_hand_values(agg):
    g = _load()
    m = np.array([[[float(Fraction(x)) for x in row] for row in g["m_bar"]]])
    want = np.array([math.log(float(Fraction(a))) - math.log(n) for a, n in zip(g[agg], g["N"])])
    got = oracle.target_scores(m, 1, 0, -1, agg=agg, eps=0.0)
    np.testing.assert_allclose(got[0, 0], want, rtol=0, atol=1e-14)
    raw = oracle.target_scores(m, 1, 0, -1, agg=agg, eps=0.0, normalize=False)
    np.testing.assert_allclose(raw[0, 0], [math.log(float(Fraction(a))) for a in g[agg]], rtol=0, atol=1e-14)


def test_hand_masses_match_oracle_future_mass():
    """The golden m_bar rows are what the oracle's future mass gives for the two
    stated heads (checks the fixture against the pinned mass oracle)."""
    g = _load()
    Q = np.zeros((1, 1, 3, 4))
    K = np.random.default_rng(0).standard_normal((1, 1, 3, 4))
    with_bias = oracle.future_mass(Q, K, 1.0, np.array([math.log(2.0), 0.0, 0.0]))[0, 0]
    no_bias = oracle.future_mass(Q, K, 1.0)[0, 0]
    np.testing.assert_allclose(with_bias, [float(Fraction(x)) for x in g["m_bar"][0]], atol=1e-14)
    np.testing.assert_allclose(no_bias, [float(Fraction(x)) for x in g["m_bar"][1]], atol=1e-14)


@pytest.mark.parametrize("w,h", [(0, -1), (1, -1), (1, 16), (4, 9)])
def test_harmonic_target(w, h):
    """Q = 0: all heads carry the harmonic masses, so max and mean agree and
    r_t = log(H_hi - H_lo + eps) - log(max(1, band size))."""
    T, G = 64, 4
    Q = np.zeros((1, G, T, 8))
    K = np.random.default_rng(1).standard_normal((1, 1, T, 8))
    m = oracle.future_mass(Q, K, 0.3, None, w, h)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    t = np.arange(T)
    hi = np.full(T, T) if h < 0 else np.minimum(T, t + h + 1)
    lo = np.minimum(t + w, T)
    mass = np.where(lo < hi, H[hi] - H[lo], 0.0)
    n = np.maximum(1, hi - lo)
    for agg in ("max", "mean"):
        r = oracle.target_scores(m, 1, w, h, agg=agg, eps=1e-6)
        np.testing.assert_allclose(r[0, 0], np.log(mass + 1e-6) - np.log(n), rtol=0, atol=1e-12)


def test_max_is_existential_mean_is_average():
    """One head attending strongly, three not: max follows the strong head, mean
    divides its mass by G (App. B.1's existential vs shared-utility criteria)."""
    m = np.zeros((1, 4, 2))
    m[0, 2] = [0.8, 0.4]
    r_max = oracle.target_scores(m, 1, 0, -1, "max", eps=0.0, normalize=False)
    r_mean = oracle.target_scores(m, 1, 0, -1, "mean", eps=0.0, normalize=False)
    np.testing.assert_allclose(np.exp(r_max[0, 0]), [0.8, 0.4])
    np.testing.assert_allclose(np.exp(r_mean[0, 0]), [0.2, 0.1])


def test_grouping_uses_contiguous_heads():
    m = np.ones((1, 4, 3))
    m[0, 1] = 5.0  # KV head 0 (query heads 0, 1)
    m[0, 2] = 7.0  # KV head 1 (query heads 2, 3)
    r = oracle.target_scores(m, 2, 0, -1, "max", eps=0.0, normalize=False)
    np.testing.assert_allclose(np.exp(r[0]), [[5, 5, 5], [7, 7, 7]])


def test_bad_arguments():
    with pytest.raises(ValueError):
        oracle.target_scores(np.ones((1, 3, 4)), 2, 0, -1)
    with pytest.raises(ValueError):
        oracle.target_scores(np.ones((1, 2, 4)), 1, 0, -1, agg="median")
