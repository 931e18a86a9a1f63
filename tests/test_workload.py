"""The seeded input generator: determinism, recipe properties, bf16 rounding."""
import math

import numpy as np
import pytest

import workload
from workload import gen


def test_same_seed_same_bits():
    a = workload.make("qwen3_4b_t4k", T=256)
    b = workload.make("qwen3_4b_t4k", T=256, threads=1)
    np.testing.assert_array_equal(a.q_bits, b.q_bits)
    np.testing.assert_array_equal(a.k_bits, b.k_bits)
    c = workload.make("qwen3_4b_t16k_w1024", T=256)
    assert not np.array_equal(a.k_bits, c.k_bits[:1])


def test_slice_regeneration_matches_full():
    w = workload.make("qwen3_8b_t32k", T=300, B=2)
    q, k = workload.make_slice("qwen3_8b_t32k", 1, 5, T=300)
    np.testing.assert_array_equal(w.k_bits[1, 5], k)
    np.testing.assert_array_equal(w.q_bits[1, 20:24], q)


def test_bf16_rounding_is_rne_like_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(100000) * 10.0 ** rng.integers(-6, 6, 100000)).astype(np.float32)
    x[:4] = [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.0 - 2.0 ** -8, 0.0]  # ties
    ours = workload.bf16_round_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_rmsnorm_row_norm():
    x = np.random.default_rng(0).standard_normal((64, 128)).astype(np.float32) * 7
    y = workload.rmsnorm(x)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), math.sqrt(128), rtol=1e-5)


def test_rope_preserves_norm_and_position_zero():
    x = np.random.default_rng(1).standard_normal((50, 128)).astype(np.float32)
    y = workload.rope(x)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-5)
    np.testing.assert_allclose(y[0], x[0], rtol=0, atol=0)


def test_rope_relative_position_property():
    """<rope(q)_i, rope(k)_j> depends on i - j only (same q, k at every position)."""
    rng = np.random.default_rng(2)
    q = rng.standard_normal(64).astype(np.float32)
    k = rng.standard_normal(64).astype(np.float32)
    Qr = workload.rope(np.tile(q, (40, 1)))
    Kr = workload.rope(np.tile(k, (40, 1)))
    assert float(Qr[10] @ Kr[7]) == pytest.approx(float(Qr[30] @ Kr[27]), rel=1e-4)


def test_sink_bias_and_scale():
    w = workload.make("qwen3_4b_t4k", T=128)
    assert w.bias is not None and w.bias[0] == 3.0 and np.all(w.bias[1:] == 0)
    assert w.scale == float(np.float32(1 / math.sqrt(128)))
    assert workload.make("qwen3_8b_t32k", T=128, B=1).bias is None
    assert workload.make("tiny").scale == 0.125


def test_heavy_hitters_count_and_norm():
    T = 1000
    w = workload.make("qwen3_8b_t32k", T=T, B=1)
    from oracle import bf16_bits_to_f64  # decoding only
    k = bf16_bits_to_f64(w.k_bits[0, 3])
    n = np.linalg.norm(k, axis=1)
    big = n > 2.5 * math.sqrt(128)
    assert big.sum() == math.ceil(0.01 * T)
    np.testing.assert_allclose(n[big], 4 * math.sqrt(128), rtol=2e-2)


def test_cluster_segments_shift_mixture():
    """Cluster labels follow each 8192-position segment's own mixture."""
    T = 3 * 8192
    rng = np.random.default_rng([4, 0, 0])
    mu, pis, c_k, c_q = gen.cluster_labels(rng, T, 128, 4)
    assert mu.shape == (16, 128) and pis.shape == (3, 16) and c_q.shape == (4, T)
    np.testing.assert_allclose(pis.sum(axis=1), 1.0)
    for s in range(3):
        freq = np.bincount(c_k[s * 8192:(s + 1) * 8192], minlength=16) / 8192
        assert np.max(np.abs(freq - pis[s])) < 0.03
    assert np.max(np.abs(pis[0] - pis[1])) > 0.1
    w = workload.make("long_t128k", T=2 * 8192, Hq=4, Hkv=1)
    assert w.q_bits.shape == (1, 4, 2 * 8192, 128)


def test_tiny_is_plain_normal():
    w = workload.make("tiny")
    from oracle import bf16_bits_to_f64
    q = bf16_bits_to_f64(w.q_bits)
    assert abs(q.mean()) < 0.02 and abs(q.std() - 1) < 0.02
