"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Bar (per query head and key): |gpu - oracle| <= 2e-3 * oracle for every key whose
query range is non-empty, exactly 0 for keys whose range is empty; the pass-1 LSE
within 5e-4 absolute. Inputs are the same bf16 bit patterns on both sides, from
the seeded generator in ``workload``.
"""
import math
import os

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu

REL = 2e-3
LSE_ABS = 5e-4
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))  # host threads for the blocked oracle


def _dev(bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _run(w: workload.Workload, window: int, horizon: int, bias=None):
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    b = None
    bias = w.bias if bias is None else bias
    if bias is not None:
        b = torch.from_numpy(np.ascontiguousarray(bias, dtype=np.float32)).to("cuda")
    out, lse = kv.kvpop_future_attn_target(q, k, w.scale, window, horizon, key_bias=b)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def _empty_mask(T: int, window: int) -> np.ndarray:
    return np.arange(T) + window > T - 1


def _check_out(got, ref, window, what=""):
    T = got.shape[-1]
    empty = _empty_mask(T, window)
    assert np.all(got[..., empty] == 0.0), what + ": keys with an empty query range must be exactly 0"
    g, r = got[..., ~empty], ref[..., ~empty]
    assert np.all(r > 1e-30), what + ": oracle value below the relative-error floor"
    rel = np.abs(g - r) / r
    worst = np.unravel_index(np.argmax(rel), rel.shape) if rel.size else None
    assert rel.size == 0 or rel.max() <= REL, "%s: max rel err %.3e at %s (gpu %r, oracle %r)" % (
        what, rel.max(), worst, g[worst], r[worst])


def _check_lse(got, ref, what=""):
    err = np.abs(got - ref)
    assert err.max() <= LSE_ABS, "%s: lse max abs err %.3e" % (what, err.max())


def _cfg(B, Hq, Hkv, T, D, seed, kind="normal", sink=False):
    return dict(seed=seed, B=B, Hq=Hq, Hkv=Hkv, T=T, D=D, scale=1.0 / math.sqrt(D), kind=kind, sink=sink,
                bands=[(0, -1)])


# ---------------------------------------------------------------------------
# small and ragged shapes, every band type, against the materialising oracle
# ---------------------------------------------------------------------------

SHAPES = [
    # B, Hq, Hkv, T, D
    (1, 1, 1, 1, 64),
    (1, 1, 1, 2, 128),
    (1, 2, 1, 3, 64),
    (1, 4, 2, 17, 128),
    (3, 4, 4, 63, 64),
    (1, 8, 1, 64, 128),
    (2, 4, 1, 65, 128),
    (1, 2, 2, 127, 64),
    (1, 8, 2, 129, 128),
    (1, 6, 2, 200, 128),
    (1, 5, 1, 100, 64),
    (1, 16, 1, 96, 128),
    (3, 4, 1, 1000, 128),
    (1, 8, 4, 1000, 64),
    (1, 4, 1, 1537, 128),
]
BANDS = [(0, -1), (1, -1), (1, 1), (1, 1024), (256, -1), (0, 5), (3, 70), (0, 0)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dHq%dHkv%dT%dD%d" % s)
def test_shapes_all_bands(shape):
    B, Hq, Hkv, T, D = shape
    w = workload.make(_cfg(B, Hq, Hkv, T, D, seed=T * 7 + Hq))
    lse_ref = oracle.row_lse(w.q_bits, w.k_bits, w.scale)
    for window, horizon in BANDS:
        out, lse = _run(w, window, horizon)
        _check_lse(lse, lse_ref, "shape %s" % (shape,))
        ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, None, window, horizon, lse=lse_ref)
        _check_out(out, ref, window, "shape %s band %s" % (shape, (window, horizon)))


BAND_PAIRS = [((0, -1), (1, 1024)), ((1, 1), (0, 5)), ((256, -1), (0, -1)), ((3, 70), (0, 0)), ((1, 40), (1, 40))]


@pytest.mark.parametrize("shape", [SHAPES[i] for i in (3, 6, 8, 12, 13, 14)], ids=lambda s: "B%dHq%dHkv%dT%dD%d" % s)
def test_two_bands_one_sweep(shape):
    """kvpop_future_attn_bands: both bands from one sweep, each against the oracle,
    and against kvpop_future_attn_from_lse on that band alone (same terms, up to the
    fp32 summation order)."""
    B, Hq, Hkv, T, D = shape
    w = workload.make(_cfg(B, Hq, Hkv, T, D, seed=T * 3 + Hq, kind="rope", sink=True))
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    bias = torch.from_numpy(w.bias).to("cuda")
    lse = kv.kvpop_row_lse(q, k, w.scale, key_bias=bias)
    lse_ref = oracle.row_lse(w.q_bits, w.k_bits, w.scale, w.bias)
    for bands in BAND_PAIRS:
        outs = kv.kvpop_future_attn_bands(q, k, lse, w.scale, bands, key_bias=bias)
        singles = [kv.kvpop_future_attn_from_lse(q, k, lse, w.scale, a, h, key_bias=bias) for a, h in bands]
        torch.cuda.synchronize()
        for (a, h), o, s1 in zip(bands, outs, singles):
            got = o.cpu().numpy().astype(np.float64)
            ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, a, h, lse=lse_ref)
            _check_out(got, ref, a, "shape %s bands %s band %s" % (shape, bands, (a, h)))
            np.testing.assert_allclose(got, s1.cpu().numpy(), rtol=1e-5, atol=0)
        # the order the bands are given in changes nothing, bit for bit
        rev = kv.kvpop_future_attn_bands(q, k, lse, w.scale, bands[::-1], key_bias=bias)
        torch.cuda.synchronize()
        for o, r in zip(outs, rev[::-1]):
            np.testing.assert_array_equal(o.cpu().numpy(), r.cpu().numpy())


@pytest.mark.parametrize("T", [5, 130, 700])
def test_random_bias_and_masked_keys(T):
    """Random per-key bias, with every 7th key (from key 1 on) at -inf: masked keys
    get exactly 0, all others the oracle's value within the relative bar."""
    w = workload.make(_cfg(1, 4, 2, T, 128, seed=31 + T, kind="rope"))
    rng = np.random.default_rng(T)
    bias = rng.standard_normal(T).astype(np.float32) * 2
    masked = np.zeros(T, bool)
    masked[1::7] = True
    bias[masked] = -np.inf
    lse_ref = oracle.row_lse(w.q_bits, w.k_bits, w.scale, bias)
    for window, horizon in [(0, -1), (1, 3), (2, -1)]:
        out, lse = _run(w, window, horizon, bias=bias)
        _check_lse(lse, lse_ref, "bias")
        ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, bias, window, horizon, lse=lse_ref)
        assert np.all(out[..., masked] == 0.0)
        keep = ~masked
        live = keep & ~_empty_mask(T, window)
        assert np.all(out[..., ~live] == 0.0)
        rel = np.abs(out[..., live] - ref[..., live]) / ref[..., live]
        assert rel.max() <= REL, "bias band %s: max rel err %.3e" % ((window, horizon), rel.max())


@pytest.mark.parametrize("T,D", [(1000, 128), (2100, 64)])
def test_logits_far_above_the_diagonal_reference(T, D):
    """Pass 1 takes its reference maximum from the tiles on a query block's diagonal
    and sums later tiles against it; a tile whose terms exceed 2^64 is redone
    exactly. Here key 0 carries a bias of +60 and keys T/2 .. T/2+4 one of +45
    (N(0,1) inputs keep the other logits within a few units), so every query block
    that reaches those keys below its diagonal sees terms about 2^87 and 2^65 above
    its reference and takes the redo. LSE and future mass must still match the
    oracle, on every key (the unbiased keys' masses are about e^-60)."""
    w = workload.make(_cfg(1, 8, 2, T, D, seed=77 + T))
    bias = np.zeros(T, np.float32)
    bias[0] = 60.0
    bias[T // 2:T // 2 + 5] = 45.0
    lse_ref = oracle.row_lse(w.q_bits, w.k_bits, w.scale, bias)
    for window, horizon in [(0, -1), (1, 256)]:
        out, lse = _run(w, window, horizon, bias=bias)
        _check_lse(lse, lse_ref, "large bias")
        ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, bias, window, horizon, lse=lse_ref)
        _check_out(out, ref, window, "large bias band %s" % ((window, horizon),))


@pytest.mark.parametrize("shape", [(1, 32, 8, 2048), (1, 32, 8, 4096), (8, 8, 2, 4100), (9, 8, 2, 4100)],
                         ids=lambda s: "B%dHq%dHkv%dT%d" % s)
def test_pass1_block_forms(shape):
    """Pass 1 has four launch forms, by grid size (P = 4 query heads per workgroup,
    full-height blocks of 64 queries, 256 CUs):
      B=1, 32/8, T=2048: 256 full-height blocks fit on the CUs one each, so 512
        half-height blocks (NQ = 2, 4 waves), and the grid holds two per CU: heavy
        and light blocks paired on each CU;
      B=1, 32/8, T=4096: 512 full-height blocks as 8 waves of 2 subtiles, paired;
      B=8, 8/2, T=4100: NQ = 4, 1040 blocks, heaviest first;
      B=9, 8/2, T=4100: NQ = 4, 1170 blocks, heaviest first, a grid that is not a
        multiple of the workgroups per CU.
    Key 0 carries a bias of +60 and keys T/2 .. T/2+4 one of +45, so every form
    also takes the exact redo of off-diagonal steps. Every LSE row of eight query
    heads (all KV heads, first and last batch row) must match the oracle."""
    B, Hq, Hkv, T = shape
    D = 128
    w = workload.make(_cfg(B, Hq, Hkv, T, D, seed=900 + B + T))
    bias = np.zeros(T, np.float32)
    bias[0] = 60.0
    bias[T // 2:T // 2 + 5] = 45.0
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    bd = torch.from_numpy(bias).to("cuda")
    lse = kv.kvpop_row_lse(q, k, w.scale, key_bias=bd).cpu().numpy().astype(np.float64)
    heads = sorted({(b, qh) for b in (0, B - 1) for qh in range(0, Hq, max(1, Hq // 4))} | {(B - 1, Hq - 1)})
    for b, qh in heads:
        ref = oracle.row_lse_blocked(w.q_bits[b, qh], w.k_bits[b, qh // w.G], w.scale, bias, block=512,
                                     threads=THREADS)
        _check_lse(lse[b, qh], ref, "b%d qh%d" % (b, qh))


def test_tiny_config():
    """T=512, one head, D=64, N(0,1) inputs, scale 1/8, full future (window 0)."""
    w = workload.make("tiny")
    out, lse = _run(w, 0, -1)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale)
    _check_lse(lse, oracle.row_lse(w.q_bits, w.k_bits, w.scale), "tiny")
    _check_out(out, ref, 0, "tiny")
    assert out.sum() == pytest.approx(512.0, rel=1e-4)


def test_window_beyond_sequence_gives_zeros():
    w = workload.make(_cfg(1, 2, 1, 100, 128, seed=5))
    for window, horizon in [(100, -1), (150, 200), (99, 99)]:
        out, _ = _run(w, window, horizon)
        if window >= 100:
            assert np.all(out == 0.0)
        else:
            assert np.all(out[..., 1:] == 0.0) and np.all(out[..., 0] > 0)


# ---------------------------------------------------------------------------
# the benchmark workloads
# ---------------------------------------------------------------------------

def test_qwen3_4b_t4k_sink():
    """Qwen3-4B shape, T=4096, sink bias on key 0, full future: one query head per KV
    head (covering every g) against the blocked oracle, all heads by the row sum."""
    w = workload.make("qwen3_4b_t4k")
    out, lse = _run(w, 0, -1)
    np.testing.assert_allclose(out.sum(axis=-1), w.T, rtol=REL)
    for h in range(w.Hkv):
        qh = h * w.G + h % w.G
        q, k = w.q_bits[0, qh], w.k_bits[0, h]
        lse_ref = oracle.row_lse_blocked(q, k, w.scale, w.bias)
        _check_lse(lse[0, qh], lse_ref, "4k head %d" % qh)
        ref = oracle.future_mass_blocked(q, k, w.scale, w.bias, 0, -1, lse=lse_ref)
        _check_out(out[0, qh], ref, 0, "4k head %d" % qh)


def test_qwen3_4b_w1024_band():
    """Finite horizon W=1024 (j < i <= j + W) with the sink, on a 4096-token cut of
    the T=16384, B=2 workload (same recipe and seed) against the blocked oracle."""
    w = workload.make("qwen3_4b_t16k_w1024", T=4096, B=1)
    out, lse = _run(w, 1, 1024)
    for qh in (0, 13, 31):
        q, k = w.q_bits[0, qh], w.k_bits[0, qh // w.G]
        lse_ref = oracle.row_lse_blocked(q, k, w.scale, w.bias)
        ref = oracle.future_mass_blocked(q, k, w.scale, w.bias, 1, 1024, lse=lse_ref)
        _check_out(out[0, qh], ref, 1, "w1024 head %d" % qh)


def test_qwen3_4b_w1024_full_size_sampled():
    """Full T=16384, B=2 W=1024 workload: sampled keys against the oracle's columns."""
    w = workload.make("qwen3_4b_t16k_w1024")
    out, lse = _run(w, 1, 1024)
    rng = np.random.default_rng(0)
    for b, qh in [(0, 3), (1, 30)]:
        q, k = w.q_bits[b, qh], w.k_bits[b, qh // w.G]
        cols = sorted(set(rng.integers(0, w.T, 6).tolist()) | {0, 1, w.T - 1025, w.T - 2, w.T - 1})
        ref = oracle.future_mass_columns(q, k, w.scale, cols, w.bias, 1, 1024)
        got = out[b, qh, cols]
        for c, g, r in zip(cols, got, ref):
            if c + 1 > w.T - 1:
                assert g == 0.0
            else:
                assert abs(g - r) <= REL * r, (b, qh, c, g, r)
        rows = rng.integers(0, w.T, 8).tolist()
        np.testing.assert_allclose(lse[b, qh, rows], oracle.row_lse_rows(q, k, w.scale, rows, w.bias), atol=LSE_ABS,
                                   rtol=0)


def test_qwen3_4b_w1024_full_size_one_head_exhaustive():
    """Full T=16384, B=2 W=1024 workload with the sink: every key and every LSE row
    of one (b, query head) against the blocked oracle."""
    w = workload.make("qwen3_4b_t16k_w1024")
    out, lse = _run(w, 1, 1024)
    b, qh = 1, 22
    q, k = w.q_bits[b, qh], w.k_bits[b, qh // w.G]
    lse_ref = oracle.row_lse_blocked(q, k, w.scale, w.bias, threads=THREADS)
    _check_lse(lse[b, qh], lse_ref, "16k W=1024 b%d qh%d" % (b, qh))
    ref = oracle.future_mass_blocked(q, k, w.scale, w.bias, 1, 1024, lse=lse_ref, threads=THREADS)
    _check_out(out[b, qh], ref, 1, "16k W=1024 b%d qh%d" % (b, qh))


def test_qwen3_8b_t32k_full_scale():
    """Qwen3-8B shape at T=32768, B=4, heavy hitters: the full workload on the GPU,
    every head by the row sum, sampled LSE rows and the last keys of several heads
    against the oracle."""
    w = workload.make("qwen3_8b_t32k")
    out, lse = _run(w, 0, -1)
    np.testing.assert_allclose(out.sum(axis=-1), w.T, rtol=REL)
    rng = np.random.default_rng(1)
    for b, qh in [(0, 0), (1, 9), (2, 22), (3, 31)]:
        q, k = w.q_bits[b, qh], w.k_bits[b, qh // w.G]
        rows = sorted(rng.integers(0, w.T, 6).tolist() + [0, w.T - 1])
        np.testing.assert_allclose(lse[b, qh, rows], oracle.row_lse_rows(q, k, w.scale, rows), atol=LSE_ABS, rtol=0)
        cols = list(range(w.T - 40, w.T))
        ref = oracle.future_mass_columns(q, k, w.scale, cols)
        _check_out(out[b, qh, cols][None], ref[None], 0, "32k b%d qh%d tail" % (b, qh))


def test_groups_taken_in_batches_per_xcd():
    """64 (b, KV head) groups give each XCD 8 groups; with 32 key blocks of 256 each
    XCD then runs them 4 at a time, one batch after the other. Every key column of
    every head must be written exactly once (the output starts as NaN), the masses
    of each head must sum to T (each query's probabilities sum to 1), and the first
    and last heads must match the oracle on every key."""
    B, H, T, D = 8, 8, 8000, 64
    w = workload.make(dict(seed=404, B=B, Hq=H, Hkv=H, T=T, D=D, scale=1.0 / math.sqrt(D), kind="rope",
                           sink=False, bands=[(0, -1)]))
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    out = torch.full((B, H, T), float("nan"), device="cuda")
    lse = torch.empty((B, H, T), device="cuda")
    kv.kvpop_future_attn_target(q, k, w.scale, 0, -1, lse_ws=lse, out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    np.testing.assert_allclose(got.sum(axis=-1), T, rtol=REL)
    for b, qh in [(0, 0), (B - 1, H - 1)]:
        lse_ref = oracle.row_lse_blocked(w.q_bits[b, qh], w.k_bits[b, qh], w.scale)
        _check_lse(lse[b, qh].cpu().numpy().astype(np.float64), lse_ref, "batches b%d h%d" % (b, qh))
        ref = oracle.future_mass_blocked(w.q_bits[b, qh], w.k_bits[b, qh], w.scale, None, 0, -1, lse=lse_ref)
        _check_out(got[b, qh], ref, 0, "batches b%d h%d" % (b, qh))
    # The fused epilogue takes the same launch order; with one query head per KV head
    # its mean score is log(mass + eps) - log N_t of that head's own masses.
    sc = torch.full((B, H, T), float("nan"), device="cuda")
    kv.kvpop_future_attn_scores(q, k, lse, w.scale, 0, -1, agg="mean", eps=1e-8, normalize=True, scores=sc)
    torch.cuda.synchronize()
    sc = sc.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(sc))
    want = oracle.target_scores(got, H, 0, -1, "mean", 1e-8)
    assert np.abs(sc - want).max() <= 1e-5


def test_qwen3_8b_t32k_one_head_exhaustive():
    """One (b, query head) of the T=32768 workload, every key, blocked oracle."""
    b, qh = 2, 6
    q, k = workload.make_slice("qwen3_8b_t32k", b, qh // 4)
    q = q[qh % 4]
    w = workload.make("qwen3_8b_t32k")
    assert np.array_equal(w.q_bits[b, qh], q)
    out, lse = _run(w, 0, -1)
    lse_ref = oracle.row_lse_blocked(q, k, w.scale, block=2048)
    _check_lse(lse[b, qh], lse_ref, "32k exhaustive")
    ref = oracle.future_mass_blocked(q, k, w.scale, lse=lse_ref, block=2048)
    _check_out(out[b, qh], ref, 0, "32k exhaustive")


# ---------------------------------------------------------------------------
# closed forms at full length (T = 131072)
# ---------------------------------------------------------------------------

def _harmonic(n):
    # H_n in fp64 by direct summation in reverse (small to large)
    return np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, n + 1))])


@pytest.mark.timeout(900)
def test_long_t128k_as_generated():
    """The T=131072 workload exactly as generated (B=1, 32 query heads on 8 KV heads,
    drifting clusters) in the benchmark's launch sequence: pass 1 once, then pass 2
    for the bands (0, -1) and (1, 4096) from that one LSE. With B * Hkv = 8 every
    XCD runs one (b, KV head) group in an unsplit launch. Checked: the full-band
    masses of every head sum to T; sampled LSE rows of two query heads of every KV
    head; every LSE row and every key of both bands for query head 5 (KV head 1);
    every LSE row and every key of the W = 4096 band for query head 30 (KV head 7)."""
    w = workload.make("long_t128k")
    assert (w.B, w.Hq, w.Hkv, w.T, w.D) == (1, 32, 8, 131072, 128) and w.bands == [(0, -1), (1, 4096)]
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    lse_d = kv.kvpop_row_lse(q, k, w.scale)
    outs_d = [kv.kvpop_future_attn_from_lse(q, k, lse_d, w.scale, a, h) for a, h in w.bands]
    torch.cuda.synchronize()
    lse = lse_d.cpu().numpy().astype(np.float64)
    full, wband = [o.cpu().numpy().astype(np.float64) for o in outs_d]
    del q, k, lse_d, outs_d
    np.testing.assert_allclose(full.sum(axis=-1), w.T, rtol=REL)
    rng = np.random.default_rng(5)
    for h in range(w.Hkv):
        for qh in (h * w.G, h * w.G + 3):
            rows = sorted(set(rng.integers(0, w.T, 4).tolist()) | {0, 8191, 8192, w.T - 1})
            np.testing.assert_allclose(lse[0, qh, rows], oracle.row_lse_rows(w.q_bits[0, qh], w.k_bits[0, h], w.scale,
                                                                             rows), atol=LSE_ABS, rtol=0)
    # both bands from one sweep: the same masses up to the fp32 summation order
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    lse_d = torch.from_numpy(lse.astype(np.float32)).to("cuda")
    fused = kv.kvpop_future_attn_bands(q, k, lse_d, w.scale, w.bands)
    torch.cuda.synchronize()
    del q, k, lse_d
    for o, ref in zip(fused, (full, wband)):
        np.testing.assert_allclose(o.cpu().numpy(), ref, rtol=2e-5, atol=0)
    for qh, bands in [(5, [0, 1]), (30, [1])]:
        qv, kv_ = w.q_bits[0, qh], w.k_bits[0, qh // w.G]
        lse_ref = oracle.row_lse_blocked(qv, kv_, w.scale, block=512, threads=THREADS)
        _check_lse(lse[0, qh], lse_ref, "128k qh%d" % qh)
        for i in bands:
            a, h = w.bands[i]
            ref = oracle.future_mass_blocked(qv, kv_, w.scale, None, a, h, lse=lse_ref, block=512, threads=THREADS)
            _check_out((full, wband)[i][0, qh], ref, a, "128k qh%d band %s" % (qh, (a, h)))


def test_long_constant_keys_harmonic():
    """Every key equal (k_t = k) with the workload's random queries: each row is
    uniform whatever Q is, so LSE_d = scale <q_d, k> + log(d + 1) and the masses are
    the harmonic forms of Q = 0, at T = 131072 on real MFMA tiles."""
    T = 131072
    w = workload.make("long_t128k", Hq=4, Hkv=1)
    w.k_bits[:] = w.k_bits[:, :, 777:778, :]
    H = _harmonic(T + 1)
    t = np.arange(T)
    out, lse = _run(w, 0, -1)
    kk = oracle.bf16_bits_to_f64(w.k_bits[0, 0, 0])
    for qh in range(4):
        a = w.scale * (oracle.bf16_bits_to_f64(w.q_bits[0, qh]) @ kk)
        np.testing.assert_allclose(lse[0, qh], a + np.log(t + 1.0), atol=LSE_ABS, rtol=0)
    _check_out(out, np.broadcast_to(H[T] - H[t], out.shape), 0, "constant keys full")
    out, _ = _run(w, 1, 4096)
    ref = np.where(t + 1 <= T - 1, H[np.minimum(T, t + 4097)] - H[np.minimum(t + 1, T)], 0.0)
    _check_out(out, np.broadcast_to(ref, out.shape), 1, "constant keys W=4096")


def test_long_q_zero_harmonic():
    """Q = 0: every row uniform, out_t = H_T - H_t (window 0) and H_{min(T,t+W+1)} -
    H_{t+1} for the (1, W) band; LSE_d = log(d + 1)."""
    T = 131072
    w = workload.make("long_t128k", Hq=4, Hkv=1)
    w.q_bits[:] = 0
    H = _harmonic(T + 1)
    t = np.arange(T)
    out, lse = _run(w, 0, -1)
    np.testing.assert_allclose(lse[0, 0], np.log(t + 1.0), atol=LSE_ABS, rtol=0)
    _check_out(out, np.broadcast_to(H[T] - H[t], out.shape), 0, "harmonic full")
    out, _ = _run(w, 1, 4096)
    ref = np.where(t + 1 <= T - 1, H[np.minimum(T, t + 4097)] - H[np.minimum(t + 1, T)], 0.0)
    _check_out(out, np.broadcast_to(ref, out.shape), 1, "harmonic W=4096")


def test_long_constant_query_prefix_form():
    """All queries of a head equal: p_{d->t} = e^{a_t} / Z_d, so the full-future mass
    is e^{a_t} * sum_{d >= t} 1 / Z_d -- prefix sums in fp64, real MFMA tiles."""
    T = 131072
    w = workload.make("long_t128k", Hq=2, Hkv=1)
    w.q_bits[:] = w.q_bits[:, :, 1000:1001, :]
    out, lse = _run(w, 0, -1)
    for qh in range(2):
        qv = oracle.bf16_bits_to_f64(w.q_bits[0, qh, 0])
        kk = oracle.bf16_bits_to_f64(w.k_bits[0, 0])
        a = w.scale * (kk @ qv)
        mx = a.max()
        Z = np.cumsum(np.exp(a - mx))  # scaled by e^{-mx}
        suffix = np.cumsum((1.0 / Z)[::-1])[::-1]
        ref = np.exp(a - mx) * suffix
        np.testing.assert_allclose(lse[0, qh], np.log(Z) + mx, atol=LSE_ABS, rtol=0)
        _check_out(out[0, qh][None], ref[None], 0, "constant query head %d" % qh)


# ---------------------------------------------------------------------------
# structural properties of the GPU path
# ---------------------------------------------------------------------------

def test_deterministic_bitwise():
    w = workload.make("qwen3_4b_t4k")
    a, la = _run(w, 0, -1)
    b, lb = _run(w, 0, -1)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_locality_of_finite_horizon():
    """With band (1, W), out_t depends only on Q rows t+1..t+W and K rows 0..t+W;
    changing Q and K rows beyond t0 + W leaves keys t <= t0 bitwise unchanged."""
    T, W, t0 = 2000, 100, 900
    w = workload.make(_cfg(1, 4, 1, T, 128, seed=77, kind="rope"))
    a, _ = _run(w, 1, W)
    w2 = workload.make(_cfg(1, 4, 1, T, 128, seed=78, kind="rope"))
    w.q_bits[:, :, t0 + W + 1:] = w2.q_bits[:, :, t0 + W + 1:]
    w.k_bits[:, :, t0 + W + 1:] = w2.k_bits[:, :, t0 + W + 1:]
    b, _ = _run(w, 1, W)
    assert np.array_equal(a[..., :t0 + 1], b[..., :t0 + 1])
    assert not np.array_equal(a, b)


def test_external_lse_pass2_only():
    """kvpop_future_attn_from_lse uses the given normaliser: lse + 0.25 scales every
    output by exp(-0.25)."""
    w = workload.make(_cfg(1, 4, 2, 300, 128, seed=9, kind="rope"))
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    lse = kv.kvpop_row_lse(q, k, w.scale)
    o1 = kv.kvpop_future_attn_from_lse(q, k, lse, w.scale, 0, -1)
    o2 = kv.kvpop_future_attn_from_lse(q, k, lse + 0.25, w.scale, 0, -1)
    torch.cuda.synchronize()
    np.testing.assert_allclose(o2.cpu().numpy(), o1.cpu().numpy() * math.exp(-0.25), rtol=1e-5)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale)
    _check_out(o1.cpu().numpy().astype(np.float64), ref, 0, "from_lse")


def test_gqa_head_permutation():
    """Permuting the query heads inside a group permutes the outputs (bitwise)."""
    w = workload.make(_cfg(1, 8, 2, 500, 128, seed=12, kind="rope"))
    a, _ = _run(w, 0, -1)
    perm = [2, 0, 3, 1, 5, 4, 7, 6]
    w.q_bits = np.ascontiguousarray(w.q_bits[:, perm])
    b, _ = _run(w, 0, -1)
    assert np.array_equal(b, a[:, perm])
