"""Pass 2's guard (Sec. 3.2 eq. sparse_lse_main; App. D.3 eq. sparse_lse_app): with a
caller-supplied normaliser below the dense one, or a large per-key bias, the
summands exp(l(d, t) - LSE_d) are no longer probabilities and can leave the range
that pass 2's fast linear fp32 sweep holds. The kernel must then take its exact
sweep and return the mass itself: within the relative 2e-3 bar of the fp64 oracle,
+inf exactly where the mass exceeds the fp32 range, 0 for keys biased -inf, and
never NaN.

The cases run three launch forms: kvpop_future_attn_from_lse on a small grid (the
query heads of each key block spread over several workgroups), the same on a grid
of 2048 workgroups or more (every head in one workgroup), and
kvpop_future_attn_scores with its per-head masses (the fused epilogue's launch)."""
import math

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu
REL = 2e-3
FLT_MAX = float(np.finfo(np.float32).max)
TINY = 1e-30  # masses below this are in or near fp32's subnormal range


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _f32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda")


def _check(got, ref, window, what):
    """got: fp32 GPU masses; ref: fp64 oracle masses (same shape [..., T])."""
    T = got.shape[-1]
    assert not np.isnan(got).any(), what + ": NaN in the output"
    empty = np.arange(T) + window > T - 1
    assert np.all(got[..., empty] == 0.0), what + ": empty bands must be exactly 0"
    g, r = got[..., ~empty], ref[..., ~empty]
    over = r > FLT_MAX * (1 + REL)
    near = (r >= FLT_MAX * (1 - REL)) & ~over
    assert np.all(np.isposinf(g[over])), what + ": masses beyond the fp32 range must be +inf"
    zero = r == 0.0
    assert np.all(g[zero] == 0.0), what + ": keys never attended must be exactly 0"
    tiny = (r > 0) & (r < TINY)
    assert np.all((g[tiny] >= 0) & (g[tiny] <= TINY)), what + ": sub-1e-30 masses"
    ok = ~over & ~near & ~zero & ~tiny
    assert np.all(np.isfinite(g[ok])), what + ": finite masses must stay finite"
    rel = np.abs(g[ok] - r[ok]) / r[ok]
    assert rel.size == 0 or rel.max() <= REL, "%s: max rel err %.3e" % (what, rel.max())
    return int(over.sum())


def _run_all(w, lse, bias, window, horizon):
    """Masses from the small-grid (head-split) launch and from the fused-epilogue launch."""
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    b = _f32(bias) if bias is not None else None
    lse_d = _f32(lse)
    split = kv.kvpop_future_attn_from_lse(q, k, lse_d, w.scale, window, horizon, key_bias=b)
    _, epi = kv.kvpop_future_attn_scores(q, k, lse_d, w.scale, window, horizon, agg="max", eps=1e-8, key_bias=b,
                                         write_mass=True)
    torch.cuda.synchronize()
    return split.cpu().numpy().astype(np.float64), epi.cpu().numpy().astype(np.float64)


def _cfg(B, Hq, Hkv, T, D, seed):
    return dict(seed=seed, B=B, Hq=Hq, Hkv=Hkv, T=T, D=D, scale=1.0 / math.sqrt(D), kind="rope", sink=True,
                bands=[(0, -1)])


@pytest.mark.parametrize("band", [(0, -1), (1, 200)])
def test_normaliser_80_below_on_some_rows(band):
    """LSE_d lowered by 80 on three rows: their summands are e^80 times a probability,
    so fast column sums pass 2^64 and the exact sweep must give the finite mass."""
    w = workload.make(_cfg(1, 4, 2, 700, 128, seed=501))
    lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale, w.bias)
    lse[:, :, [150, 151, 600]] -= 80.0
    lse32 = lse.astype(np.float32)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, *band, lse=lse32.astype(np.float64))
    assert ref.max() > 2.0 ** 64
    split, epi = _run_all(w, lse32, w.bias, *band)
    _check(split, ref, band[0], "split")
    _check(epi, ref, band[0], "epilogue launch")


def test_normaliser_100_below_gives_inf():
    """LSE_d lowered by 100 on one row: every key that row attends with probability
    above ~1.3e-5 has a mass beyond the fp32 range (+inf); keys after it are
    unaffected; keys biased -inf stay exactly 0."""
    T = 700
    w = workload.make(_cfg(1, 4, 1, T, 128, seed=502))
    bias = w.bias.copy()
    bias[5::37] = -np.inf
    lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale, bias)
    lse[:, :, 400] -= 100.0
    lse32 = lse.astype(np.float32)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, bias, 0, -1, lse=lse32.astype(np.float64))
    split, epi = _run_all(w, lse32, bias, 0, -1)
    assert _check(split, ref, 0, "split") > 100
    _check(epi, ref, 0, "epilogue launch")
    assert np.all(split[..., 5::37] == 0.0) and np.all(epi[..., 5::37] == 0.0)


def test_evicted_heavy_key():
    """A sparse normaliser whose mask drops one key lying ~100 logits above every
    key it keeps (App. D.3): that key's summands are ~e^100, its mass is +inf in
    fp32, and every other key's mass matches the oracle on the same normaliser."""
    T, D, jstar = 600, 128, 37
    rng = np.random.default_rng(503)
    q = rng.standard_normal((1, 2, T, D)).astype(np.float32) + 1.0
    k = rng.standard_normal((1, 1, T, D)).astype(np.float32)
    k[0, 0, jstar] = 10.0  # <q, k_j*> * scale ~ 10 * 128 / sqrt(128) ~ 113
    w = workload.Workload(name="heavy", B=1, Hq=2, Hkv=1, T=T, D=D, scale=float(np.float32(1 / math.sqrt(D))),
                          q_bits=workload.bf16_round_bits(q), k_bits=workload.bf16_round_bits(k), bias=None)
    mask = np.tril(np.ones((T, T), dtype=bool))
    mask[:, jstar] = False
    mask[jstar, jstar] = False
    mask[jstar, 0] = True  # row j* still keeps key 0 (a sink)
    lse = np.stack([oracle.sparse_row_lse(w.q_bits[0, g], w.k_bits[0, 0], w.scale, mask) for g in range(2)])[None]
    lse32 = lse.astype(np.float32)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, None, 0, -1, lse=lse32.astype(np.float64))
    logits = oracle.causal_logits(w.q_bits[0, 0], w.k_bits[0, 0], w.scale)
    assert np.min(logits[jstar:, jstar] - np.max(np.where(mask, logits, -np.inf)[jstar:], axis=1)) > 60
    assert np.all(ref[..., jstar] > FLT_MAX * 2)
    split, epi = _run_all(w, lse32, None, 0, -1)
    _check(split, ref, 0, "split")
    _check(epi, ref, 0, "epilogue launch")
    assert np.all(np.isposinf(split[..., jstar]))


@pytest.mark.parametrize("T", [3000, 16384])
def test_bias_minus_80_on_a_dominant_key(T):
    """A key biased -80 whose raw logit is ~102 above the rest dominates most rows;
    factoring exp(-80) out of its sum would overflow (e^80 per row). The dense
    normaliser from pass 1 and the masses must match the blocked oracle."""
    D, jstar = 128, 11
    rng = np.random.default_rng(504 + T)
    q = rng.standard_normal((1, 4, T, D)).astype(np.float32) + 1.0
    k = rng.standard_normal((1, 1, T, D)).astype(np.float32)
    k[0, 0, jstar] = 9.0  # raw logit ~ 9 * 128 / sqrt(128) ~ 102, ~22 after the bias
    bias = np.zeros(T, np.float32)
    bias[jstar] = -80.0
    w = workload.Workload(name="b80", B=1, Hq=4, Hkv=1, T=T, D=D, scale=float(np.float32(1 / math.sqrt(D))),
                          q_bits=workload.bf16_round_bits(q), k_bits=workload.bf16_round_bits(k), bias=bias)
    qd, kd, bd = _dev(w.q_bits), _dev(w.k_bits), _f32(bias)
    out, lse = kv.kvpop_future_attn_target(qd, kd, w.scale, 0, -1, key_bias=bd)
    _, epi = kv.kvpop_future_attn_scores(qd, kd, lse, w.scale, 0, -1, key_bias=bd, write_mass=True)
    torch.cuda.synchronize()
    out = out.cpu().numpy().astype(np.float64)
    epi = epi.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    for g in (0, 3):
        lse_ref = oracle.row_lse_blocked(w.q_bits[0, g], w.k_bits[0, 0], w.scale, bias, threads=8)
        assert np.abs(lse[0, g] - lse_ref).max() <= 5e-4
        ref = oracle.future_mass_blocked(w.q_bits[0, g], w.k_bits[0, 0], w.scale, bias, 0, -1, lse=lse_ref,
                                         threads=8)
        assert ref[jstar] > 0.5 * (T - jstar)  # the key takes most of every later row
        _check(out[0, g][None], ref[None], 0, "target head %d" % g)
        _check(epi[0, g][None], ref[None], 0, "epilogue head %d" % g)
    np.testing.assert_allclose(out.sum(axis=-1), T, rtol=REL)


def test_bias_plus_100():
    """A key biased +100 takes every later row; masses of the keys before it stay
    finite and accurate, the key's own mass is the number of rows it takes, and no
    launch produces NaN (exp(100) does not fit fp32)."""
    T = 900
    w = workload.make(_cfg(1, 4, 2, T, 128, seed=505))
    bias = np.zeros(T, np.float32)
    bias[450] = 100.0
    lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale, bias)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, bias, 0, -1, lse=lse)
    split, epi = _run_all(w, lse.astype(np.float32), bias, 0, -1)
    _check(split, ref, 0, "split")
    _check(epi, ref, 0, "epilogue launch")
    np.testing.assert_allclose(split[..., 450], T - 450, rtol=REL)


def test_unsplit_launch_with_lowered_normaliser():
    """A grid of 2048 workgroups (not split) with LSE_d lowered by 85 on a few rows of
    every head, and by 100 on one row of one head."""
    B, H, T, D = 8, 8, 8192, 64
    w = workload.make(dict(seed=506, B=B, Hq=H, Hkv=H, T=T, D=D, scale=1.0 / math.sqrt(D), kind="rope",
                           sink=False, bands=[(0, -1)]))
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    lse = kv.kvpop_row_lse(q, k, w.scale)
    lse[:, :, [1000, 5000, 8191]] -= 85.0
    lse[3, 5, 7000] -= 100.0
    out = kv.kvpop_future_attn_from_lse(q, k, lse, w.scale, 0, -1)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    lse_h = lse.cpu().numpy().astype(np.float64)
    for b, h in [(0, 0), (3, 5), (7, 7)]:
        ref = oracle.future_mass_blocked(w.q_bits[b, h], w.k_bits[b, h], w.scale, None, 0, -1, lse=lse_h[b, h],
                                         threads=8)
        _check(got[b, h][None], ref[None], 0, "unsplit b%d h%d" % (b, h))
    assert np.isposinf(got[3, 5]).sum() > 100
    assert np.isfinite(got[0, 0]).all()


def test_two_bands_with_lowered_normaliser():
    """Both bands of one sweep take the exact path when the normaliser is 80 below
    the dense one on a few rows, each within the bar of the oracle."""
    T = 900
    w = workload.make(_cfg(1, 4, 1, T, 128, seed=507))
    lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale, w.bias)
    lse[:, :, [300, 301, 880]] -= 80.0
    lse32 = lse.astype(np.float32)
    bands = [(0, -1), (1, 128)]
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    outs = kv.kvpop_future_attn_bands(q, k, _f32(lse32), w.scale, bands, key_bias=_f32(w.bias))
    torch.cuda.synchronize()
    for (a, h), o in zip(bands, outs):
        ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, a, h, lse=lse32.astype(np.float64))
        assert ref.max() > 2.0 ** 64
        _check(o.cpu().numpy().astype(np.float64), ref, a, "band %s" % ((a, h),))
