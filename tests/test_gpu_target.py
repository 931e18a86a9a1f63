"""Parity of the fused target epilogue (App. D.4 step 5) with the oracle.

scores[b, h, t] = log(agg_g m_bar + eps) - log N_t is compared in absolute terms:
a 2e-3 relative error on the masses is at most ~2e-3 on their logarithm, so the bar
is |gpu - oracle| <= 2e-3 (+ 1e-5 for the fp32 logarithm itself).
"""
import math

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu
ABS = 2e-3 + 1e-5


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _cfg(B, Hq, Hkv, T, D, seed, kind="rope", sink=False):
    return dict(seed=seed, B=B, Hq=Hq, Hkv=Hkv, T=T, D=D, scale=1.0 / math.sqrt(D), kind=kind, sink=sink,
                bands=[(0, -1)])


def _scores(w, window, horizon, agg, eps, normalize, bias=None, write_mass=False):
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    bias = w.bias if bias is None else bias
    b = torch.from_numpy(np.ascontiguousarray(bias, dtype=np.float32)).to("cuda") if bias is not None else None
    lse = kv.kvpop_row_lse(q, k, w.scale, key_bias=b)
    sc, out = kv.kvpop_future_attn_scores(q, k, lse, w.scale, window, horizon, agg=agg, eps=eps,
                                          normalize=normalize, key_bias=b, write_mass=write_mass)
    mass = kv.kvpop_future_attn_from_lse(q, k, lse, w.scale, window, horizon, key_bias=b)
    torch.cuda.synchronize()
    return (sc.cpu().numpy().astype(np.float64), None if out is None else out.cpu().numpy(),
            mass.cpu().numpy())


def _check(got, ref, what):
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(got), fin), what + ": infinite entries differ"
    assert np.all(got[~fin] == ref[~fin]), what
    err = np.abs(got[fin] - ref[fin])
    assert err.max() <= ABS, "%s: max abs err %.3e" % (what, err.max())


CASES = [
    # B, Hq, Hkv, T, D, window, horizon
    (1, 4, 1, 300, 128, 0, -1),
    (2, 8, 2, 257, 128, 1, 64),
    (1, 6, 2, 200, 64, 3, -1),
    (1, 5, 1, 130, 128, 0, 10),
    (1, 16, 2, 96, 128, 1, -1),
    (1, 1, 1, 70, 64, 0, 0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B%dHq%dHkv%dT%dD%d_w%d_h%d" % c)
@pytest.mark.parametrize("agg", ["max", "mean"])
def test_scores_match_oracle(case, agg):
    B, Hq, Hkv, T, D, win, hor = case
    w = workload.make(_cfg(B, Hq, Hkv, T, D, seed=T + Hq))
    m_ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, None, win, hor)
    for eps, normalize in [(1e-8, True), (1e-3, False), (0.0, True)]:
        got, out, mass = _scores(w, win, hor, agg, eps, normalize, write_mass=True)
        ref = oracle.target_scores(m_ref, Hkv, win, hor, agg=agg, eps=eps, normalize=normalize)
        _check(got, ref, "case %s agg %s eps %g norm %s" % (case, agg, eps, normalize))
        # the per-head masses written by the fused kernel are the plain pass-2 masses,
        # bit for bit (a launch this small spreads plain pass 2's query heads over
        # more workgroups; each still sums its keys' terms in the same order)
        np.testing.assert_array_equal(out, mass)


def test_scores_with_sink_and_masked_keys():
    T = 400
    w = workload.make(_cfg(1, 8, 2, T, 128, seed=41, sink=True))
    bias = w.bias.copy()
    bias[5::9] = -np.inf
    m_ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, bias, 1, 50)
    for agg in ("max", "mean"):
        got, _, _ = _scores(w, 1, 50, agg, 1e-8, True, bias=bias)
        _check(got, oracle.target_scores(m_ref, 2, 1, 50, agg=agg, eps=1e-8), "sink/masked " + agg)


def test_scores_full_size_sampled():
    """T=32768 benchmark workload: the last 48 keys of two KV heads (all 4 query
    heads each) against the oracle's columns."""
    w = workload.make("qwen3_8b_t32k")
    got, out, mass = _scores(w, 0, -1, "max", 1e-8, True, write_mass=True)
    # the fused and plain launches sum every key's terms in one order
    np.testing.assert_array_equal(out, mass)
    cols = list(range(w.T - 48, w.T))
    for b, h in [(0, 2), (3, 7)]:
        m = np.stack([oracle.future_mass_columns(w.q_bits[b, h * 4 + g], w.k_bits[b, h], w.scale, cols)
                      for g in range(4)])
        r = np.log(m.max(axis=0) + 1e-8) - np.log(np.maximum(1, w.T - np.array(cols)))
        assert np.max(np.abs(got[b, h, cols] - r)) <= ABS


def test_scores_one_batch_row_full_length():
    """B = 1, T = 32768: plain pass 2 spreads each key block's query heads over two
    workgroups, the fused launch keeps them in one. Both sum each key's terms in the
    same order (bit for bit), and keys of the last key blocks match the oracle's
    columns."""
    w = workload.make("qwen3_8b_t32k", B=1)
    _, out, mass = _scores(w, 0, -1, "mean", 1e-8, True, write_mass=True)
    np.testing.assert_array_equal(out, mass)
    cols = [32000, 32300, 32511, 32512] + list(range(w.T - 8, w.T))
    for qh in (5, 26):
        m = oracle.future_mass_columns(w.q_bits[0, qh], w.k_bits[0, qh // 4], w.scale, cols)
        rel = np.abs(mass[0, qh, cols] - m) / m
        assert rel.max() <= 2e-3, "qh %d: mass max rel err %.3e" % (qh, rel.max())
