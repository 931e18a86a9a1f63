"""Parity of the running top-k sparse attention forward (Sec. 3.2, App. C.1, C.3)
with the fp64 oracle.

The GPU gets token lifetimes (evict) from its own running top-k; the oracle builds
the mask from ranks and cutoffs by eq. running_topk_mask_app, independently of the
lifetimes, and runs the masked softmax in fp64 on the same bf16 inputs.

Tolerance, from the arithmetic. The kernel rounds each probability p to bf16
(relative error at most 2^-8) before the product with v and normalises by the sum
of the unrounded fp32 probabilities; the output is then rounded to bf16 (at most
2^-8 relative). So per element
    |o_gpu - o| <= 2^-8 (sum_t p_t |v_t| + |o|)
up to fp32 terms of order 1e-6 relative, which the bound's 1e-3 slack covers. The
LSE comes from fp32 logits and sums: 5e-4 absolute, as for the dense pass."""
import math

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu
LSE_ABS = 5e-4


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _bf16_to_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _cfg(B, Hq, Hkv, T, D, seed, sink=False):
    return dict(seed=seed, B=B, Hq=Hq, Hkv=Hkv, T=T, D=D, scale=1.0 / math.sqrt(D), kind="rope", sink=sink,
                bands=[(0, -1)])


def _gpu_ranking(scores, s, w, k):
    out = kv.kvpop_running_topk(torch.from_numpy(scores).to("cuda"), s, w, k, labels=False, evict=True)
    return out["evict"], out["rank"].cpu().numpy(), out["cutoff"].cpu().numpy()


def _check_rows(o_gpu, lse_gpu, q_bits, k_bits, v_bits, scale, mask_rows, rows, bias, what):
    O, lse, A = oracle.sparse_attention(q_bits[rows], k_bits, v_bits, scale, mask_rows, bias)
    got_o = o_gpu[rows]
    bound = 2.0 ** -8 * (A + np.abs(O)) * 1.001 + 1e-6
    err = np.abs(got_o - O)
    bad = err > bound
    assert not bad.any(), "%s: %d elements out of bound, worst excess %.3e (err %.3e)" % (
        what, bad.sum(), (err - bound).max(), err.max())
    lerr = np.abs(lse_gpu[rows] - lse)
    assert lerr.max() <= LSE_ABS, "%s: lse err %.3e" % (what, lerr.max())


def _run_case(B, Hq, Hkv, T, D, s, w, k, seed, sink=False, rows=None):
    wl = workload.make(_cfg(B, Hq, Hkv, T, D, seed, sink))
    v_bits = workload.make_values(wl)
    scores = workload.make_scores(wl)
    evict, rank_g, cut_g = _gpu_ranking(scores, s, w, k)
    bias = torch.from_numpy(wl.bias).to("cuda") if wl.bias is not None else None
    o, lse = kv.kvpop_sparse_attn_fwd(_dev(wl.q_bits), _dev(wl.k_bits), _dev(v_bits), evict, wl.scale,
                                      key_bias=bias)
    torch.cuda.synchronize()
    o = _bf16_to_f64(o)
    lse = lse.cpu().numpy().astype(np.float64)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            rank = oracle.ranks_from_priority(oracle.static_priority_f32(scores[b, h], 0.0))
            tau = oracle.running_cutoff_fenwick(rank, s, w, k)
            np.testing.assert_array_equal(rank_g[b, h], rank)
            np.testing.assert_array_equal(cut_g[b, h], tau)
            rr = np.arange(T) if rows is None else np.asarray(rows)
            M = oracle.running_topk_mask_rows(rank, tau, s, w, rr)
            for g in range(G):
                qh = h * G + g
                _check_rows(o[b, qh], lse[b, qh], wl.q_bits[b, qh], wl.k_bits[b, h], v_bits[b, h], wl.scale, M,
                            rr, wl.bias, "b%d qh%d" % (b, qh))
    return o, lse


CASES = [
    # B, Hq, Hkv, T, D, sinks, window, k
    (1, 4, 1, 300, 128, 4, 16, 20),      # G=4: two heads per wave
    (2, 8, 2, 257, 128, 2, 8, 40),       # ragged tail, B=2
    (1, 2, 2, 333, 64, 1, 5, 30),        # G=1: one head, two query blocks per wave
    (1, 4, 2, 200, 64, 0, 0, 7),         # G=2, no sinks, no window
    (1, 16, 2, 150, 128, 3, 1, 12),      # G=8: quarter-height tiles
    (1, 4, 1, 1, 128, 1, 1, 1),          # a single token
    (1, 4, 1, 45, 128, 60, 4, 3),        # all tokens are sinks: dense causal
    (1, 4, 1, 700, 128, 4, 64, 1000),    # never saturated: every eligible key kept
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B%dHq%dHkv%dT%dD%d_s%dw%dk%d" % c)
def test_matches_oracle(case):
    _run_case(*case, seed=sum(case))


def test_runs_of_several_tiles_with_ragged_ends():
    """B=1, 32 query / 8 KV heads, T=20000: 313 query tiles of 64 per group (the last
    with 32 queries). Runs take at least T / 8192 tiles, so each workgroup takes a run
    of 3 consecutive tiles (the last run holds one) and rebuilds its key lists
    incrementally from tile to tile. Rows of the first run, around a later run
    boundary and of the last tile, every head of every group."""
    T = 20000
    rows = np.r_[0:3, 60:70, 127:130, 189:195, 156 * 64 - 3:156 * 64 + 3, 312 * 64 - 2:T]
    _run_case(1, 32, 8, T, 128, 4, 256, 512, seed=21, rows=rows)


def test_sink_bias():
    """The +3 logit sink of the synthetic workloads as a key bias."""
    _run_case(1, 8, 2, 400, 128, 4, 32, 50, seed=7, sink=True)


def _lifetime_case(T, D, evict_np, seed, Hq=4, Hkv=1, rows=None):
    wl = workload.make(_cfg(1, Hq, Hkv, T, D, seed))
    v_bits = workload.make_values(wl)
    ev = torch.from_numpy(np.ascontiguousarray(evict_np, dtype=np.int32)).to("cuda")
    o, lse = kv.kvpop_sparse_attn_fwd(_dev(wl.q_bits), _dev(wl.k_bits), _dev(v_bits), ev, wl.scale)
    torch.cuda.synchronize()
    o = _bf16_to_f64(o)
    lse = lse.cpu().numpy().astype(np.float64)
    G = Hq // Hkv
    rr = np.arange(T) if rows is None else np.asarray(rows)
    for h in range(Hkv):
        M = oracle.lifetime_mask(evict_np[0, h], rr)
        has = M.any(axis=1)
        for g in range(G):
            qh = h * G + g
            # queries that keep nothing: o = 0, lse = -inf
            assert np.all(o[0, qh][rr[~has]] == 0) and np.all(np.isneginf(lse[0, qh][rr[~has]]))
            if has.any():
                _check_rows(o[0, qh], lse[0, qh], wl.q_bits[0, qh], wl.k_bits[0, h], v_bits[0, h], wl.scale,
                            M[has], rr[has], None, "lifetimes qh%d" % qh)


def test_dense_causal_lifetimes():
    """evict = T for every key: plain causal attention."""
    T = 1000
    _lifetime_case(T, 128, np.full((1, 1, T), T), seed=3)


def test_long_dense_causal_uses_several_windows():
    """Dense causal at T = 9000 keeps more keys than one LDS list holds, so the kernel
    scans and processes several position windows; sampled rows against the oracle."""
    T = 9000
    rows = [0, 1, 31, 32, 4095, 4096, 5000, 8191, 8192, 8999]
    _lifetime_case(T, 128, np.full((1, 2, T), T), seed=4, Hq=4, Hkv=2, rows=rows)


def test_sliding_window_lifetimes():
    T, w = 600, 37
    _lifetime_case(T, 64, (np.arange(T) + w)[None, None, :], seed=5)


def test_arbitrary_lifetimes():
    """Random lifetimes, including keys that are never kept (evict <= t), keys kept
    to the end, values above T and negative values; some queries keep nothing."""
    T = 500
    rng = np.random.default_rng(6)
    t = np.arange(T)
    ev = t + rng.integers(-5, 60, size=T)
    ev[rng.random(T) < 0.1] = 10 ** 9
    ev[rng.random(T) < 0.05] = -7
    _lifetime_case(T, 128, ev[None, None, :], seed=6)


def test_deterministic():
    wl = workload.make(_cfg(1, 4, 1, 500, 128, 11))
    v = _dev(workload.make_values(wl))
    evict, _, _ = _gpu_ranking(workload.make_scores(wl), 4, 16, 64)
    q, k = _dev(wl.q_bits), _dev(wl.k_bits)
    o1, l1 = kv.kvpop_sparse_attn_fwd(q, k, v, evict, wl.scale)
    o2, l2 = kv.kvpop_sparse_attn_fwd(q, k, v, evict, wl.scale)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_paper_budget_at_benchmark_size():
    """The paper's budget (s=4, w=256, k=2016) on the Qwen3-8B-shaped T=32768 layout
    (B=4, 32 query / 8 KV heads, D=128): sampled query rows of three (b, KV head)
    groups against the oracle, every head of each group."""
    B, Hq, Hkv, T, D = 4, 32, 8, 32768, 128
    s, w, k = 4, 256, 2016
    wl = workload.make("qwen3_8b_t32k")
    assert (wl.B, wl.Hq, wl.Hkv, wl.T, wl.D) == (B, Hq, Hkv, T, D)
    v_bits = workload.make_values(wl)
    scores = workload.make_scores(wl)
    evict, _, cut_g = _gpu_ranking(scores, s, w, k)
    o, lse = kv.kvpop_sparse_attn_fwd(_dev(wl.q_bits), _dev(wl.k_bits), _dev(v_bits), evict, wl.scale)
    torch.cuda.synchronize()
    rng = np.random.default_rng(12)
    rows = np.array(sorted(set(rng.integers(0, T, 24).tolist()) | {0, 63, 64, s + w + k - 2, s + w + k - 1,
                                                                    T - 65, T - 64, T - 1}))
    G = Hq // Hkv
    for b, h in [(0, 0), (1, 5), (3, 7)]:
        rank = oracle.ranks_from_priority(oracle.static_priority_f32(scores[b, h], 0.0))
        tau = oracle.running_cutoff_fenwick(rank, s, w, k)
        np.testing.assert_array_equal(cut_g[b, h], tau)
        M = oracle.running_topk_mask_rows(rank, tau, s, w, rows)
        assert M.sum(axis=1).max() == s + w + k
        for g in range(G):
            qh = h * G + g
            o_rows = _bf16_to_f64(o[b, qh, torch.from_numpy(rows).to("cuda")])
            full = np.zeros((T, D))
            full[rows] = o_rows
            lse_full = np.zeros(T)
            lse_full[rows] = lse[b, qh, torch.from_numpy(rows).to("cuda")].cpu().numpy()
            _check_rows(full, lse_full, wl.q_bits[b, qh], wl.k_bits[b, h], v_bits[b, h], wl.scale, M, rows,
                        wl.bias, "b%d qh%d" % (b, qh))
    assert torch.isfinite(lse).all()


def test_large_logits_take_the_exact_path():
    """Keys after position 100 scaled by 16 (exact in bf16): their logits exceed the
    first block's maximum by far more than 2^64, so the fast variant flags its tiles
    and the exact variant (online rescaling) recomputes them. Dense causal lifetimes."""
    T, D = 300, 128
    wl = workload.make(_cfg(1, 4, 1, T, D, seed=13))
    k_bits = wl.k_bits.copy()
    kf = k_bits.view(np.uint16).astype(np.uint32) << 16
    kf = kf.view(np.float32)
    kf[:, :, 100:] *= 16.0
    k_bits = (kf.view(np.uint32) >> 16).astype(np.uint16)
    v_bits = workload.make_values(wl)
    ev = torch.full((1, 1, T), T, dtype=torch.int32, device="cuda")
    o, lse = kv.kvpop_sparse_attn_fwd(_dev(wl.q_bits), _dev(k_bits), _dev(v_bits), ev, wl.scale)
    torch.cuda.synchronize()
    o = _bf16_to_f64(o)
    lse = lse.cpu().numpy().astype(np.float64)
    rows = np.arange(T)
    M = oracle.lifetime_mask(np.full(T, T), rows)
    _, lse_ref, _ = oracle.sparse_attention(wl.q_bits[0, 0], k_bits[0, 0], v_bits[0, 0], wl.scale, M)
    assert (lse_ref[150:] - lse_ref[:32].max()).max() * 1.4427 > 64  # the case is what it claims to be
    for qh in range(4):
        _check_rows(o[0, qh], lse[0, qh], wl.q_bits[0, qh], k_bits[0, 0], v_bits[0, 0],
                    wl.scale, M, rows, None, "qh%d" % qh)


def test_long_context_t131072():
    """The long-context workload (B=1, 32/8 heads, D=128, T=131072, clustered keys) under
    the paper's budget: sampled query rows of two KV-head groups, every head."""
    s, w, k = 4, 256, 2016
    wl = workload.make("long_t128k")
    T, Hq, Hkv = wl.T, wl.Hq, wl.Hkv
    v_bits = workload.make_values(wl)
    scores = workload.make_scores(wl)
    evict, _, cut_g = _gpu_ranking(scores, s, w, k)
    o, lse = kv.kvpop_sparse_attn_fwd(_dev(wl.q_bits), _dev(wl.k_bits), _dev(v_bits), evict, wl.scale)
    torch.cuda.synchronize()
    rng = np.random.default_rng(22)
    rows = np.array(sorted(set(rng.integers(0, T, 16).tolist()) | {0, 4095, 4096, 65535, 65536, T - 1}))
    G = Hq // Hkv
    rows_dev = torch.from_numpy(rows).to("cuda")
    for h in (0, 6):
        rank = oracle.ranks_from_priority(oracle.static_priority_f32(scores[0, h], 0.0))
        tau = oracle.running_cutoff_fenwick(rank, s, w, k)
        np.testing.assert_array_equal(cut_g[0, h], tau)
        M = oracle.running_topk_mask_rows(rank, tau, s, w, rows)
        for g in range(G):
            qh = h * G + g
            full = np.zeros((T, wl.D))
            full[rows] = _bf16_to_f64(o[0, qh, rows_dev])
            lse_full = np.zeros(T)
            lse_full[rows] = lse[0, qh, rows_dev].cpu().numpy()
            _check_rows(full, lse_full, wl.q_bits[0, qh], wl.k_bits[0, h], v_bits[0, h], wl.scale, M, rows, wl.bias,
                        "qh%d" % qh)
    assert torch.isfinite(lse).all()
