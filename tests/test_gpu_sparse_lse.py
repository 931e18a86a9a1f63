"""Future mass from the student's sparse normaliser (App. D.3, eq. sparse_lse_app):
pass 2 through kvpop_future_attn_from_lse with LSE~ computed by the oracle over a
running top-k mask (App. C.1). Evicted keys then carry summands above 1; the bar
is the same relative 2e-3 per key against the oracle on the same fp32 normaliser."""
import math

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu
REL = 2e-3


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _sparse_lse(w, s, win, k, seed):
    """Per query head: LSE~ over the running top-k mask of random static priorities
    (one priority vector per KV head, as the scorer would produce)."""
    rng = np.random.default_rng(seed)
    lse = np.empty((w.B, w.Hq, w.T))
    kept = []
    for b in range(w.B):
        for h in range(w.Hkv):
            rank = oracle.ranks_from_priority(rng.standard_normal(w.T))
            tau = oracle.running_cutoff_fenwick(rank, s, win, k)
            M = oracle.running_topk_mask(rank, tau, s, win)
            kept.append(M.sum(axis=1).max())
            for g in range(w.G):
                qh = h * w.G + g
                lse[b, qh] = oracle.sparse_row_lse(w.q_bits[b, qh], w.k_bits[b, h], w.scale, M, w.bias)
    return lse.astype(np.float32), max(kept)


@pytest.mark.parametrize("T,band", [(1024, (0, -1)), (700, (1, 200)), (513, (3, -1))])
def test_sparse_normaliser_parity(T, band):
    cfg = dict(seed=90 + T, B=1, Hq=8, Hkv=2, T=T, D=128, scale=1 / math.sqrt(128), kind="rope", sink=True,
               bands=[band])
    w = workload.make(cfg)
    lse32, kept = _sparse_lse(w, s=4, win=64, k=96, seed=T)
    assert kept == 4 + 64 + 96
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    b = torch.from_numpy(w.bias).to("cuda")
    lse_d = torch.from_numpy(lse32).to("cuda")
    out = kv.kvpop_future_attn_from_lse(q, k, lse_d, w.scale, band[0], band[1], key_bias=b)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, band[0], band[1], lse=lse32.astype(np.float64))
    empty = np.arange(T) + band[0] > T - 1
    assert np.all(got[..., empty] == 0)
    r = ref[..., ~empty]
    rel = np.abs(got[..., ~empty] - r) / r
    assert rel.max() <= REL, rel.max()
    # the sparse normaliser is smaller than the dense one, so some summands exceed 1
    dense = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, band[0], band[1])
    assert np.all(ref >= dense * (1 - 1e-12))
    assert ref.max() > dense.max()
    # and the fused target epilogue works from it as well
    sc, _ = kv.kvpop_future_attn_scores(q, k, lse_d, w.scale, band[0], band[1], agg="max", eps=1e-8,
                                        key_bias=b)
    torch.cuda.synchronize()
    want = oracle.target_scores(ref, w.Hkv, band[0], band[1], "max", 1e-8)
    assert np.max(np.abs(sc.cpu().numpy() - want)) <= REL + 1e-5


def test_all_ones_mask_gives_dense_target():
    """k >= T keeps every key: LSE~ = LSE and the target equals the dense one."""
    T = 400
    cfg = dict(seed=77, B=1, Hq=4, Hkv=1, T=T, D=128, scale=1 / math.sqrt(128), kind="rope", sink=False,
               bands=[(0, -1)])
    w = workload.make(cfg)
    lse32, _ = _sparse_lse(w, s=2, win=16, k=T, seed=1)
    dense_lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale)
    np.testing.assert_allclose(lse32, dense_lse, rtol=1e-6, atol=1e-6)
    q, k = _dev(w.q_bits), _dev(w.k_bits)
    out = kv.kvpop_future_attn_from_lse(q, k, torch.from_numpy(lse32).to("cuda"), w.scale, 0, -1)
    dense_gpu, _ = kv.kvpop_future_attn_target(q, k, w.scale, 0, -1)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.cpu().numpy(), dense_gpu.cpu().numpy(), rtol=1e-4)
