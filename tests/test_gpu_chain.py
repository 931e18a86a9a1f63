"""The target chain of one training step with every stage on the GPU, each stage
checked against the oracle:

1. dense row LSE and pass 2 with the fused target epilogue (App. D.4, App. B.1-B.2);
2. the running top-k of the static priorities those scores define, with per-head
   decay (App. B.3, App. C.1-C.2);
3. the sparse attention forward under that mask (Sec. 3.2, App. C.3);
4. pass 2 again, from the sparse forward's normaliser (App. D.3).

Each GPU stage takes the previous GPU stage's output, so the test also covers the
hand-over between entry points. Integer decisions (ranks, cutoffs, lifetimes) are
taken on both sides from the same fp32 scores, as in the ranking tests; the
floating-point stages use the bars of their own tests (2e-3 relative per key mass,
2^-8 (A + |O|) per output element, 5e-4 absolute per LSE)."""
import math

import numpy as np
import pytest

import oracle
import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu
REL = 2e-3
LSE_ABS = 5e-4


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


@pytest.mark.parametrize("T,budget", [(1536, (4, 64, 96)), (2500, (2, 128, 300))])
def test_target_chain(T, budget):
    s, win, kk = budget
    cfg = dict(seed=321 + T, B=1, Hq=8, Hkv=2, T=T, D=128, scale=1 / math.sqrt(128), kind="rope", sink=True,
               bands=[(0, -1)])
    w = workload.make(cfg)
    v_bits = workload.make_values(w)
    q, k, v = _dev(w.q_bits), _dev(w.k_bits), _dev(v_bits)
    bias = torch.from_numpy(w.bias).to("cuda")

    # 1. dense LSE, per-head masses and per-KV-head target scores
    lse = kv.kvpop_row_lse(q, k, w.scale, key_bias=bias)
    scores, mass = kv.kvpop_future_attn_scores(q, k, lse, w.scale, 0, -1, agg="max", eps=1e-8, normalize=True,
                                               key_bias=bias, write_mass=True)
    torch.cuda.synchronize()
    ref_lse = oracle.row_lse(w.q_bits, w.k_bits, w.scale, w.bias)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() <= LSE_ABS
    ref_mass = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, 0, -1)
    rel = np.abs(mass.cpu().numpy() - ref_mass) / ref_mass
    assert rel.max() <= REL, rel.max()
    sc = scores.cpu().numpy()
    want = oracle.target_scores(ref_mass, w.Hkv, 0, -1, "max", 1e-8)
    assert np.abs(sc - want).max() <= REL + 1e-5

    # 2. running top-k on the GPU's scores, per-head decay
    lg = np.log(np.array([0.999, 0.9999])).astype(np.float32)
    tk = kv.kvpop_running_topk(scores, s, win, kk, log_gamma=torch.from_numpy(lg).to("cuda"), labels=True,
                               evict=True)
    torch.cuda.synchronize()
    masks = []
    for h in range(w.Hkv):
        rank = oracle.ranks_from_priority(oracle.static_priority_f32(sc[0, h], lg[h]))
        tau = oracle.running_cutoff_fenwick(rank, s, win, kk)
        y, tb = oracle.teacher_labels(rank, tau, s, win)
        np.testing.assert_array_equal(tk["rank"][0, h].cpu().numpy(), rank)
        np.testing.assert_array_equal(tk["cutoff"][0, h].cpu().numpy(), tau)
        np.testing.assert_array_equal(tk["label"][0, h].cpu().numpy(), y)
        np.testing.assert_array_equal(tk["boundary"][0, h].cpu().numpy(), tb)
        np.testing.assert_array_equal(tk["evict"][0, h].cpu().numpy(), oracle.eviction_times(rank, tau, s, win))
        masks.append(oracle.running_topk_mask(rank, tau, s, win))
    assert all(m.sum(axis=1).max() == s + win + kk for m in masks)  # the budget saturates

    # 3. sparse forward under the GPU's lifetimes; the oracle builds its mask from
    # the ranks and cutoffs
    o, lse_sp = kv.kvpop_sparse_attn_fwd(q, k, v, tk["evict"], w.scale, key_bias=bias)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy().astype(np.float64)
    lse_sp_np = lse_sp.cpu().numpy()
    ref_lse_sp = np.empty_like(ref_lse)
    for qh in range(w.Hq):
        h = qh // w.G
        O, L, A = oracle.sparse_attention(w.q_bits[0, qh], w.k_bits[0, h], v_bits[0, h], w.scale, masks[h], w.bias)
        bound = 2.0 ** -8 * (A + np.abs(O)) * 1.001 + 1e-6
        assert np.all(np.abs(o[0, qh] - O) <= bound), qh
        assert np.abs(lse_sp_np[0, qh] - L).max() <= LSE_ABS, qh
        ref_lse_sp[0, qh] = L
    assert np.all(ref_lse_sp <= ref_lse + 1e-12)  # a subset of the keys: the normaliser can only shrink

    # 4. pass 2 from the sparse normaliser, on the same fp32 values on both sides
    mass_sp = kv.kvpop_future_attn_from_lse(q, k, lse_sp, w.scale, 0, -1, key_bias=bias)
    torch.cuda.synchronize()
    ref = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, 0, -1, lse=lse_sp_np.astype(np.float64))
    rel = np.abs(mass_sp.cpu().numpy() - ref) / ref
    assert rel.max() <= REL, rel.max()
    # under the smaller normaliser no key's mass falls (evicted keys carry summands
    # above 1), checked on the oracle's own sparse normaliser
    own = oracle.future_mass(w.q_bits, w.k_bits, w.scale, w.bias, 0, -1, lse=ref_lse_sp)
    assert np.all(own >= ref_mass * (1 - 1e-12)) and own.max() > ref_mass.max()
