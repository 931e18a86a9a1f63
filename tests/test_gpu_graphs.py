"""The entry points allocate nothing and launch only kernels on the stream they are
given (small pass-2 launches clear their output with a fill kernel, not a memset), so
the whole target chain can be captured in a HIP graph. A captured chain (pass 1,
pass 2, the fused target epilogue, the running top-k and the sparse forward) is
replayed several times, with other work on the stream and host synchronisations
between the replays, and every replay must reproduce the eager results bit for bit."""
import math

import numpy as np
import pytest

import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def test_captured_chain_replays_match_eager():
    w = workload.make(dict(seed=808, B=1, Hq=8, Hkv=2, T=777, D=128, scale=1 / math.sqrt(128), kind="rope",
                           sink=True, bands=[(0, -1)]))
    q, k, v = _dev(w.q_bits), _dev(w.k_bits), _dev(workload.make_values(w))
    bias = torch.from_numpy(w.bias).to("cuda")
    B, Hq, Hkv, T, D = w.B, w.Hq, w.Hkv, w.T, w.D
    lse = torch.empty(B, Hq, T, device="cuda")
    mass = torch.empty(B, Hq, T, device="cuda")
    scores = torch.empty(B, Hkv, T, device="cuda")
    o = torch.empty(B, Hq, T, D, dtype=torch.bfloat16, device="cuda")
    lse_sp = torch.empty(B, Hq, T, device="cuda")
    mass_sp = torch.empty(B, Hq, T, device="cuda")
    ws = torch.empty(kv.kvpop_running_topk_workspace_size(B, Hkv, T), dtype=torch.uint8, device="cuda")

    def chain():
        kv.kvpop_future_attn_target(q, k, w.scale, 0, -1, key_bias=bias, lse_ws=lse, out=mass)
        kv.kvpop_future_attn_scores(q, k, lse, w.scale, 0, -1, agg="max", key_bias=bias, scores=scores)
        tk = kv.kvpop_running_topk(scores, 4, 32, 64, labels=True, evict=True, workspace=ws)
        kv.kvpop_sparse_attn_fwd(q, k, v, tk["evict"], w.scale, key_bias=bias, o=o, lse=lse_sp)
        kv.kvpop_future_attn_from_lse(q, k, lse_sp, w.scale, 0, -1, key_bias=bias, out=mass_sp)
        return tk

    tk = chain()
    torch.cuda.synchronize()
    ref = dict(lse=lse.clone(), mass=mass.clone(), scores=scores.clone(), o=o.clone(), lse_sp=lse_sp.clone(),
               mass_sp=mass_sp.clone(), **{n: t.clone() for n, t in tk.items()})

    side = torch.cuda.Stream()  # default priority
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        chain()  # warm up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tk_g = chain()
    torch.cuda.synchronize()

    for rep in range(3):
        for t in (lse, mass, scores, lse_sp, mass_sp):
            t.fill_(float("nan"))  # eager work between the replays
        o.zero_()
        for t in tk_g.values():
            t.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = dict(lse=lse, mass=mass, scores=scores, o=o, lse_sp=lse_sp, mass_sp=mass_sp, **tk_g)
        assert set(got) == set(ref)
        for name in ref:
            assert torch.equal(got[name], ref[name]), (rep, name)
