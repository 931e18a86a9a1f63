"""Every entry point runs on the stream it is given (the ABI's `stream` argument):
the same calls on a second stream, passed explicitly or taken from the current
stream, give bit-identical results to the default stream's (the kernels are
deterministic)."""
import math

import numpy as np
import pytest

import workload

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def _all_calls(q, k, v, bias, scale, stream):
    lse = kv.kvpop_row_lse(q, k, scale, key_bias=bias, stream=stream)
    mass = kv.kvpop_future_attn_from_lse(q, k, lse, scale, 1, 300, key_bias=bias, stream=stream)
    mass2, lse2 = kv.kvpop_future_attn_target(q, k, scale, 0, -1, key_bias=bias, stream=stream)
    scores, _ = kv.kvpop_future_attn_scores(q, k, lse2, scale, 0, -1, agg="mean", key_bias=bias, stream=stream)
    tk = kv.kvpop_running_topk(scores, 4, 32, 64, labels=True, evict=True, stream=stream)
    o, lse_sp = kv.kvpop_sparse_attn_fwd(q, k, v, tk["evict"], scale, key_bias=bias, stream=stream)
    return dict(lse=lse, mass=mass, mass2=mass2, lse2=lse2, scores=scores, o=o, lse_sp=lse_sp, **tk)


@pytest.mark.parametrize("explicit", [True, False])
def test_side_stream_matches_default_stream(explicit):
    w = workload.make(dict(seed=55, B=1, Hq=8, Hkv=2, T=777, D=128, scale=1 / math.sqrt(128), kind="rope",
                           sink=True, bands=[(0, -1)]))
    q, k, v = _dev(w.q_bits), _dev(w.k_bits), _dev(workload.make_values(w))
    bias = torch.from_numpy(w.bias).to("cuda")
    torch.cuda.synchronize()
    ref = _all_calls(q, k, v, bias, w.scale, None)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()  # default priority
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        got = _all_calls(q, k, v, bias, w.scale, side if explicit else None)
    side.synchronize()
    torch.cuda.synchronize()
    assert set(got) == set(ref)
    for name in ref:
        assert torch.equal(got[name], ref[name]), name
