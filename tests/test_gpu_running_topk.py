"""Running top-k ranking on the GPU against the oracle, bit-exact (App. B.3, App. C,
Sec. 3.1 eq. teacher_label). Priorities are compared in float32 on both sides (the
ranking is an integer decided by them); ranks, cutoffs, labels and boundary tokens
must match exactly."""
import math

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
import paper_2607_05061_amd as kv  # noqa: E402

pytestmark = pytest.mark.gpu


def _expected(scores, log_gamma, s, w, k, queries=None):
    B, H, T = scores.shape
    exp = {n: np.empty((B, H, T), dtype=np.int64) for n in ("rank", "cutoff", "label", "boundary", "evict")}
    for b in range(B):
        for h in range(H):
            lg = 0.0 if log_gamma is None else log_gamma[h]
            prio = oracle.static_priority_f32(scores[b, h], lg)
            rank = oracle.ranks_from_priority(prio)
            tau = oracle.running_cutoff_fenwick(rank, s, w, k)
            y, tb = oracle.teacher_labels(rank, tau, s, w, queries)
            exp["rank"][b, h], exp["cutoff"][b, h] = rank, tau
            exp["label"][b, h], exp["boundary"][b, h] = y, tb
            exp["evict"][b, h] = oracle.eviction_times(rank, tau, s, w)
    return exp


def _run(scores, log_gamma, s, w, k, labels=True, evict=True):
    sc = torch.from_numpy(scores).to("cuda")
    lg = torch.from_numpy(np.asarray(log_gamma, dtype=np.float32)).to("cuda") if log_gamma is not None else None
    out = kv.kvpop_running_topk(sc, s, w, k, log_gamma=lg, labels=labels, evict=evict)
    torch.cuda.synchronize()
    return {n: v.cpu().numpy().astype(np.int64) for n, v in out.items()}


def test_hand_case():
    scores = np.array([[[5.0, 2.0, 4.0, 1.0, 3.0]]], dtype=np.float32)  # ranks (0, 3, 1, 4, 2)
    got = _run(scores, None, 1, 1, 2)
    np.testing.assert_array_equal(got["rank"][0, 0], [0, 3, 1, 4, 2])
    np.testing.assert_array_equal(got["cutoff"][0, 0], [5, 5, 5, 3, 3])
    np.testing.assert_array_equal(got["label"][0, 0], [0, 0, 1, 1, -1])
    np.testing.assert_array_equal(got["boundary"][0, 0], [-1, -1, 1, 1, 1])
    np.testing.assert_array_equal(got["evict"][0, 0], [5, 5, 5, 4, 5])


CASES = [
    # B, H, T, s, w, k
    (1, 1, 1, 0, 0, 1),
    (1, 2, 2, 0, 1, 1),
    (2, 3, 17, 1, 2, 3),
    (1, 2, 300, 4, 16, 20),
    (2, 2, 1000, 4, 64, 128),
    (1, 1, 4097, 4, 256, 1000),
    (1, 2, 513, 0, 0, 1),
    (1, 1, 600, 10, 5, 700),   # never saturated
    (1, 1, 50, 60, 3, 2),      # sinks beyond T: nothing eligible
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B%dH%dT%d_s%dw%dk%d" % c)
@pytest.mark.parametrize("decay", [False, True])
def test_matches_oracle(case, decay):
    B, H, T, s, w, k = case
    rng = np.random.default_rng(T * 7 + k)
    scores = rng.standard_normal((B, H, T)).astype(np.float32) * 3
    log_gamma = np.log(rng.uniform(0.99, 0.9999, size=H)).astype(np.float32) if decay else None
    got = _run(scores, log_gamma, s, w, k)
    exp = _expected(scores, log_gamma, s, w, k)
    for n in ("rank", "cutoff", "label", "boundary", "evict"):
        np.testing.assert_array_equal(got[n], exp[n], err_msg=n)


def test_ties_break_to_earlier_position():
    rng = np.random.default_rng(3)
    scores = (np.round(rng.standard_normal((2, 2, 700)) * 2) / 2).astype(np.float32)  # many exact ties
    got = _run(scores, None, 2, 8, 40)
    exp = _expected(scores, None, 2, 8, 40)
    for n in ("rank", "cutoff", "label", "boundary", "evict"):
        np.testing.assert_array_equal(got[n], exp[n], err_msg=n)


def test_ties_across_sorted_chunks():
    """Exact ties spanning the 4096-position chunks that the ranking sorts one
    workgroup each (three whole chunks and a ragged one): every tie still breaks to the
    earlier position, an all-equal sequence ranks by position, and -0.0 ties +0.0."""
    rng = np.random.default_rng(8)
    T = 3 * 4096 + 123
    scores = (np.round(rng.standard_normal((1, 3, T)) * 2) / 2).astype(np.float32)
    scores[0, 1] = 1.5
    scores[0, 2, ::2] = -0.0
    scores[0, 2, 1::2] = 0.0
    scores[0, 2, 5000:5010] = 2.0
    got = _run(scores, None, 4, 256, 2016)
    exp = _expected(scores, None, 4, 256, 2016)
    for n in ("rank", "cutoff", "label", "boundary", "evict"):
        np.testing.assert_array_equal(got[n], exp[n], err_msg=n)
    np.testing.assert_array_equal(got["rank"][0, 1], np.arange(T))


def test_labels_optional():
    scores = np.random.default_rng(4).standard_normal((1, 2, 200)).astype(np.float32)
    got = _run(scores, None, 1, 4, 10, labels=False, evict=False)
    assert set(got) == {"rank", "cutoff"}
    exp = _expected(scores, None, 1, 4, 10)
    np.testing.assert_array_equal(got["cutoff"], exp["cutoff"])


def test_paper_budget_at_benchmark_size():
    """The paper's budget (s=4, w=256, k=2016) on the Qwen3-8B-shaped T=32768 layout
    (B=4, 8 KV heads) with learned-decay-range log gammas: ranks and cutoffs of every
    sequence exactly, labels and boundaries on sampled queries."""
    B, H, T, s, w, k = 4, 8, 32768, 4, 256, 2016
    rng = np.random.default_rng(5)
    scores = rng.standard_normal((B, H, T)).astype(np.float32)
    log_gamma = (math.log(0.999) + rng.random(H) * (math.log(0.999999) - math.log(0.999))).astype(np.float32)
    got = _run(scores, log_gamma, s, w, k)
    qs = sorted(set(rng.integers(0, T, 64).tolist()) | {0, s + w - 1, s + w, s + w + k - 2, s + w + k - 1, T - 1})
    for b, h in [(0, 0), (1, 5), (3, 7)]:
        e = _expected(scores[b:b + 1, h:h + 1], log_gamma[h:h + 1], s, w, k, queries=qs)
        np.testing.assert_array_equal(got["rank"][b, h], e["rank"][0, 0])
        np.testing.assert_array_equal(got["cutoff"][b, h], e["cutoff"][0, 0])
        np.testing.assert_array_equal(got["evict"][b, h], e["evict"][0, 0])
        np.testing.assert_array_equal(got["label"][b, h, qs], e["label"][0, 0, qs])
        np.testing.assert_array_equal(got["boundary"][b, h, qs], e["boundary"][0, 0, qs])
    # every sequence: ranks are a permutation, cutoffs monotone once saturated
    for b in range(B):
        for h in range(H):
            assert np.array_equal(np.sort(got["rank"][b, h]), np.arange(T))
            c = got["cutoff"][b, h]
            assert np.all(np.diff(c[s + w + k - 1:]) <= 0) and np.all(c[:s + w + k - 1] == T)


def test_long_context_t131072():
    """T = 131072 (the long-context workload's length), paper budget, decay on: ranks,
    cutoffs and eviction queries of two heads in full, labels and boundaries sampled."""
    H, T, s, w, k = 4, 131072, 4, 256, 2016
    rng = np.random.default_rng(21)
    scores = rng.standard_normal((1, H, T)).astype(np.float32)
    log_gamma = np.log(np.linspace(0.999, 0.999999, H)).astype(np.float32)
    got = _run(scores, log_gamma, s, w, k)
    qs = sorted(set(rng.integers(0, T, 48).tolist()) | {0, s + w + k - 1, T - 1})
    for h in (0, 3):
        e = _expected(scores[:, h:h + 1], log_gamma[h:h + 1], s, w, k, queries=qs)
        for n in ("rank", "cutoff", "evict"):
            np.testing.assert_array_equal(got[n][0, h], e[n][0, 0], err_msg=n)
        np.testing.assert_array_equal(got["label"][0, h, qs], e["label"][0, 0, qs])
        np.testing.assert_array_equal(got["boundary"][0, h, qs], e["boundary"][0, 0, qs])


@pytest.mark.parametrize("T", [32771, 32772, 40000, 136072])
def test_each_wavelet_build(T):
    """The wavelet levels are built in LDS up to n = T - s = 32767 eligible positions
    (T = 32771) and in rounds through global memory beyond (T = 32772, the first size
    past LDS; T = 40000 and 136072, ragged last rounds). Ranks, cutoffs and eviction
    queries of every position exactly, labels and boundaries on sampled queries."""
    s, w, k = 4, 256, 2016
    rng = np.random.default_rng(T)
    scores = rng.standard_normal((1, 2, T)).astype(np.float32)
    log_gamma = np.log(np.array([0.9999, 0.99999])).astype(np.float32)
    got = _run(scores, log_gamma, s, w, k)
    qs = sorted(set(rng.integers(0, T, 40).tolist()) | {0, s + w + k - 1, T - 1})
    for h in range(2):
        e = _expected(scores[:, h:h + 1], log_gamma[h:h + 1], s, w, k, queries=qs)
        for n in ("rank", "cutoff", "evict"):
            np.testing.assert_array_equal(got[n][0, h], e[n][0, 0], err_msg=n)
        np.testing.assert_array_equal(got["label"][0, h, qs], e["label"][0, 0, qs])
        np.testing.assert_array_equal(got["boundary"][0, h, qs], e["boundary"][0, 0, qs])


def test_queries_from_lds_ragged_length():
    """64 sequences of T = 12411 (a ragged last block of queries): the query kernel
    copies each sequence's wavelet levels into LDS once its grid covers the chip.
    Ranks, cutoffs and eviction queries of three sequences exactly, labels and
    boundaries on sampled queries."""
    B, H, T, s, w, k = 8, 8, 12411, 4, 256, 2016
    rng = np.random.default_rng(77)
    scores = rng.standard_normal((B, H, T)).astype(np.float32)
    log_gamma = np.log(np.linspace(0.999, 0.99999, H)).astype(np.float32)
    got = _run(scores, log_gamma, s, w, k)
    qs = sorted(set(rng.integers(0, T, 48).tolist()) | {0, s + w + k - 2, s + w + k - 1, T - 1})
    for b, h in [(0, 0), (3, 5), (7, 7)]:
        e = _expected(scores[b:b + 1, h:h + 1], log_gamma[h:h + 1], s, w, k, queries=qs)
        for n in ("rank", "cutoff", "evict"):
            np.testing.assert_array_equal(got[n][b, h], e[n][0, 0], err_msg=n)
        np.testing.assert_array_equal(got["label"][b, h, qs], e["label"][0, 0, qs])
        np.testing.assert_array_equal(got["boundary"][b, h, qs], e["boundary"][0, 0, qs])
