"""Host-side logic of bench.py (no GPU): the pair count of a band, the classification
of profiled kernel names, the lookup of recorded HBM traffic by source hash, and the
refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("T", [1, 2, 7, 40])
def test_band_pairs_brute_force(T):
    for window in range(0, T + 2):
        for horizon in [-1] + list(range(window, T + 3)):
            want = sum(1 for d in range(T) for t in range(d + 1)
                       if d - t >= window and (horizon < 0 or d - t <= horizon))
            assert bench.band_pairs(T, window, horizon) == want, (T, window, horizon)


@pytest.mark.parametrize("T", [1, 5, 23])
def test_union_pairs_brute_force(T):
    bands_list = [[(0, -1)], [(0, -1), (1, 4)], [(2, 3), (5, 9)], [(1, 1), (0, 0)], [(3, -1), (0, 2)], [(1, 6), (4, 9)]]
    for bands in bands_list:
        want = sum(1 for d in range(T) for t in range(d + 1)
                   if any(d - t >= a and (h < 0 or d - t <= h) for a, h in bands))
        assert bench.union_pairs(T, bands) == want, (T, bands)


def test_band_pairs_full_future_is_causal_count():
    assert bench.band_pairs(32768, 0, -1) == 32768 * 32769 // 2


def test_kernel_key():
    ns = "void kvpop::(anonymous namespace)::"
    assert bench.kernel_key(ns + "sparse_attn_fwd_kernel<128, 2, false, false>(kvpop::SparseLaunch)") == \
        "sparse_attn_fwd_kernel"
    assert bench.kernel_key(ns + "sparse_attn_fwd_kernel<64, 1, true, true>(kvpop::SparseLaunch)") == \
        "sparse_attn_fwd_kernel_exact"
    assert bench.kernel_key(ns + "future_mass_kernel<128, 2, 4, false, true>(...)") == "future_mass_kernel"
    assert bench.kernel_key(ns + "row_lse_kernel<128, 4, false>(...)") == "row_lse_kernel"
    assert bench.kernel_key("kvpop::topk_prepare_kernel(...)") == "topk_prepare_kernel"
    assert bench.kernel_key("__amd_rocclr_copyBuffer") is None


def test_traffic_lookup_follows_the_source_hash(tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    good = bench.kernel_source_hash("future_mass_kernel")
    rec = {"workload": "w", "kernels": {
        "future_mass_kernel": {"hbm_bytes_per_launch": 123.0, "source_sha256": good},
        "row_lse_kernel": {"hbm_bytes_per_launch": 456.0, "source_sha256": "0" * 64}}}
    path.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.traffic_for("future_mass_kernel", "w") == 123.0
    assert bench.traffic_for("row_lse_kernel", "w") is None          # taken on another source
    assert bench.traffic_for("future_mass_kernel", "other") is None  # another workload
    assert bench.traffic_for("sparse_attn_fwd_kernel", "w") is None  # not recorded
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench.traffic_for("future_mass_kernel", "w") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "--gpus 1" in (r.stdout + r.stderr)
