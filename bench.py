"""Benchmark of the future-attention target hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
pass 1 (row LSE) followed by pass 2 (future mass) for each band of the workload,
through the C ABI, on torch's current stream, with every input resident in HBM
before timing starts.

Prints ONE JSON line on stdout. The metric is key-query pairs per second,
B * Hq * T (T + 1) / 2 / seconds-per-step (every causal pair is scored at least
once), plus MFMA utilisation = algorithmic MFMA flops (2 * D per scored pair and
pass; masked tile work not counted) / time / dense bf16 peak.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config NAME] [--skip-cpu]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "key-query pairs/sec and MFMA util (% bf16 peak), Qwen3-8B-shaped layer at T=32k"
PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk/CU
CSRC = os.path.join(ROOT, "paper_2607_05061_amd", "csrc")
# The source file of each kernel whose HBM traffic is recorded (the fast and exact
# variants of the sparse forward are told apart by their last template argument).
KERNEL_SOURCES = {
    "row_lse_kernel": "kvpop_kernels.hip",
    "future_mass_kernel": "kvpop_kernels.hip",
    "sparse_attn_fwd_kernel": "kvpop_sparse_attn.hip",
    "sparse_attn_fwd_kernel_exact": "kvpop_sparse_attn.hip",
    "topk_chunk_sort_kernel": "kvpop_topk.hip",
    "topk_merge_rank_kernel": "kvpop_topk.hip",
    "topk_prepare_kernel": "kvpop_topk.hip",
    "topk_query_lds_kernel": "kvpop_topk.hip",
    "topk_query_kernel": "kvpop_topk.hip",
    "topk_evict_kernel": "kvpop_topk.hip",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
TOPK_BUDGET = (4, 256, 2016)  # sinks s, protected window w, top-k k: the paper's fixed budget B = s + w + k = 2276


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def band_pairs(T: int, window: int, horizon: int) -> int:
    """Number of (query d, key t) pairs with window <= d - t <= horizon, 0 <= t <= d < T."""
    hi = T - 1 if horizon < 0 else min(horizon, T - 1)
    if window > hi:
        return 0
    n = hi - window + 1
    return n * T - (window + hi) * n // 2


def union_pairs(T: int, bands) -> int:
    """Pairs (d, t) that lie in at least one of one or two bands."""
    pairs = sum(band_pairs(T, a, b) for a, b in bands)
    if len(bands) == 2:
        (a0, h0), (a1, h1) = bands
        lo = max(a0, a1)
        hi = min(h0 if h0 >= 0 else T - 1, h1 if h1 >= 0 else T - 1)
        if lo <= hi:
            pairs -= band_pairs(T, lo, hi)
    return pairs


def kernel_source_hash(kernel: str) -> str:
    with open(os.path.join(CSRC, KERNEL_SOURCES[kernel]), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def kernel_key(name: str):
    """The KERNEL_SOURCES key of a profiled kernel name, or None."""
    if "sparse_attn_fwd_kernel" in name:
        args = name.split("sparse_attn_fwd_kernel", 1)[1]
        args = args[:args.index(">")] if ">" in args else args
        return "sparse_attn_fwd_kernel_exact" if args.rstrip().endswith("true") else "sparse_attn_fwd_kernel"
    for k in KERNEL_SOURCES:
        if k in name:
            return k
    return None


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or None when
    absent or taken on a different source of that kernel."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    k = t.get("kernels", {}).get(kernel)
    if t.get("workload") != workload or not k or k.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return k.get("hbm_bytes_per_launch")


def host_cores():
    """os.cpu_count(), the CPUs this process may run on (what `nproc` prints), and
    the BLAS library's thread count."""
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    return os.cpu_count() or 1, len(os.sched_getaffinity(0)), int(blas)


def cpu_baseline(w, band, min_seconds: float = 10.0):
    """The fp64 oracle, as it stands, on (batch row, KV head) groups of the same
    workload, taken in order until at least ``min_seconds`` have passed: per group
    its G query heads, row LSE then future mass, in the oracle's blocked form with
    its row blocks on every CPU this process may use."""
    import numpy as np
    import oracle
    n_cpu, n_proc, blas = host_cores()
    threads = n_proc
    T = w.T
    groups = 0
    t0 = time.perf_counter()
    for b in range(w.B):
        for h in range(w.Hkv):
            k = w.k_bits[b, h]
            for g in range(w.G):
                q = w.q_bits[b, h * w.G + g]
                lse = oracle.row_lse_blocked(q, k, w.scale, w.bias, block=512, threads=threads)
                out = oracle.future_mass_blocked(q, k, w.scale, w.bias, band[0], band[1], lse=lse, block=512,
                                                 threads=threads)
                assert np.isfinite(out).all()
            groups += 1
            if time.perf_counter() - t0 >= min_seconds:
                break
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = time.perf_counter() - t0
    pairs = groups * w.G * T * (T + 1) // 2
    return {
        "value": pairs / dt,
        "unit": "pairs/s",
        "cores": int(threads),
        "kind": "oracle",
        "os_cpu_count": int(n_cpu),
        "nproc": int(n_proc),
        "blas_threads": int(blas),
        "sample": "the first %d (b, kv head) group(s) of %s: %d query heads each, %d pairs in all (every causal "
                  "pair once), row LSE then future mass with band %s; fp64 numpy oracle, blocked 512-row form, "
                  "row blocks on %d host threads (BLAS held to one thread per block); %.1f s"
                  % (groups, w.name, w.G, pairs, tuple(band), threads, dt),
    }


COPY_BYTES = 1 << 30  # calibration copy: 1 GiB read + 1 GiB written


def copy_calibrate():
    """A plain device-to-device copy of COPY_BYTES, three times, so that rocprofv3's
    FETCH_SIZE / WRITE_SIZE counters can be scaled against a known byte count."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("copied %d bytes x3" % COPY_BYTES)


def traffic_summary(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, workload, out_path=TRAFFIC_FILE):
    """Fold four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE for this benchmark
    and for the calibration copy) into HBM bytes per launch per kernel."""
    import csv
    import glob

    def per_kernel(d, counter):
        vals = {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                name = r["Kernel_Name"]
                key = kernel_key(name)
                if key is None:
                    key = next((c for c in ("copy", "elementwise") if c in name), None)
                if key is not None:
                    vals.setdefault(key, []).append(float(r["Counter_Value"]))
        return vals

    def copy_factor(d, counter):
        v = per_kernel(d, counter)
        cands = v.get("copy") or v.get("elementwise") or []
        kib = max(cands)  # the 1 GiB copy dominates any other copy-like launch
        return (COPY_BYTES / 1024.0) / kib, kib

    ff, fk = copy_factor(copy_fetch_dir, "FETCH_SIZE")
    wf, wk = copy_factor(copy_write_dir, "WRITE_SIZE")
    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")
    kernels = {}
    for k in KERNEL_SOURCES:
        if k in fetch and k in write:
            fb = sum(fetch[k]) / len(fetch[k]) * 1024.0 * ff
            wb = sum(write[k]) / len(write[k]) * 1024.0 * wf
            kernels[k] = {"fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                          "hbm_bytes_per_launch": fb + wb, "launches": len(fetch[k]),
                          "source": KERNEL_SOURCES[k], "source_sha256": kernel_source_hash(k)}
    res = {"workload": workload,
           "copy_calibration": {"bytes": COPY_BYTES, "fetch_kib_read": fk, "write_kib_read": wk,
                                "fetch_factor": ff, "write_factor": wf},
           "kernels": kernels}
    with open(out_path, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="qwen3_8b_t32k")
    ap.add_argument("--skip-cpu", action="store_true", help="omit the CPU oracle baseline")
    ap.add_argument("--copy-calibrate", action="store_true",
                    help="only run the 1 GiB calibration copy (for rocprofv3 FETCH_SIZE/WRITE_SIZE scaling)")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="fold rocprofv3 counter CSVs into profiles/hbm_traffic.json and exit")
    args = ap.parse_args()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary, workload=args.config)
        return
    if args.copy_calibrate:
        copy_calibrate()
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the future-attention target runs on a single MI355X "
              "(every (batch, KV head) group is independent; see the sharding design). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_05061_amd as kv
    import workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    w = workload.make(args.config)
    log("generated %s in %.1f s" % (args.config, time.perf_counter() - t_gen))
    q = torch.from_numpy(w.q_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    k = torch.from_numpy(w.k_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    bias = torch.from_numpy(w.bias).to(dev) if w.bias is not None else None
    shape = (w.B, w.Hq, w.T)
    lse = torch.empty(shape, dtype=torch.float32, device=dev)
    outs = [torch.empty(shape, dtype=torch.float32, device=dev) for _ in w.bands]

    def step(evs=None):
        if evs:
            evs[0].record()
        kv.kvpop_row_lse(q, k, w.scale, key_bias=bias, lse=lse)
        if evs:
            evs[1].record()
        # every band of the workload from one pass-2 sweep
        kv.kvpop_future_attn_bands(q, k, lse, w.scale, w.bands, key_bias=bias, outs=outs)
        if evs:
            evs[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    total_ms = evs[0][0].elapsed_time(evs[-1][-1])
    ms_step = total_ms / args.steps
    p1_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    p2_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))

    pairs_causal = w.B * w.Hq * w.T * (w.T + 1) // 2
    # Pairs pass 2 evaluates: the union of the bands (a pair in two bands is computed once).
    pairs_p2 = w.B * w.Hq * union_pairs(w.T, w.bands)
    flops_p1 = 2.0 * w.D * pairs_causal
    flops_p2 = 2.0 * w.D * pairs_p2
    value = pairs_causal / (ms_step * 1e-3)
    util = (flops_p1 + flops_p2) / (ms_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)

    # Dominant kernel: the longest average launch.
    cands = [("row_lse_kernel", p1_ms, flops_p1), ("future_mass_kernel", p2_ms, flops_p2)]
    name, dur, fl = max(cands, key=lambda c: c[1])
    achieved = fl / (dur * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_for(name, w.name),
                "kernel": name, "avg_launch_ms": round(dur, 4)}

    # The same step with the target epilogue fused into pass 2 (App. D.4 step 5):
    # per-KV-head scores log(max_g m_bar + eps) - log N_t instead of per-head masses.
    scores = torch.empty((w.B, w.Hkv, w.T), dtype=torch.float32, device=dev)

    def step_scores(evs):
        evs[0].record()
        kv.kvpop_row_lse(q, k, w.scale, key_bias=bias, lse=lse)
        evs[1].record()
        win, hor = w.bands[0]
        kv.kvpop_future_attn_scores(q, k, lse, w.scale, win, hor, agg="max", eps=1e-8, normalize=True,
                                    key_bias=bias, scores=scores)
        evs[2].record()

    n_epi = max(1, args.steps // 2)
    evs2 = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_epi)]
    for s in range(n_epi):
        step_scores(evs2[s])
    torch.cuda.synchronize()
    epi = {"band": list(w.bands[0]), "agg": "max", "steps": n_epi,
           "ms_per_step": round(evs2[0][0].elapsed_time(evs2[-1][-1]) / n_epi, 4),
           "pass2_with_epilogue_ms": round(float(np.mean([e[1].elapsed_time(e[2]) for e in evs2])), 4)}

    # Running top-k on the live target (App. B.3, App. C): ranks, cutoffs, teacher labels
    # and boundary tokens per (batch, KV head), with the paper's fixed budget and a
    # per-head decay in the learned range.
    s_, w_, k_ = TOPK_BUDGET
    lg = torch.tensor(np.log(np.linspace(0.999, 0.999999, w.Hkv)), dtype=torch.float32, device=dev)
    ws = torch.empty(kv.kvpop_running_topk_workspace_size(w.B, w.Hkv, w.T), dtype=torch.uint8, device=dev)
    for _ in range(2):
        kv.kvpop_running_topk(scores, s_, w_, k_, log_gamma=lg, workspace=ws)
    n_tk = max(1, args.steps // 2)
    ev_tk = [torch.cuda.Event(enable_timing=True) for _ in range(n_tk + 1)]
    ev_tk[0].record()
    for i in range(n_tk):
        tk = kv.kvpop_running_topk(scores, s_, w_, k_, log_gamma=lg, workspace=ws)
        ev_tk[i + 1].record()
    torch.cuda.synchronize()
    tk_ms = ev_tk[0].elapsed_time(ev_tk[-1]) / n_tk
    assert bool((torch.sort(tk["rank"], dim=-1).values == torch.arange(w.T, device=dev, dtype=torch.int32)).all()), \
        "ranks are not a permutation"
    topk = {"budget": {"sinks": s_, "window": w_, "k": k_}, "steps": n_tk, "ms": round(tk_ms, 4),
            "tokens_per_s": w.B * w.Hkv * w.T / (tk_ms * 1e-3)}

    # Running top-k sparse attention forward (Sec. 3.2, App. C) under that budget's
    # mask, then pass 2 from its sparse LSE (App. D.3): the paper's training-time
    # target, which needs no dense pass 1.
    tk = kv.kvpop_running_topk(scores, s_, w_, k_, log_gamma=lg, labels=False, evict=True, workspace=ws)
    evict = tk["evict"]
    v = torch.from_numpy(workload.make_values(w).view(np.int16)).view(torch.bfloat16).to(dev)
    o_sp = torch.empty_like(q)
    lse_sp = torch.empty(shape, dtype=torch.float32, device=dev)
    mass_sp = torch.empty(shape, dtype=torch.float32, device=dev)
    tt = torch.arange(w.T, device=dev, dtype=torch.int64)
    kept_pairs = int((evict.to(torch.int64).clamp(max=w.T) - tt).clamp(min=0).sum()) * w.G
    for _ in range(2):
        kv.kvpop_sparse_attn_fwd(q, k, v, evict, w.scale, key_bias=bias, o=o_sp, lse=lse_sp)
    n_sp = max(1, args.steps // 2)
    ev_sp = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_sp)]
    win0, hor0 = w.bands[0]
    for i in range(n_sp):
        ev_sp[i][0].record()
        kv.kvpop_sparse_attn_fwd(q, k, v, evict, w.scale, key_bias=bias, o=o_sp, lse=lse_sp)
        ev_sp[i][1].record()
        kv.kvpop_future_attn_from_lse(q, k, lse_sp, w.scale, win0, hor0, key_bias=bias, out=mass_sp)
        ev_sp[i][2].record()
    torch.cuda.synchronize()
    sp_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev_sp]))
    p2s_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev_sp]))
    assert bool(torch.isfinite(lse_sp).all()), "sparse LSE not finite"
    sp_flops = 4.0 * w.D * kept_pairs
    sp_tf = sp_flops / (sp_ms * 1e-3) / 1e12
    sparse = {"budget": {"sinks": s_, "window": w_, "k": k_}, "steps": n_sp, "ms": round(sp_ms, 4),
              "kept_pairs": kept_pairs, "pairs_per_s": kept_pairs / (sp_ms * 1e-3),
              "roofline": {"bound": "mfma", "achieved": round(sp_tf, 2), "peak": PEAK_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": round(sp_tf / PEAK_BF16_TFLOPS, 4),
                           "traffic": traffic_for("sparse_attn_fwd_kernel", w.name),
                           "kernel": "sparse_attn_fwd_kernel", "avg_launch_ms": round(sp_ms, 4)},
              "pass2_from_sparse_lse_ms": round(p2s_ms, 4)}
    del v, o_sp, mass_sp

    # Parity sanity on the live result: full-future masses of a head sum to T.
    for i, (a, b) in enumerate(w.bands):
        if a == 0 and b < 0:
            rs = outs[i].double().sum(dim=-1)
            err = float((rs / w.T - 1).abs().max())
            log("row-sum check band %s: max |sum/T - 1| = %.2e" % ((a, b), err))
            assert err < 2e-3, "row-sum invariant violated"

    cpu = None
    if not args.skip_cpu:
        log("timing the CPU oracle on one KV-head group ...")
        cpu = cpu_baseline(w, w.bands[0])

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "T": w.T, "D": w.D,
                   "bands": [list(b) for b in w.bands], "key_bias": w.bias is not None},
        "mfma_util": round(util, 4),
        "pass_ms": {"row_lse": round(p1_ms, 4), "future_mass": round(p2_ms, 4)},
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "target_epilogue": epi,
        "running_topk": topk,
        "sparse_attention": sparse,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
