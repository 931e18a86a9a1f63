"""Seeded generator of synthetic Q/K workloads shaped like the paper's models.

The paper trains on Qwen3-4B/8B activations at sequence length 16384 (Sec. 4,
experimental setup; App. F). Neither the data nor the weights are available, so the
workloads here are synthetic stand-ins with the same head counts and head size:

* rows are RMS-normalised (unit weight, eps 1e-6), so each row has norm ~ sqrt(D);
* rotary position embedding in the rotate-half convention, base 1e6, with the
  angles p * theta_i evaluated in float64 (p * theta reaches ~1.3e5 rad);
* cast to bfloat16 with round-to-nearest-even; the bit patterns are what both the
  GPU path and the oracle consume.

Each (batch row b, KV head h) slice is drawn from its own stream
``numpy.random.default_rng([seed, b, h])``, so a single slice can be regenerated
without generating the whole workload (the oracle's sampled checks rely on this).

Layouts: Q is ``[B, Hq, T, D]`` and K is ``[B, Hkv, T, D]``, both uint16 bf16 bits,
contiguous; query head ``qh`` reads KV head ``qh // G`` (contiguous groups).
"""
from __future__ import annotations

import concurrent.futures as _cf
import math
import os
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = ["CONFIGS", "Workload", "make", "make_slice", "bf16_round_bits", "rmsnorm", "rope"]


# Workload descriptions. window/horizon follow the library's convention: key j
# collects mass from queries i with j + window <= i <= j + horizon (horizon < 0:
# up to the last position).
CONFIGS = {
    "tiny": dict(seed=0, B=1, Hq=1, Hkv=1, T=512, D=64, scale=1.0 / 8.0, kind="normal",
                 sink=False, bands=[(0, -1)]),
    "qwen3_4b_t4k": dict(seed=1, B=1, Hq=32, Hkv=8, T=4096, D=128, scale=1.0 / math.sqrt(128.0),
                         kind="rope", sink=True, bands=[(0, -1)]),
    "qwen3_4b_t16k_w1024": dict(seed=2, B=2, Hq=32, Hkv=8, T=16384, D=128, scale=1.0 / math.sqrt(128.0),
                                kind="rope", sink=True, bands=[(1, 1024)]),
    "qwen3_8b_t32k": dict(seed=3, B=4, Hq=32, Hkv=8, T=32768, D=128, scale=1.0 / math.sqrt(128.0),
                          kind="heavy", sink=False, bands=[(0, -1)]),
    "long_t128k": dict(seed=4, B=1, Hq=32, Hkv=8, T=131072, D=128, scale=1.0 / math.sqrt(128.0),
                       kind="clusters", sink=False, bands=[(0, -1), (1, 4096)]),
}


def bf16_round_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); return uint16 bits.

    NaN is not expected in generated data; infinities pass through unchanged.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # RNE: add 0x7FFF plus the lowest kept bit, then truncate.
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def rmsnorm(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """Unit-weight RMS normalisation along the last axis (float32 in, float32 out)."""
    ms = np.mean(np.square(x, dtype=np.float32), axis=-1, keepdims=True, dtype=np.float32)
    return (x / np.sqrt(ms + np.float32(eps))).astype(np.float32)


def _rope_tables(T: int, D: int, base: float):
    half = D // 2
    theta = base ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    ang = np.arange(T, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def rope(x: np.ndarray, base: float = 1e6, tables=None) -> np.ndarray:
    """Rotate-half rotary embedding over positions 0..T-1 of ``x[..., T, D]``."""
    T, D = x.shape[-2], x.shape[-1]
    half = D // 2
    cos, sin = tables if tables is not None else _rope_tables(T, D, base)
    x1 = x[..., :half]
    x2 = x[..., half:]
    out = np.empty_like(x, dtype=np.float32)
    out[..., :half] = x1 * cos - x2 * sin
    out[..., half:] = x2 * cos + x1 * sin
    return out


@dataclass
class Workload:
    """One synthetic problem instance (host arrays).

    q_bits: uint16 [B, Hq, T, D]; k_bits: uint16 [B, Hkv, T, D];
    bias: float32 [T] or None (added to every logit of key column t);
    scale: softmax scale, a float32 value; bands: list of (window, horizon).
    """
    name: str
    B: int
    Hq: int
    Hkv: int
    T: int
    D: int
    scale: float
    q_bits: np.ndarray
    k_bits: np.ndarray
    bias: Optional[np.ndarray]
    bands: list = field(default_factory=list)
    seed: int = 0

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


def cluster_labels(rng, T: int, D: int, G: int, n_c: int = 16, seg: int = 8192):
    """Drifting-topic structure: n_c Gaussian centres; segment s = t // seg has its
    own mixture pi_s ~ Dirichlet(0.5); key t and each query head's position t pick
    a centre from pi_s. Returns (mu [n_c, D], pis [n_seg, n_c], c_k [T], c_q [G, T])."""
    mu = rng.standard_normal((n_c, D), dtype=np.float32)
    n_seg = -(-T // seg)
    pis = rng.dirichlet(np.full(n_c, 0.5), size=n_seg)
    seg_of_t = np.arange(T) // seg
    cdf = np.cumsum(pis, axis=1)[seg_of_t]

    def draw():
        u = rng.random(T)
        return np.minimum((u[:, None] > cdf).sum(axis=1), n_c - 1)

    c_k = draw()
    c_q = np.stack([draw() for _ in range(G)])
    return mu, pis, c_k, c_q


def _slice_fp32(cfg: dict, b: int, h: int, tables) -> tuple[np.ndarray, np.ndarray]:
    """Draw K [T, D] and the G query heads Q [G, T, D] (float32, before bf16 rounding)."""
    T, D = cfg["T"], cfg["D"]
    G = cfg["Hq"] // cfg["Hkv"]
    rng = np.random.default_rng([cfg["seed"], b, h])
    kind = cfg["kind"]
    if kind == "normal":
        k = rng.standard_normal((T, D), dtype=np.float32)
        q = rng.standard_normal((G, T, D), dtype=np.float32)
        return q, k
    if kind == "clusters":
        mu, pis, c_k, c_q = cluster_labels(rng, T, D, G)
        k = mu[c_k] + np.float32(0.5) * rng.standard_normal((T, D), dtype=np.float32)
        q = np.empty((G, T, D), dtype=np.float32)
        for g in range(G):
            q[g] = mu[c_q[g]] + rng.standard_normal((T, D), dtype=np.float32)
    else:
        k = rng.standard_normal((T, D), dtype=np.float32)
        q = rng.standard_normal((G, T, D), dtype=np.float32)
    k = rope(rmsnorm(k), tables=tables)
    q = rope(rmsnorm(q), tables=tables)
    if kind == "heavy":
        n_hh = -(-T // 100)  # ceil(0.01 T)
        pos = rng.choice(T, size=n_hh, replace=False)
        k[pos] *= np.float32(4.0)  # exact in bf16: a power-of-two scaling
    return q, k


def make_slice(name_or_cfg, b: int, h: int, T: Optional[int] = None):
    """Regenerate one (b, KV head h) slice: returns (q_bits [G,T,D], k_bits [T,D])."""
    cfg = dict(CONFIGS[name_or_cfg]) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    if T is not None:
        cfg["T"] = T
    tables = _rope_tables(cfg["T"], cfg["D"], 1e6) if cfg["kind"] != "normal" else None
    q, k = _slice_fp32(cfg, b, h, tables)
    return bf16_round_bits(q), bf16_round_bits(k)


def make(name_or_cfg, T: Optional[int] = None, B: Optional[int] = None, threads: Optional[int] = None,
         **overrides) -> Workload:
    """Generate a full workload. ``T``/``B``/``overrides`` shrink a config for tests."""
    cfg = dict(CONFIGS[name_or_cfg]) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    name = name_or_cfg if isinstance(name_or_cfg, str) else cfg.get("name", "custom")
    if T is not None:
        cfg["T"] = T
    if B is not None:
        cfg["B"] = B
    cfg.update(overrides)
    Bn, Hq, Hkv, T, D = cfg["B"], cfg["Hq"], cfg["Hkv"], cfg["T"], cfg["D"]
    G = Hq // Hkv
    q_bits = np.empty((Bn, Hq, T, D), dtype=np.uint16)
    k_bits = np.empty((Bn, Hkv, T, D), dtype=np.uint16)
    tables = _rope_tables(T, D, 1e6) if cfg["kind"] != "normal" else None

    def one(bh):
        b, h = bh
        q, k = _slice_fp32(cfg, b, h, tables)
        q_bits[b, h * G:(h + 1) * G] = bf16_round_bits(q)
        k_bits[b, h] = bf16_round_bits(k)

    jobs = [(b, h) for b in range(Bn) for h in range(Hkv)]
    nthr = threads if threads is not None else min(len(jobs), max(1, min(16, os.cpu_count() or 1)))
    if nthr <= 1 or len(jobs) == 1:
        for j in jobs:
            one(j)
    else:
        with _cf.ThreadPoolExecutor(nthr) as ex:
            list(ex.map(one, jobs))
    bias = None
    if cfg.get("sink"):
        bias = np.zeros(T, dtype=np.float32)
        bias[0] = 3.0
    scale = float(np.float32(cfg["scale"]))
    return Workload(name=name, B=Bn, Hq=Hq, Hkv=Hkv, T=T, D=D, scale=scale, q_bits=q_bits,
                    k_bits=k_bits, bias=bias, bands=list(cfg["bands"]), seed=int(cfg["seed"]))


def make_values(w: "Workload") -> np.ndarray:
    """Value rows for a workload, bf16 bits [B, Hkv, T, D]: N(0, 1) per element from the
    stream ``default_rng([seed, b, h, 1])`` (independent of the Q/K streams)."""
    v = np.empty((w.B, w.Hkv, w.T, w.D), dtype=np.uint16)
    for b in range(w.B):
        for h in range(w.Hkv):
            rng = np.random.default_rng([w.seed, b, h, 1])
            v[b, h] = bf16_round_bits(rng.standard_normal((w.T, w.D), dtype=np.float32))
    return v


def make_scores(w: "Workload") -> np.ndarray:
    """Per-token scorer outputs r[b, h, t] (float32 [B, Hkv, T]) standing in for a
    learned scorer's predictions: N(0, 1) from ``default_rng([seed, b, h, 2])``."""
    r = np.empty((w.B, w.Hkv, w.T), dtype=np.float32)
    for b in range(w.B):
        for h in range(w.Hkv):
            r[b, h] = np.random.default_rng([w.seed, b, h, 2]).standard_normal(w.T, dtype=np.float32)
    return r
