"""KVpop future-attention target on MI355X (gfx950).

A thin ctypes binding over the in-tree ``libkvpop.so`` (C ABI in ``include/kvpop.h``).
Every function here only marshals arguments: it checks tensor placement, dtype and
layout, derives the dimensions, allocates outputs with PyTorch when the caller
passes none, and calls the C entry point of the same name on the current HIP
stream. All arithmetic runs in the library's HIP kernels; there is no fallback.

Quantities (KVpop App. D.1): for query head qh and key position t,

    lse[b, qh, d] = log sum_{t <= d} exp(scale <q_d, k_t> + bias_t)       (pass 1)
    out[b, qh, t] = sum_{d = t + window}^{min(T - 1, t + horizon)}
                    exp(scale <q_d, k_t> + bias_t - lse[b, qh, d])       (pass 2)

with query head qh reading KV head qh // (Hq // Hkv); horizon < 0 = no limit.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

__all__ = [
    "KVPOP_OK", "KVPOP_EINVAL", "KVPOP_EUNSUPPORTED", "KVPOP_EHIP", "KvpopDims", "KvpopError",
    "lib", "lib_path", "kvpop_row_lse", "kvpop_future_attn_from_lse", "kvpop_future_attn_target",
    "kvpop_future_attn_scores", "kvpop_strerror", "kvpop_abi_version", "KVPOP_AGG_MAX", "KVPOP_AGG_MEAN",
    "KvpopTopkDims", "kvpop_running_topk", "kvpop_running_topk_workspace_size", "kvpop_sparse_attn_fwd",
    "kvpop_running_topk_noalloc", "KVPOP_ETOOBIG", "KVPOP_NOALLOC_SCRATCH_BYTES", "kvpop_future_attn_bands",
]

KVPOP_OK = 0
KVPOP_EINVAL = 1
KVPOP_EUNSUPPORTED = 2
KVPOP_EHIP = 3
KVPOP_ETOOBIG = 4
KVPOP_NOALLOC_SCRATCH_BYTES = 32 << 20
KVPOP_AGG_MAX = 0
KVPOP_AGG_MEAN = 1
ABI_VERSION = 3

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
_LIB: Optional[ctypes.CDLL] = None


class KvpopDims(ctypes.Structure):
    """Mirror of ``kvpop_dims`` in include/kvpop.h."""
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("seq_len", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("scale", ctypes.c_float),
    ]


class KvpopTopkDims(ctypes.Structure):
    """Mirror of ``kvpop_topk_dims`` in include/kvpop.h."""
    _fields_ = [("batch", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("seq_len", ctypes.c_int32)]


class KvpopError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s failed with status %d: %s" % (where, status, kvpop_strerror(status)))
        self.status = status


def lib_path() -> str:
    return os.environ.get("KVPOP_LIB", os.path.join(_PKG_DIR, "libkvpop.so"))


def lib() -> ctypes.CDLL:
    """Load the built library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError("libkvpop.so not found at %s: build it with "
                               "`python -m paper_2607_05061_amd.build`" % path)
        L = ctypes.CDLL(path)
        P, I32, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
        D = ctypes.POINTER(KvpopDims)
        L.kvpop_row_lse.argtypes = [D, P, P, P, P, P]
        L.kvpop_row_lse.restype = ctypes.c_int
        L.kvpop_future_attn_from_lse.argtypes = [D, P, P, P, P, I32, I32, P, P]
        L.kvpop_future_attn_from_lse.restype = ctypes.c_int
        L.kvpop_future_attn_bands.argtypes = [D, P, P, P, P, I32, ctypes.POINTER(I32), ctypes.POINTER(I32),
                                              ctypes.POINTER(P), P]
        L.kvpop_future_attn_bands.restype = ctypes.c_int
        L.kvpop_future_attn_target.argtypes = [D, P, P, P, I32, I32, P, P, P]
        L.kvpop_future_attn_target.restype = ctypes.c_int
        L.kvpop_future_attn_scores.argtypes = [D, P, P, P, P, I32, I32, I32, F, I32, P, P, P]
        L.kvpop_future_attn_scores.restype = ctypes.c_int
        L.kvpop_running_topk_workspace_size.argtypes = [ctypes.POINTER(KvpopTopkDims)]
        L.kvpop_running_topk_workspace_size.restype = ctypes.c_size_t
        L.kvpop_running_topk.argtypes = [ctypes.POINTER(KvpopTopkDims), P, P, I32, I32, I32, P, P, P, P, P, P,
                                         ctypes.c_size_t, P]
        L.kvpop_running_topk.restype = ctypes.c_int
        L.kvpop_running_topk_noalloc.argtypes = [ctypes.POINTER(KvpopTopkDims), P, P, I32, I32, I32, P, P, P, P, P,
                                                 P]
        L.kvpop_running_topk_noalloc.restype = ctypes.c_int
        L.kvpop_sparse_attn_fwd.argtypes = [ctypes.POINTER(KvpopDims), P, P, P, P, P, P, P, P]
        L.kvpop_sparse_attn_fwd.restype = ctypes.c_int
        L.kvpop_strerror.argtypes = [ctypes.c_int]
        L.kvpop_strerror.restype = ctypes.c_char_p
        L.kvpop_abi_version.argtypes = []
        L.kvpop_abi_version.restype = ctypes.c_int
        if L.kvpop_abi_version() != ABI_VERSION:
            raise RuntimeError("libkvpop ABI version %d, binding expects %d" % (L.kvpop_abi_version(), ABI_VERSION))
        _LIB = L
    return _LIB


def kvpop_strerror(status: int) -> str:
    return lib().kvpop_strerror(int(status)).decode()


def kvpop_abi_version() -> int:
    return int(lib().kvpop_abi_version())


# ---------------------------------------------------------------------------
# torch-tensor marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch  # noqa: WPS433 (PyTorch only provides device memory and streams)
    return torch


def _dims(q, k, scale: float) -> KvpopDims:
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("q must be [B, Hq, T, D] and k [B, Hkv, T, D]")
    B, Hq, T, D = q.shape
    if k.shape[0] != B or k.shape[2] != T or k.shape[3] != D:
        raise ValueError("q %s and k %s disagree on B, T or D" % (tuple(q.shape), tuple(k.shape)))
    return KvpopDims(B, Hq, k.shape[1], T, D, float(scale))


def _check_tensor(x, name: str, dtype, device):
    torch = _torch()
    if not isinstance(x, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if x.device.type != "cuda" or (device is not None and x.device != device):
        raise ValueError("%s must be on the GPU device of q" % name)
    if x.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, x.dtype))
    if not x.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _stream_ptr(stream, device) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return int(s.cuda_stream)


def _prep_inputs(q, k, key_bias):
    torch = _torch()
    _check_tensor(q, "q", torch.bfloat16, None)
    _check_tensor(k, "k", torch.bfloat16, q.device)
    if key_bias is not None:
        _check_tensor(key_bias, "key_bias", torch.float32, q.device)
        if key_bias.dim() != 1 or key_bias.shape[0] != q.shape[2]:
            raise ValueError("key_bias must be [T]")
    return q.data_ptr(), k.data_ptr(), (key_bias.data_ptr() if key_bias is not None else None)


def _prep_out(x, name, shape, device):
    torch = _torch()
    if x is None:
        return torch.empty(shape, dtype=torch.float32, device=device)
    _check_tensor(x, name, torch.float32, device)
    if tuple(x.shape) != tuple(shape):
        raise ValueError("%s must have shape %s" % (name, tuple(shape)))
    return x


def kvpop_row_lse(q, k, scale: float, key_bias=None, lse=None, stream=None):
    """Pass 1: dense causal row log-normaliser, fp32 [B, Hq, T] (eq. dense_lse_app)."""
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    lse = _prep_out(lse, "lse", (d.batch, d.n_q_heads, d.seq_len), q.device)
    st = lib().kvpop_row_lse(ctypes.byref(d), qp, kp, bp, lse.data_ptr(), _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_row_lse")
    return lse


def kvpop_future_attn_from_lse(q, k, lse, scale: float, window: int = 0, horizon: int = -1, key_bias=None,
                               out=None, stream=None):
    """Pass 2: per-key future mass from a given normaliser, fp32 [B, Hq, T] (eq. future_mass_app)."""
    torch = _torch()
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    _check_tensor(lse, "lse", torch.float32, q.device)
    if tuple(lse.shape) != (d.batch, d.n_q_heads, d.seq_len):
        raise ValueError("lse must be [B, Hq, T]")
    out = _prep_out(out, "out", (d.batch, d.n_q_heads, d.seq_len), q.device)
    st = lib().kvpop_future_attn_from_lse(ctypes.byref(d), qp, kp, bp, lse.data_ptr(), int(window), int(horizon),
                                          out.data_ptr(), _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_future_attn_from_lse")
    return out


def kvpop_future_attn_bands(q, k, lse, scale: float, bands, key_bias=None, outs=None, stream=None):
    """Pass 2 for one or two (window, horizon) bands from one normaliser in one sweep;
    returns a list of fp32 [B, Hq, T] masses, one per band."""
    torch = _torch()
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    _check_tensor(lse, "lse", torch.float32, q.device)
    shape = (d.batch, d.n_q_heads, d.seq_len)
    if tuple(lse.shape) != shape:
        raise ValueError("lse must be [B, Hq, T]")
    bands = [(int(a), int(b)) for a, b in bands]
    if not 1 <= len(bands) <= 2:
        raise ValueError("one or two bands")
    outs = [None] * len(bands) if outs is None else list(outs)
    if len(outs) != len(bands):
        raise ValueError("one output per band")
    outs = [_prep_out(o, "outs[%d]" % i, shape, q.device) for i, o in enumerate(outs)]
    n = len(bands)
    win = (ctypes.c_int32 * n)(*[b[0] for b in bands])
    hor = (ctypes.c_int32 * n)(*[b[1] for b in bands])
    ptr = (ctypes.c_void_p * n)(*[o.data_ptr() for o in outs])
    st = lib().kvpop_future_attn_bands(ctypes.byref(d), qp, kp, bp, lse.data_ptr(), n, win, hor, ptr,
                                       _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_future_attn_bands")
    return outs


def kvpop_future_attn_target(q, k, scale: float, window: int = 0, horizon: int = -1, key_bias=None,
                             lse_ws=None, out=None, stream=None) -> Tuple["object", "object"]:
    """Both passes; returns (out, lse) where lse is the dense normaliser of pass 1."""
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    shape = (d.batch, d.n_q_heads, d.seq_len)
    lse_ws = _prep_out(lse_ws, "lse_ws", shape, q.device)
    out = _prep_out(out, "out", shape, q.device)
    st = lib().kvpop_future_attn_target(ctypes.byref(d), qp, kp, bp, int(window), int(horizon), lse_ws.data_ptr(),
                                        out.data_ptr(), _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_future_attn_target")
    return out, lse_ws


def kvpop_future_attn_scores(q, k, lse, scale: float, window: int = 0, horizon: int = -1, agg: str = "max",
                             eps: float = 1e-8, normalize: bool = True, key_bias=None, scores=None, out=None,
                             write_mass: bool = False, stream=None):
    """Pass 2 plus the target epilogue (App. D.4 step 5): per-KV-head scores
    log(agg_g m_bar + eps) - log N_t, fp32 [B, Hkv, T]. Returns (scores, out), where
    out holds the per-head masses if ``write_mass`` (or ``out``) is given, else None."""
    torch = _torch()
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    _check_tensor(lse, "lse", torch.float32, q.device)
    if tuple(lse.shape) != (d.batch, d.n_q_heads, d.seq_len):
        raise ValueError("lse must be [B, Hq, T]")
    if agg not in ("max", "mean"):
        raise ValueError("agg must be 'max' or 'mean'")
    scores = _prep_out(scores, "scores", (d.batch, d.n_kv_heads, d.seq_len), q.device)
    if out is not None or write_mass:
        out = _prep_out(out, "out", (d.batch, d.n_q_heads, d.seq_len), q.device)
    st = lib().kvpop_future_attn_scores(ctypes.byref(d), qp, kp, bp, lse.data_ptr(), int(window), int(horizon),
                                        KVPOP_AGG_MAX if agg == "max" else KVPOP_AGG_MEAN, float(eps),
                                        int(bool(normalize)), out.data_ptr() if out is not None else None,
                                        scores.data_ptr(), _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_future_attn_scores")
    return scores, out


def kvpop_running_topk_workspace_size(batch: int, n_heads: int, seq_len: int) -> int:
    d = KvpopTopkDims(batch, n_heads, seq_len)
    return int(lib().kvpop_running_topk_workspace_size(ctypes.byref(d)))


def kvpop_running_topk(scores, sinks: int, window: int, topk: int, log_gamma=None, labels: bool = True,
                       evict: bool = False, workspace=None, stream=None):
    """Ranks, running cutoffs and (optionally) teacher labels and boundary tokens, and
    token eviction queries, for scores [B, H, T] (App. B.3, App. C). Returns a dict of
    int32 tensors."""
    torch = _torch()
    _check_tensor(scores, "scores", torch.float32, None)
    if scores.dim() != 3:
        raise ValueError("scores must be [B, H, T]")
    B, H, T = scores.shape
    if log_gamma is not None:
        _check_tensor(log_gamma, "log_gamma", torch.float32, scores.device)
        if tuple(log_gamma.shape) != (H,):
            raise ValueError("log_gamma must be [H]")
    need = kvpop_running_topk_workspace_size(B, H, T)
    if need == 0:
        raise ValueError("invalid dimensions")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=scores.device)
    elif workspace.numel() * workspace.element_size() < need or workspace.device != scores.device:
        raise ValueError("workspace must hold %d bytes on the device of scores" % need)
    out = {n: torch.empty((B, H, T), dtype=torch.int32, device=scores.device) for n in ("rank", "cutoff")}
    if labels:
        out["label"] = torch.empty((B, H, T), dtype=torch.int32, device=scores.device)
        out["boundary"] = torch.empty((B, H, T), dtype=torch.int32, device=scores.device)
    if evict:
        out["evict"] = torch.empty((B, H, T), dtype=torch.int32, device=scores.device)
    d = KvpopTopkDims(B, H, T)
    st = lib().kvpop_running_topk(ctypes.byref(d), scores.data_ptr(),
                                  log_gamma.data_ptr() if log_gamma is not None else None, int(sinks), int(window),
                                  int(topk), out["rank"].data_ptr(), out["cutoff"].data_ptr(),
                                  out["label"].data_ptr() if labels else None,
                                  out["boundary"].data_ptr() if labels else None,
                                  out["evict"].data_ptr() if evict else None, workspace.data_ptr(),
                                  workspace.numel() * workspace.element_size(), _stream_ptr(stream, scores.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_running_topk")
    return out


def kvpop_running_topk_noalloc(scores, sinks: int, window: int, topk: int, log_gamma=None, labels: bool = True,
                               evict: bool = False, out=None, stream=None):
    """kvpop_running_topk without a workspace: the library's own per-GPU scratch array
    serves instead (see include/kvpop.h). ``out`` may hold preallocated int32 [B, H, T]
    outputs ("rank", "cutoff" and, as requested, "label", "boundary", "evict"), so that
    the call itself allocates nothing; missing ones are allocated here."""
    torch = _torch()
    _check_tensor(scores, "scores", torch.float32, None)
    if scores.dim() != 3:
        raise ValueError("scores must be [B, H, T]")
    B, H, T = scores.shape
    if log_gamma is not None:
        _check_tensor(log_gamma, "log_gamma", torch.float32, scores.device)
        if tuple(log_gamma.shape) != (H,):
            raise ValueError("log_gamma must be [H]")
    names = ["rank", "cutoff"] + (["label", "boundary"] if labels else []) + (["evict"] if evict else [])
    res = {}
    for n in names:
        x = (out or {}).get(n)
        if x is None:
            x = torch.empty((B, H, T), dtype=torch.int32, device=scores.device)
        else:
            _check_tensor(x, n, torch.int32, scores.device)
            if tuple(x.shape) != (B, H, T):
                raise ValueError("%s must be [B, H, T]" % n)
        res[n] = x
    d = KvpopTopkDims(B, H, T)
    ptr = lambda n: res[n].data_ptr() if n in res else None  # noqa: E731
    st = lib().kvpop_running_topk_noalloc(ctypes.byref(d), scores.data_ptr(),
                                          log_gamma.data_ptr() if log_gamma is not None else None, int(sinks),
                                          int(window), int(topk), ptr("rank"), ptr("cutoff"), ptr("label"),
                                          ptr("boundary"), ptr("evict"), _stream_ptr(stream, scores.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_running_topk_noalloc")
    return res


def kvpop_sparse_attn_fwd(q, k, v, evict, scale: float, key_bias=None, o=None, lse=None, stream=None):
    """Running top-k sparse attention forward (Sec. 3.2, App. C): key t of KV head h is
    kept by query q iff t <= q < evict[b, h, t]. Returns (o bf16 [B, Hq, T, D],
    lse fp32 [B, Hq, T])."""
    torch = _torch()
    d = _dims(q, k, scale)
    qp, kp, bp = _prep_inputs(q, k, key_bias)
    _check_tensor(v, "v", torch.bfloat16, q.device)
    if tuple(v.shape) != tuple(k.shape):
        raise ValueError("v must have the shape of k")
    _check_tensor(evict, "evict", torch.int32, q.device)
    if tuple(evict.shape) != (d.batch, d.n_kv_heads, d.seq_len):
        raise ValueError("evict must be [B, Hkv, T]")
    if o is None:
        o = torch.empty(tuple(q.shape), dtype=torch.bfloat16, device=q.device)
    else:
        _check_tensor(o, "o", torch.bfloat16, q.device)
        if tuple(o.shape) != tuple(q.shape):
            raise ValueError("o must have the shape of q")
    lse = _prep_out(lse, "lse", (d.batch, d.n_q_heads, d.seq_len), q.device)
    st = lib().kvpop_sparse_attn_fwd(ctypes.byref(d), qp, kp, v.data_ptr(), bp, evict.data_ptr(), o.data_ptr(),
                                     lse.data_ptr(), _stream_ptr(stream, q.device))
    if st != KVPOP_OK:
        raise KvpopError(st, "kvpop_sparse_attn_fwd")
    return o, lse
