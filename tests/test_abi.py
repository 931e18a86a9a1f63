"""The C ABI library loads, exports every declared entry point, and rejects bad
arguments with the documented status before launching anything (no GPU needed)."""
import ctypes
import math
import os
import re

import pytest

import paper_2607_05061_amd as kv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvpop.h")

pytestmark = pytest.mark.skipif(not os.path.exists(kv.lib_path()),
                                reason="libkvpop.so not built (python -m paper_2607_05061_amd.build)")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(kvpop_\w+)\s*\(", src, flags=re.M)


def test_header_declares_the_entry_points():
    names = set(_declared_functions())
    assert names == {"kvpop_row_lse", "kvpop_future_attn_from_lse", "kvpop_future_attn_target",
                     "kvpop_future_attn_scores", "kvpop_running_topk", "kvpop_running_topk_workspace_size",
                     "kvpop_sparse_attn_fwd", "kvpop_strerror", "kvpop_abi_version", "kvpop_running_topk_noalloc",
                     "kvpop_future_attn_bands"}


def test_library_exports_every_declared_symbol():
    L = kv.lib()
    for name in _declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_abi_version_and_strerror():
    assert kv.kvpop_abi_version() == kv.ABI_VERSION == 3
    texts = {c: kv.kvpop_strerror(c) for c in (kv.KVPOP_OK, kv.KVPOP_EINVAL, kv.KVPOP_EUNSUPPORTED, kv.KVPOP_EHIP,
                                               kv.KVPOP_ETOOBIG, 99)}
    assert texts[kv.KVPOP_OK] == "success"
    assert "invalid" in texts[kv.KVPOP_EINVAL]
    assert "unsupported" in texts[kv.KVPOP_EUNSUPPORTED]
    assert "HIP" in texts[kv.KVPOP_EHIP]
    assert "unknown" in texts[99]
    assert "no-allocation" in texts[kv.KVPOP_ETOOBIG]
    assert len(set(texts.values())) == 6


# Fake device addresses: never dereferenced, because every call below must be
# rejected during validation.
A, B_, C_, D_, E_ = 0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000


def _dims(B=1, Hq=4, Hkv=2, T=64, D=128, scale=0.125):
    return kv.KvpopDims(B, Hq, Hkv, T, D, scale)


def _lse(d, q=A, k=B_, bias=None, out=C_):
    return kv.lib().kvpop_row_lse(ctypes.byref(d) if d is not None else None, q, k, bias, out, None)


def _p2(d, q=A, k=B_, bias=None, lse=C_, w=0, h=-1, out=D_):
    return kv.lib().kvpop_future_attn_from_lse(ctypes.byref(d) if d is not None else None, q, k, bias, lse, w, h, out,
                                               None)


def _tgt(d, q=A, k=B_, bias=None, w=0, h=-1, ws=C_, out=D_):
    return kv.lib().kvpop_future_attn_target(ctypes.byref(d) if d is not None else None, q, k, bias, w, h, ws, out,
                                             None)


def _sc(d, q=A, k=B_, bias=None, lse=C_, w=0, h=-1, agg=0, eps=1e-8, norm=1, out=None, scores=D_):
    return kv.lib().kvpop_future_attn_scores(ctypes.byref(d) if d is not None else None, q, k, bias, lse, w, h, agg,
                                             eps, norm, out, scores, None)


def _bd(d, q=A, k=B_, bias=None, lse=C_, bands=((0, -1), (1, 4096)), outs=(D_, E_), n=None, null=None):
    n = len(bands) if n is None else n
    m = max(1, len(bands))
    w = (ctypes.c_int32 * m)(*[b[0] for b in bands])
    h = (ctypes.c_int32 * m)(*[b[1] for b in bands])
    o = (ctypes.c_void_p * max(1, len(outs)))(*outs)
    args = {"w": w, "h": h, "o": o}
    if null:
        args[null] = None
    return kv.lib().kvpop_future_attn_bands(ctypes.byref(d) if d is not None else None, q, k, bias, lse, n,
                                            args["w"], args["h"], args["o"], None)


EINVAL, EUNS = kv.KVPOP_EINVAL, kv.KVPOP_EUNSUPPORTED


def test_bands_argument_checks():
    """kvpop_future_attn_bands validates like pass 2, per band (fake pointers, nothing launched)."""
    d = _dims()
    assert _bd(None) == EINVAL
    assert _bd(d, n=0) == EINVAL
    assert _bd(d, n=3) == EINVAL
    for name in ("w", "h", "o"):
        assert _bd(d, null=name) == EINVAL, name
    assert _bd(d, lse=None) == EINVAL
    assert _bd(d, lse=C_ + 8) == EUNS
    assert _bd(d, bands=((0, -1), (-1, 5))) == EINVAL
    assert _bd(d, bands=((3, 2), (1, 5))) == EINVAL
    assert _bd(d, outs=(D_, D_ + 64)) == EINVAL       # the two outputs overlap
    assert _bd(d, outs=(D_, C_)) == EINVAL            # an output over the normaliser
    assert _bd(d, outs=(D_, A + 16)) == EINVAL        # an output over q
    assert _bd(d, outs=(D_, E_ + 4)) == EUNS
    assert _bd(d, outs=(None, E_)) == EINVAL
    assert _bd(_dims(D=96)) == EUNS


@pytest.mark.parametrize("call", [_lse, _p2, _tgt, _sc])
def test_bad_dims(call):
    assert call(None) == EINVAL
    for kw in (dict(B=0), dict(Hq=0), dict(Hkv=0), dict(T=0), dict(D=0), dict(B=-1), dict(T=-5)):
        assert call(_dims(**kw)) == EINVAL, kw
    assert call(_dims(Hq=6, Hkv=4)) == EINVAL
    for s in (0.0, -0.1, math.inf, math.nan):
        assert call(_dims(scale=s)) == EINVAL, s
    for dd in (32, 96, 256, 80):
        assert call(_dims(D=dd)) == EUNS, dd
    assert call(_dims(T=(1 << 24) + 1)) == EUNS


@pytest.mark.parametrize("call", [_lse, _p2, _tgt, _sc])
def test_null_and_misaligned_pointers(call):
    d = _dims()
    assert call(d, q=None) == EINVAL
    assert call(d, k=None) == EINVAL
    assert call(d, q=A + 8) == EUNS
    assert call(d, k=B_ + 2) == EUNS
    assert call(d, bias=E_ + 4) == EUNS


def test_output_pointer_checks():
    d = _dims()
    assert _lse(d, out=None) == EINVAL
    assert _lse(d, out=C_ + 4) == EUNS
    assert _p2(d, out=None) == EINVAL
    assert _p2(d, lse=None) == EINVAL
    assert _p2(d, lse=C_ + 8) == EUNS
    assert _tgt(d, ws=None) == EINVAL
    assert _tgt(d, out=None) == EINVAL


def test_overlapping_buffers_rejected():
    d = _dims()  # Q is 1*4*64*128*2 = 64 KiB
    assert _lse(d, out=A + 4096) == EINVAL          # lse inside Q
    assert _p2(d, out=C_) == EINVAL                # out == lse
    assert _tgt(d, ws=D_, out=D_ + 16) == EINVAL    # out overlaps workspace
    assert _p2(d, bias=E_, out=E_) == EINVAL        # out over the bias


def test_epilogue_option_checks():
    d = _dims()
    assert _sc(d, agg=2) == EINVAL
    assert _sc(d, agg=-1) == EINVAL
    assert _sc(d, norm=2) == EINVAL
    assert _sc(d, eps=-1e-3) == EINVAL
    assert _sc(d, eps=math.inf) == EINVAL
    assert _sc(d, eps=math.nan) == EINVAL
    assert _sc(d, scores=None) == EINVAL
    assert _sc(d, scores=D_ + 4) == EUNS
    assert _sc(d, lse=None) == EINVAL
    assert _sc(d, out=D_ + 64) == EINVAL          # out overlaps scores
    assert _sc(d, scores=C_ + 16) == EINVAL       # scores inside lse
    assert _sc(d, out=E_ + 8) == EUNS             # misaligned optional out


@pytest.mark.parametrize("call", [_p2, _tgt, _sc])
def test_bad_bands(call):
    d = _dims()
    assert call(d, w=-1) == EINVAL
    assert call(d, w=3, h=2) == EINVAL
    assert call(d, w=5, h=0) == EINVAL


def test_python_binding_rejects_cpu_tensors():
    torch = pytest.importorskip("torch")
    q = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        kv.kvpop_row_lse(q, q, 0.125)


def _tk(dims=(2, 3, 100), scores=A, lg=None, s=4, w=8, k=5, rank=B_, cut=C_, lab=None, bnd=None, ev=None, ws=E_,
        wsb=None):
    d = kv.KvpopTopkDims(*dims) if dims is not None else None
    if wsb is None:
        wsb = kv.kvpop_running_topk_workspace_size(*dims) if dims is not None else 0
    return kv.lib().kvpop_running_topk(ctypes.byref(d) if d is not None else None, scores, lg, s, w, k, rank, cut,
                                       lab, bnd, ev, ws, wsb, None)


def test_running_topk_workspace_size():
    assert kv.kvpop_running_topk_workspace_size(0, 1, 10) == 0
    assert kv.kvpop_running_topk_workspace_size(1, 1, (1 << 24) + 1) == 0
    a = kv.kvpop_running_topk_workspace_size(1, 1, 1000)
    b = kv.kvpop_running_topk_workspace_size(2, 3, 1000)
    assert a > 0 and b == 6 * a and a % 4 == 0


def test_running_topk_argument_checks():
    assert _tk(dims=None) == EINVAL
    for dims in [(0, 1, 10), (1, 0, 10), (1, 1, 0)]:
        assert _tk(dims=dims, wsb=1 << 20) == EINVAL
    assert _tk(dims=(1, 1, (1 << 24) + 1), wsb=1 << 40) == EUNS
    assert _tk(s=-1) == EINVAL
    assert _tk(w=-1) == EINVAL
    assert _tk(k=0) == EINVAL
    assert _tk(scores=None) == EINVAL
    assert _tk(rank=None) == EINVAL
    assert _tk(cut=None) == EINVAL
    assert _tk(ws=None) == EINVAL
    need = kv.kvpop_running_topk_workspace_size(2, 3, 100)
    assert _tk(wsb=need - 1) == EINVAL
    assert _tk(scores=A + 4) == EUNS
    assert _tk(lab=D_ + 8) == EUNS
    assert _tk(cut=B_ + 16) == EINVAL                 # rank and cutoff overlap
    assert _tk(lab=A + 16) == EINVAL                  # label over the scores
    assert _tk(ws=C_ - 64) == EINVAL                  # workspace over the cutoff
    assert _tk(ev=D_ + 4) == EUNS                     # misaligned eviction output
    assert _tk(ev=C_ + 16) == EINVAL                  # eviction output over the cutoff


def _tkn(dims=(2, 3, 100), scores=A, lg=None, s=4, w=8, k=5, rank=B_, cut=C_, lab=None, bnd=None, ev=None):
    d = kv.KvpopTopkDims(*dims) if dims is not None else None
    return kv.lib().kvpop_running_topk_noalloc(ctypes.byref(d) if d is not None else None, scores, lg, s, w, k,
                                               rank, cut, lab, bnd, ev, None)


def test_running_topk_noalloc_argument_checks():
    """The no-allocation variant validates like kvpop_running_topk and rejects a
    problem whose workspace exceeds its scratch array (nothing is launched)."""
    assert kv.KVPOP_NOALLOC_SCRATCH_BYTES == 32 << 20
    assert _tkn(dims=None) == EINVAL
    for dims in [(0, 1, 10), (1, 0, 10), (1, 1, 0)]:
        assert _tkn(dims=dims) == EINVAL
    assert _tkn(dims=(1, 1, (1 << 24) + 1)) == EUNS
    assert _tkn(s=-1) == EINVAL
    assert _tkn(w=-1) == EINVAL
    assert _tkn(k=0) == EINVAL
    assert _tkn(scores=None) == EINVAL
    assert _tkn(rank=None) == EINVAL
    assert _tkn(cut=None) == EINVAL
    assert _tkn(scores=A + 4) == EUNS
    assert _tkn(cut=B_ + 16) == EINVAL
    assert _tkn(lab=A + 16) == EINVAL
    # the largest problems that fit, and the first ones that do not
    assert kv.kvpop_running_topk_workspace_size(4, 8, 32768) <= kv.KVPOP_NOALLOC_SCRATCH_BYTES
    assert kv.kvpop_running_topk_workspace_size(1, 8, 131072) <= kv.KVPOP_NOALLOC_SCRATCH_BYTES
    assert kv.kvpop_running_topk_workspace_size(5, 8, 32768) > kv.KVPOP_NOALLOC_SCRATCH_BYTES
    assert _tkn(dims=(5, 8, 32768)) == kv.KVPOP_ETOOBIG
    assert _tkn(dims=(1, 1, 2_000_000)) == kv.KVPOP_ETOOBIG


F_, G_ = 0x60000000, 0x70000000


def _sa(d, q=A, k=B_, v=C_, bias=None, ev=D_, o=E_, lse=F_):
    return kv.lib().kvpop_sparse_attn_fwd(ctypes.byref(d) if d is not None else None, q, k, v, bias, ev, o, lse,
                                          None)


def test_sparse_attn_argument_checks():
    """Every call here is rejected during validation (the pointers are fake)."""
    d = _dims()
    assert _sa(None) == EINVAL
    assert _sa(_dims(Hq=3, Hkv=2)) == EINVAL             # Hq % Hkv != 0
    assert _sa(_dims(Hq=6, Hkv=2)) == EUNS               # G = 3, not a power of two
    assert _sa(_dims(D=96)) == EUNS
    assert _sa(_dims(T=1 << 23)) == EUNS                 # T * D * 2 >= 2^31
    assert _sa(_dims(scale=0.0)) == EINVAL
    for name in ("q", "k", "v", "ev", "o", "lse"):
        assert _sa(d, **{name: None}) == EINVAL, name
    for name in ("q", "k", "v", "ev", "o", "lse"):
        assert _sa(d, **{name: {"q": A, "k": B_, "v": C_, "ev": D_, "o": E_, "lse": F_}[name] + 8}) == EUNS, name
    assert _sa(d, o=A + 64) == EINVAL                    # o over q
    assert _sa(d, lse=C_ + 16) == EINVAL                 # lse over v
    assert _sa(d, o=D_ - 16) == EINVAL                   # o over evict
    assert _sa(d, lse=E_ + 32) == EINVAL                 # lse over o


def test_forced_hip_error_path(monkeypatch):
    """The KVPOP_EHIP path, forced from the host (no GPU, nothing launched): with
    KVPOP_TEST_FORCE_EHIP set to a HIP error code, every entry point that passes
    validation returns KVPOP_EHIP, and kvpop_strerror(KVPOP_EHIP) returns that
    error's text on the calling thread only."""
    import threading
    code = 719  # hipErrorLaunchFailure
    monkeypatch.setenv("KVPOP_TEST_FORCE_EHIP", str(code))
    d = _dims()
    calls = [lambda: _lse(d), lambda: _p2(d), lambda: _tgt(d), lambda: _sc(d), lambda: _tk(),
             lambda: _sa(d), lambda: _tkn(), lambda: _bd(d)]
    for c in calls:
        assert c() == kv.KVPOP_EHIP
        text = kv.kvpop_strerror(kv.KVPOP_EHIP)
        assert text.startswith("HIP error: ") and len(text) > len("HIP error: ")
    # validation still comes first
    assert _lse(_dims(B=0)) == EINVAL
    assert _sa(d, q=None) == EINVAL
    # the text is per thread: a thread that has not failed sees the generic text
    seen = []
    th = threading.Thread(target=lambda: seen.append(kv.kvpop_strerror(kv.KVPOP_EHIP)))
    th.start()
    th.join()
    assert seen == ["HIP runtime error"]
    # the binding's exception carries the status and this thread's text
    err = kv.KvpopError(_lse(d), "kvpop_row_lse")
    assert err.status == kv.KVPOP_EHIP and "HIP error: " in str(err)
    monkeypatch.delenv("KVPOP_TEST_FORCE_EHIP")
    assert _lse(_dims(B=0)) == EINVAL
