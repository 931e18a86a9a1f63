"""Build the in-tree shared library ``libkvpop.so`` for gfx950 with hipcc.

Run as ``python -m paper_2607_05061_amd.build``. The library has no PyTorch
dependency: its C ABI (include/kvpop.h) takes plain device pointers. Each source
is compiled to its own object (in parallel), then the objects are linked.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libkvpop.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
SOURCES = ["kvpop_api.cpp", "kvpop_kernels.hip", "kvpop_topk.hip", "kvpop_sparse_attn.hip"]

# Packed fp32 VALU forms are disabled for all device code.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s\n%s\n%s" % (r.returncode, " ".join(cmd), r.stdout, r.stderr))


def build(out: str = LIB_PATH, verbose: bool = False, extra_flags=()) -> str:
    """Compile every source into ``out`` (atomically replaced). Returns the path."""
    tmp = out + ".tmp%d" % os.getpid()
    with tempfile.TemporaryDirectory(prefix="kvpop_build_") as objdir:
        objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        cmds = [[hipcc(), *HIP_FLAGS, *extra_flags, "-c", "-I", INCLUDE, "-I", CSRC, os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        with cf.ThreadPoolExecutor(len(cmds)) as ex:
            list(ex.map(lambda c: _run(c, verbose), cmds))
        try:
            _run([hipcc(), *HIP_FLAGS, *extra_flags, "-shared", *objs, "-o", tmp], verbose)
        except Exception:
            try:
                os.unlink(tmp)
            except OSError:
                pass
            raise
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
