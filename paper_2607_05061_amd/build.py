"""Build the in-tree shared library ``libkvpop.so`` for gfx950 with hipcc.

Run as ``python -m paper_2607_05061_amd.build``. The library has no PyTorch
dependency: its C ABI (include/kvpop.h) takes plain device pointers.
"""
from __future__ import annotations

import os
import subprocess
import sys

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


def build(out: str = LIB_PATH, verbose: bool = False, extra_flags=()) -> str:
    """Compile every source into ``out`` (atomically replaced). Returns the path."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIP_FLAGS, *extra_flags, "-shared", "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        try:
            os.unlink(tmp)
        except OSError:
            pass
        raise RuntimeError("hipcc failed (%d):\n%s\n%s" % (r.returncode, r.stdout, r.stderr))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
