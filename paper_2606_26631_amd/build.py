"""Build the HIP library libprcr.so for gfx950 (in-tree, next to this file).

Every source is compiled with hipcc for gfx950 only; the library is linked into
the package directory so that the Python binding, the tests and the benchmark
load it from the source tree.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "libprcr.so")
BUILD_DIR = os.path.join(ROOT, "_build")

# The bandwidth measurement's reference copies (a plain streaming copy and a copy
# with the rebinding kernel's access pattern), in a library of their own: they are
# not part of the PRCR path or its ABI.
COPYREF_SOURCES = ["copyref.hip"]
COPYREF_OUT = os.path.join(PKG, "libprcr_copyref.so")
SOURCES = ["api.cpp", "axis_map.cpp", "decode.hip", "decode_static.hip", "prefill.hip", "reassign.hip", "rebind.hip", "store_raw.hip"]

# Packed-FP32 instructions are disabled for all device code; the host pass of
# hipcc warns that it does not know the feature, which is harmless.
FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         f"-I{INCLUDE}", f"-I{CSRC}"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; install ROCm or set HIPCC")


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"]
    cmd = [hipcc(), *lang, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    if verbose and r.stderr.strip():
        print(r.stderr, file=sys.stderr)
    return obj


def _link(objs, out: str, verbose: bool) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libprcr.so, and the measurement's
    reference copy kernels into libprcr_copyref.so; returns libprcr.so's path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + len(COPYREF_SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES + COPYREF_SOURCES))
    _link(objs[:len(SOURCES)], OUT, verbose)
    _link(objs[len(SOURCES):], COPYREF_OUT, verbose)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
