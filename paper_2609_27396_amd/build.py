"""Build libdpara.so (gfx950) in-tree with hipcc.

    python -m paper_2609_27396_amd.build [--release-only]

Each csrc/*.hip file is compiled to an object under _build/ (in parallel), then
linked into paper_2609_27396_amd/libdpara.so.  Two test flavours are built
beside it: libdpara_asan.so instruments the host code (the C ABI's validation
and planning layer) with AddressSanitizer, and libdpara_debug.so fills every
kernel's LDS ring with NaN before its first DMA (DPARA_DEBUG_LDS_POISON), so
that a read of LDS the DMA did not write shows in the outputs.  The tests load
them through DPARA_LIB_PATH.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libdpara.so")
ASAN_LIB = os.path.join(PKG, "libdpara_asan.so")
DEBUG_LIB = os.path.join(PKG, "libdpara_debug.so")
# host-only instrumentation: each sanitizer flag applies to the host pass alone
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
DEBUG_FLAGS = ["-DDPARA_DEBUG_LDS_POISON=1"]
FLAVOURS = {"release": (LIB, "", []), "asan": (ASAN_LIB, "asan", ASAN_FLAGS), "debug": (DEBUG_LIB, "debug", DEBUG_FLAGS)}

ARCH = "gfx950"
# Packed fp32 instructions stay disabled in every HIP translation unit.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wno-unused-result"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def sources() -> list:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src: str, verbose: bool, flavour: str = "release") -> str:
    _, sub, extra = FLAVOURS[flavour]
    obj = os.path.join(BUILD, sub, os.path.basename(src)[:-4] + ".o")
    cmd = [hipcc(), *HIP_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature; that warning is expected
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return obj


def _build_flavour(verbose: bool, flavour: str) -> str:
    out, sub, _ = FLAVOURS[flavour]
    os.makedirs(os.path.join(BUILD, sub), exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, flavour), srcs))
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)
    return out


def build(verbose: bool = False, test_flavours: bool = True) -> str:
    """Build libdpara.so and (test_flavours) libdpara_asan.so and libdpara_debug.so beside it."""
    lib = _build_flavour(verbose, "release")
    if test_flavours:
        _build_flavour(verbose, "asan")
        _build_flavour(verbose, "debug")
    return lib


if __name__ == "__main__":
    print(build(verbose=True, test_flavours="--release-only" not in sys.argv))
