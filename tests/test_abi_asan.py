"""The host side of the C ABI (argument validation, workspace planning, error reporting) under
AddressSanitizer: the host-ABI tests run again, in a child process, against libdpara_asan.so (the
same library with its host code instrumented; `python -m paper_2609_27396_amd.build` makes it)
with the sanitizer runtime preloaded.  Any heap, stack or global out-of-bounds access, or use
after free, in those paths fails the run.  No GPU is touched: every call is rejected on the host
before a launch."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_LIB = os.path.join(ROOT, "paper_2609_27396_amd", "libdpara_asan.so")


def _runtime():
    pats = ("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so",
            "/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    for p in pats:
        hits = sorted(glob.glob(p))
        if hits:
            return hits[-1]
    return None


def test_host_abi_under_address_sanitizer():
    rt = _runtime()
    if not os.path.exists(ASAN_LIB) or rt is None:
        pytest.skip("libdpara_asan.so or the sanitizer runtime is missing (build with paper_2609_27396_amd.build)")
    env = dict(os.environ, LD_PRELOAD=rt, DPARA_LIB_PATH=ASAN_LIB,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=86:halt_on_error=1")
    # the child maps the instrumented library and the sanitizer runtime
    probe = ("from paper_2609_27396_amd import dpara as D; D.lib(); "
             "print(open('/proc/self/maps').read())")
    m = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert m.returncode == 0, (m.stdout + m.stderr)[-2000:]
    assert "libdpara_asan.so" in m.stdout and "libclang_rt.asan" in m.stdout
    assert "/libdpara.so" not in m.stdout
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           os.path.join(ROOT, "tests", "test_abi_host.py")]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out  # the child ran the host tests
