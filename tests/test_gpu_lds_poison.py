"""The LDS rings of the attention and GEMM kernels under poison: the parity cases that run those
kernels (attention over context and in-block keys, the fragment-ordered and LDS-pipeline GEMMs,
the two-plane LM head, the single-plane top-2 ranking of the candidates head) run again, in one
child process, against libdpara_debug.so, the same library built with DPARA_DEBUG_LDS_POISON: each
kernel fills its ring with NaN before its first DMA, so a fragment read of any LDS byte that no
DMA wrote (a wrong slot, offset or wait) turns the outputs into NaN and the oracle comparisons fail."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEBUG_LIB = os.path.join(ROOT, "paper_2609_27396_amd", "libdpara_debug.so")


def test_parity_with_poisoned_lds_rings():
    assert os.path.exists(DEBUG_LIB), "libdpara_debug.so is missing: build with paper_2609_27396_amd.build"
    env = dict(os.environ, DPARA_LIB_PATH=DEBUG_LIB)
    probe = "from paper_2609_27396_amd import dpara as D; D.lib(); print(open('/proc/self/maps').read())"
    m = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert m.returncode == 0 and "libdpara_debug.so" in m.stdout and "/libdpara.so" not in m.stdout
    cmd = [sys.executable, "-u", "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "gpu",
           "--timeout", "300", "--timeout-method", "thread",
           os.path.join(ROOT, "tests", "test_gpu_parity.py"), "-k", "small_parity or one_layer or candidates"]
    print("child: poisoned-LDS parity cases", flush=True)
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    print(out[-1500:], flush=True)
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out and " failed" not in out
