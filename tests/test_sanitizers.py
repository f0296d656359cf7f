"""The CPU checks under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle and the library's host code are rebuilt with both sanitizers (clang,
one runtime for both), and the oracle pins and the host-side tests of the C ABI
run in a child process with that runtime preloaded: any out-of-bounds access,
use after free or undefined behaviour in them aborts the run.  A planted
overflow (an output buffer one row short handed to the oracle's forward) must be
reported, which shows the sanitizer is live."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("no clang with sanitizer runtimes")
    sys.path.insert(0, ROOT)
    from oracle import build as ob
    from paper_2205_04702_amd import build as pb
    d = str(tmp_path_factory.mktemp("asan"))
    rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True, check=True).stdout.strip()
    preload = rt + (":" + os.environ["LD_PRELOAD"] if os.environ.get("LD_PRELOAD") else "")
    env = dict(os.environ, LD_PRELOAD=preload,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               ORACLE_LIB=ob.build_sanitized(d), SCRATCHPIPE_LIB=pb.build_sanitized_host(d),
               PYTHONPATH=ROOT)
    return env


def test_cpu_checks_pass_under_the_sanitizers(sanitized):
    tests = ["tests/test_oracle_training.py", "tests/test_oracle_holdmask.py",
             "tests/test_capi_host.py", "tests/test_oracle_planner.py",
             "tests/test_oracle_policies.py", "tests/test_oracle_prefetch.py",
             "tests/test_workload.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", "-k", "not exhaustive", *tests], cwd=ROOT,
                       env=sanitized, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout


def test_a_planted_overflow_is_reported(sanitized):
    code = """
import ctypes as C, numpy as np
from oracle import oracle
L = oracle.lib()
T, B, D = 1, 2, 8
tab = np.zeros((10, D), np.float32)
ids = np.array([1, 2, 3], np.int32)
off = np.array([0, 1, 3], np.int32)
out = np.zeros((T * B - 1) * D, np.float32)  # one pooled row short
ptrs = (C.c_void_p * 1)(tab.ctypes.data)
L.orc_forward.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                          C.c_void_p]
L.orc_forward(T, B, D, ptrs, ids.ctypes.data, off.ctypes.data, out.ctypes.data)
print("not caught")
"""
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=sanitized,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0 and "not caught" not in r.stdout
    assert "heap-buffer-overflow" in r.stderr
