"""Host AddressSanitizer and UndefinedBehaviorSanitizer runs (CPU only).

The oracle (gcc) and the host code of the C-ABI library (hipcc, host side
only: argument checks, workspace layout, handles) are built with
-fsanitize=address,undefined and exercised in a child process that preloads
the matching sanitizer runtime.  Any report aborts the child, which fails the
test.  Device code is not built here: GPU sanitizers are not available.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OPTS = "detect_leaks=0:abort_on_error=1:halt_on_error=1"

ORACLE_SCRIPT = r"""
import numpy as np, oracle, ttgen
c = ttgen.tiny(5, 2, (3, 4, 5), (2, 3, 2), 3, B=7, max_len=5, N=55)
c["idx"] = c["idx"].copy(); c["idx"][::4] = 57; c["idx"][1::9] = -1
V, inv = oracle.forward(c)
Vs, _ = oracle.forward(c, bags=np.array([3, 0, 13]))
assert np.array_equal(Vs, V[[3, 0, 13]]) and inv > 0
g = oracle.backward(c)
w = [np.ones(2 * k, np.uint8) for k in c["n"]]
gw = oracle.backward(c, want=w)
assert all(np.array_equal(a, b) for a, b in zip(g[:3], gw[:3]))
oracle.grouping(c)
oracle.digits(np.arange(60), c["n"])
oracle.sgd(c["G1"], g[0], 0.1)
oracle.row(c, 1, 7)
cn = ttgen.tiny_n(6, 2, (3, 2, 4, 2), (2, 1, 2, 2), 3, 9, max_len=5)
oracle.forward_n(cn)
oracle.backward_n(cn, want=[np.ones(2 * k, np.uint8) for k in cn["n"]])
print("oracle ok")
"""

LIB_SCRIPT = r"""
import ctypes as C, sys
sys.argv = ["abi"]
import pytest
sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", "tests/test_abi.py"]))
"""


def _run(script, env):
    r = subprocess.run([sys.executable, "-c", script], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-6000:])
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-6000:]
    return r


def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_asan.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-o", lib, os.path.join(ROOT, "oracle", "tt_oracle.c")])
    rt = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS=OPTS, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               TT_ORACLE_LIB=lib, PYTHONPATH=ROOT)
    assert "oracle ok" in _run(ORACLE_SCRIPT, env).stdout


def test_library_host_code_under_asan_ubsan(tmp_path):
    rts = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rts:
        pytest.skip("no clang AddressSanitizer runtime in this ROCm")
    lib = str(tmp_path / "libttemb_asan.so")
    csrc = os.path.join(ROOT, "paper_2609_03459_amd", "csrc")
    srcs = [os.path.join(csrc, f) for f in ("tt_emb.hip", "group.hip", "fwd.hip", "bwd.hip", "bwd_r32.hip", "bwd_r64.hip",
                                            "cores.hip")]
    # each -fsanitize= applies to the host compilation only (-Xarch_host); the device
    # code is built as usual, since the host objects name its code object
    subprocess.check_call(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                           "-shared", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                           "-I" + os.path.join(ROOT, "include"), "-o", lib, *srcs],
                          stderr=subprocess.DEVNULL)
    env = dict(os.environ, LD_PRELOAD=rts[0], ASAN_OPTIONS=OPTS, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               TT_EMB_LIB=lib, PYTHONPATH=ROOT)
    r = _run(LIB_SCRIPT, env)
    assert " passed" in r.stdout, r.stdout[-2000:]
