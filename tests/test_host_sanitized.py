"""The host planner and C ABI under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The host sources (psattn_host.cpp, psattn_kvcache.cpp, psattn_sched.cpp and the host side of
psattn_noalloc.hip)
are compiled with g++ against a host-only stand-in for the HIP runtime header (tests/sanitize/),
with -fsanitize=address,undefined and no recovery from undefined behaviour, and the host tests
(descriptor validation, random-forest planner coverage, packing and split plans, cross-call
plans, the KV cache manager, the scheduler) run against that build in a child process.  Any
out-of-bounds access, use after free or signed overflow in validation or planning fails here.
The build also turns on PSATTN_PLAN_CHECKS: every plan is checked so that each index the kernels
derive from it (row and slot lists, item ranges, partial rows and tiles) lies inside what it
addresses, or tree creation fails with PSATTN_E_INTERNAL.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_25683_amd", "csrc")


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(shutil.which("g++") is None or _runtime("libasan.so") is None, reason="needs g++ with libasan")
def test_host_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    lib = str(tmp_path / "libpsattn_host_sanitized.so")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fsanitize=address,undefined", "-DPSATTN_PLAN_CHECKS",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "tests", "sanitize"), "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "psattn_host.cpp"), os.path.join(CSRC, "psattn_kvcache.cpp"),
           os.path.join(CSRC, "psattn_sched.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
           "-x", "c++", os.path.join(CSRC, "psattn_noalloc.hip"), "-x", "none",
           "-o", lib]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    tests = [os.path.join(ROOT, "tests", f) for f in ("test_abi_host.py", "test_cross_call.py", "test_kv_cache.py",
                                                        "test_sched.py")]
    runner = ("import sys; sys.path.insert(0, %r); import paper_2608_25683_amd.psattn as P; P.LIB_PATH = %r; "
              "import pytest; sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider'] + %r))" % (ROOT, lib, tests))
    env = dict(os.environ, LD_PRELOAD=_runtime("libasan.so"), ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", runner], capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    log = r.stdout[-3000:] + r.stderr[-6000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, log
    assert r.returncode == 0, log
