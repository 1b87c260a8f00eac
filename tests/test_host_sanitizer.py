"""CPU tier: the library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The allocator, the prefix cache with pinning, eviction and copy-on-write, the scheduler in model
mode, the C ABI's argument checks and the launch plans are host C++; libpkv_asan.so is the same
library built with -fsanitize=address,undefined on the host code only (see
paper_2607_23815_amd/build.py --sanitize). This test reruns the CPU tests that drive that code
through the C ABI against the sanitized build, in a child process with the sanitizer runtime
preloaded; any report fails it. It is skipped when libpkv_asan.so has not been built."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_LIB = os.path.join(ROOT, "paper_2607_23815_amd", "libpkv_asan.so")
FILES = ["tests/test_abi.py", "tests/test_sched_abi.py"]


@pytest.mark.skipif(not os.path.exists(ASAN_LIB),
                    reason="libpkv_asan.so not built (python -m paper_2607_23815_amd.build "
                           "--sanitize)")
def test_host_code_under_sanitizers():
    from paper_2607_23815_amd import build as b
    runtime = b.asan_runtime()
    assert os.path.exists(runtime), runtime
    env = dict(os.environ)
    # the sanitizer runtime goes first; whatever the environment already preloads is kept
    env["LD_PRELOAD"] = ":".join(p for p in (runtime, os.environ.get("LD_PRELOAD", "")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["PKV_LIBRARY"] = ASAN_LIB
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:xdist", "-p", "no:cacheprovider"] + FILES,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail
