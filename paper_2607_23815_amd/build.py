"""Build libpkv.so (the HIP kernels for gfx950 plus the C ABI) in-tree with hipcc.

    python -m paper_2607_23815_amd.build
    python -m paper_2607_23815_amd.build --sanitize   # libpkv_asan.so, see below

--sanitize builds libpkv_asan.so with AddressSanitizer and UndefinedBehaviorSanitizer on the
host code only (the allocator, the scheduler, the C ABI's validation; every -fsanitize= goes
after -Xarch_host, so no device code is instrumented). It is for the CPU test tier: the
library is loaded through PKV_LIBRARY with the sanitizer runtime preloaded, e.g.

    LD_PRELOAD=$(python -m paper_2607_23815_amd.build --asan-runtime) \
    ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
    PKV_LIBRARY=paper_2607_23815_amd/libpkv_asan.so python -m pytest tests -m "not gpu"

(leak detection is off because the Python interpreter itself does not free everything at
exit).

Packed fp32 instructions are disabled for all device code (-packed-fp32-ops): the kernels use
plain fp32 arithmetic only. The machine scheduler runs its instruction-level-parallelism
strategy (-amdgpu-sched-strategy=max-ilp): the prefill's matrix-core/softmax block gains about
1% from it, the HBM-bound kernels are unchanged, and every kernel's output is bit-identical."""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpkv.so")
ASAN_LIB = os.path.join(PKG, "libpkv_asan.so")
SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-sanitize-recover=undefined",
                  "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
ARCH = "gfx950"

SOURCES = ["pool.cpp", "sched.cpp", "api.cpp", "kv_copy.hip", "block_copy.hip", "decode.hip",
           "prefill.hip", "mixed.hip", "validate.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libpkv.so)")


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (to preload into Python)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "lib", "llvm", "bin",
                         "clang")
    if not os.path.exists(clang):
        clang = shutil.which("clang") or "/opt/rocm/llvm/bin/clang"
    res = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True)
    return res.stdout.strip()


def build(verbose: bool = False, sanitize: bool = False) -> str:
    out = ASAN_LIB if sanitize else LIB
    tmp = out + ".tmp"
    cmd = [hipcc(), "-O1" if sanitize else "-O3", "-std=c++17", f"--offload-arch={ARCH}",
           "-fPIC", "-shared",
           "-fvisibility=hidden", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-mllvm", "-amdgpu-sched-strategy=max-ilp",
           "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include"),
           "-o", tmp] + (SANITIZE_FLAGS if sanitize else []) + \
        [os.path.join(CSRC, s) for s in SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libpkv.so")
    noise = [ln for ln in (res.stdout + res.stderr).splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "warning: feature" not in ln]
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    if "--asan-runtime" in sys.argv:
        print(asan_runtime())
    else:
        print(build(verbose=True, sanitize="--sanitize" in sys.argv))
