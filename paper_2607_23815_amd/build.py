"""Build libpkv.so (the HIP kernels for gfx950 plus the C ABI) in-tree with hipcc.

    python -m paper_2607_23815_amd.build

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
ARCH = "gfx950"

SOURCES = ["pool.cpp", "sched.cpp", "api.cpp", "kv_copy.hip", "block_copy.hip", "decode.hip",
           "prefill.hip", "mixed.hip", "validate.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libpkv.so)")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
           "-fvisibility=hidden", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-mllvm", "-amdgpu-sched-strategy=max-ilp",
           "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include"),
           "-o", tmp] + [os.path.join(CSRC, s) for s in SOURCES]
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
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
