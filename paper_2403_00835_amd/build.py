"""Build libcllm.so (HIP, gfx950) in-tree with hipcc, plus the seeded-input generator."""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libcllm.so")
KERNEL_BENCH = os.path.join(HERE, "kernel_bench")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-fp32 VALU instructions are kept out of generated code: some of their forms have been seen
# to give wrong results without an error, and the compiler would otherwise emit them from plain
# float code.
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I" + INCLUDE]
SOURCES = ["gemm.hip", "kernels.hip", "loss.hip", "capi.cpp"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops' is not a recognized" not in l]
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))


def build(verbose=False):
    """Compile every HIP source for gfx950 and link libcllm.so (always recompiles)."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        _run([HIPCC, *HIP_FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    # standalone GEMM driver (per-kernel timing, hardware byte counters): links the GEMM object
    kb_obj = os.path.join(objdir, "kernel_bench.hip.o")
    _run([HIPCC, *HIP_FLAGS, "-x", "hip", "-c", os.path.join(CSRC, "kernel_bench.hip"), "-o", kb_obj], verbose)
    _run([HIPCC, "--offload-arch=" + ARCH, kb_obj, objs[SOURCES.index("gemm.hip")], "-o", KERNEL_BENCH + ".tmp"],
         verbose)
    os.replace(KERNEL_BENCH + ".tmp", KERNEL_BENCH)
    from . import workload
    workload.build(verbose)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
