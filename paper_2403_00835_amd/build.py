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


# Host-code sanitizers (address + undefined behaviour) for the CPU test suite: every HIP source
# with its host half instrumented (the device code is built as usual), the seeded-input generator
# and the oracle, all against clang's shared sanitizer runtime. The CPU suite then runs in a child
# process that preloads that runtime and selects these libraries (CLLM_HOST_SANITIZE=1).
LLVM = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(HIPCC))), "llvm")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libasan"]


def sanitizer_runtime():
    import glob
    found = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
    if not found:
        raise RuntimeError("clang's shared address-sanitizer runtime was not found under " + LLVM)
    return found[-1]


def build_host_sanitized(verbose=False):
    """libcllm.hostsan.so, libcllm_workload.hostsan.so and liboracle.hostsan.so."""
    objdir = os.path.join(HERE, "_build", "hostsan")
    os.makedirs(objdir, exist_ok=True)
    flags = [f for f in HIP_FLAGS if f != "-O3"] + ["-O1", "-g"]
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        _run([HIPCC, *flags, *HOST_SAN, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    out = os.path.join(HERE, "libcllm.hostsan.so")
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *HOST_SAN, *objs, "-o", out + ".tmp"], verbose)
    os.replace(out + ".tmp", out)
    clang = os.path.join(LLVM, "bin", "clang")
    from . import workload
    workload.build_host_sanitized(clang, verbose)
    sys.path.insert(0, os.path.dirname(HERE))
    import oracle
    oracle.build_host_sanitized(clang, verbose)


def run_cpu_tests_sanitized(extra=()):
    """The CPU test suite (-m "not gpu") in a child process under the sanitizer runtime."""
    env = dict(os.environ)
    env["CLLM_HOST_SANITIZE"] = "1"
    env["LD_PRELOAD"] = sanitizer_runtime()
    env["LD_LIBRARY_PATH"] = os.path.join(LLVM, "lib") + (":" + env["LD_LIBRARY_PATH"] if env.get("LD_LIBRARY_PATH") else "")
    # leaks: the interpreter and its extension modules keep allocations to the end by design
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", os.path.join(os.path.dirname(HERE), "tests"), "-q", "-x", "-m", "not gpu",
           "-p", "no:cacheprovider", *extra]
    print(" ".join(cmd), flush=True)
    return subprocess.run(cmd, env=env).returncode


if __name__ == "__main__":
    if "--host-sanitize" in sys.argv:
        build_host_sanitized(verbose="-v" in sys.argv)
        sys.exit(run_cpu_tests_sanitized())
    build(verbose="-v" in sys.argv)
