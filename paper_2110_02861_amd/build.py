"""Build libbq.so in-tree with hipcc for gfx950.

    python -m paper_2110_02861_amd.build              # build
    python -m paper_2110_02861_amd.build --asm        # also write gfx950 assembly
    python -m paper_2110_02861_amd.build --sanitize   # a CPU-checking build (below)

The sanitize build compiles the host code (argument checks, codebook builder,
descriptor packing, launch wrappers) with AddressSanitizer and
UndefinedBehaviorSanitizer into _build/san/libbq.so; the device code is
compiled as usual.  It is for the CPU test suite only: load it with
BQ_SANITIZE=1 and the clang ASan runtime preloaded (see SANITIZE_ENV).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libbq.so")
SOURCES = ["bq_api.cpp", "bq_codebook.cpp", "bq_oneshot.hip", "bq_state32.hip",
           "bq_quantiles.hip"]
# the benchmark's streaming-ceiling kernel, a library of its own
STREAM_LIB = os.path.join(PKG, "libbq_stream.so")
STREAM_SOURCES = ["bq_stream.hip"]
ARCH = "gfx950"

# -ffp-contract=off: the state arithmetic must not be fused into fma, so that it
# rounds exactly as its definition.  Packed fp32 instructions are disabled.
# Correctly rounded fp32 division stays on (the HIP default).
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.sep not in c or os.path.exists(c)):
            return c
    raise RuntimeError("hipcc not found")


OBJ_DIR = os.path.join(PKG, "_build", "obj")
SAN_DIR = os.path.join(PKG, "_build", "san")
SAN_LIB = os.path.join(SAN_DIR, "libbq.so")
# host-only sanitizers: each -fsanitize= right after -Xarch_host
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xarch_host", "-g"]


def asan_runtime() -> str:
    """The clang ASan runtime of the ROCm toolchain (it carries UBSan's too)."""
    import glob
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    found = sorted(glob.glob(os.path.join(rocm, "llvm", "lib", "clang", "*", "lib", "linux",
                                          "libclang_rt.asan-x86_64.so")))
    if not found:
        raise RuntimeError("clang ASan runtime not found under " + rocm)
    return found[-1]


def sanitize_env() -> dict:
    """Environment for running the CPU tests against the sanitize builds."""
    return {"BQ_SANITIZE": "1", "LD_PRELOAD": asan_runtime(),
            "ASAN_OPTIONS": "detect_leaks=0:detect_odr_violation=0:abort_on_error=1",
            "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}


def _link(out: str, sources, verbose: bool, sanitize: bool = False) -> str:
    """Compile every source to an object, all at once in parallel, then link."""
    obj_dir = os.path.join(SAN_DIR, "obj") if sanitize else OBJ_DIR
    os.makedirs(obj_dir, exist_ok=True)
    extra = SAN_FLAGS if sanitize else []
    objs, procs = [], []
    for name in sources:
        obj = os.path.join(obj_dir, os.path.splitext(name)[0] + ".o")
        cmd = [hipcc(), *FLAGS, *extra, "-c", "-o", obj, os.path.join(CSRC, name)]
        if verbose:
            print(" ".join(cmd))
        objs.append(obj)
        procs.append((cmd, subprocess.Popen(cmd)))
    failed = [cmd for cmd, proc in procs if proc.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Build libbq.so (the library) and libbq_stream.so (the benchmark's
    streaming-ceiling kernel); return the path of libbq.so.  With sanitize,
    build only the sanitize library (_build/san/libbq.so) and return its path."""
    if sanitize:
        return _link(SAN_LIB, SOURCES, verbose, sanitize=True)
    _link(STREAM_LIB, STREAM_SOURCES, verbose)
    return _link(LIB, SOURCES, verbose)


def build_asm(out_dir: str) -> None:
    """Write the device assembly of the kernels (for inspection only)."""
    os.makedirs(out_dir, exist_ok=True)
    for name in ("bq_oneshot.hip", "bq_state32.hip", "bq_quantiles.hip"):
        cmd = [hipcc(), *FLAGS, "--cuda-device-only", "-S", "-o",
               os.path.join(out_dir, name.replace(".hip", ".s")), os.path.join(CSRC, name)]
        subprocess.run(cmd, check=True)


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
    if "--asm" in sys.argv:
        build_asm(os.path.join(PKG, "_build", "asm"))
