"""Compile tests/c/bq_c_example.c (a C99 user of include/bq.h) against the
in-tree libbq.so; called by __graft_entry__.build()."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "bq_c_example.c")
EXE = os.path.join(HERE, "bq_c_example")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


SAN_EXE = EXE + "_san"


def build(sanitize: bool = False) -> str:
    """The example against libbq.so; with sanitize, built by clang with
    AddressSanitizer and UndefinedBehaviorSanitizer against the sanitize build
    of the library (_build/san/libbq.so), as bq_c_example_san."""
    if sanitize:
        lib_dir = os.path.join(ROOT, "paper_2110_02861_amd", "_build", "san")
        rpath = "$ORIGIN/../../paper_2110_02861_amd/_build/san"
        out = SAN_EXE
        # the shared runtime, the one the sanitized library's callers preload
        cc = [os.path.join(ROCM, "llvm", "bin", "clang"), "-fsanitize=address,undefined",
              "-shared-libsan", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]
    else:
        lib_dir = os.path.join(ROOT, "paper_2110_02861_amd")
        rpath = "$ORIGIN/../../paper_2110_02861_amd"
        out = EXE
        cc = ["gcc"]
    cmd = [*cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           SRC, "-o", out + ".tmp",
           "-L", lib_dir, "-lbq",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath," + rpath, "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    import sys
    print(build(sanitize="--sanitize" in sys.argv))
