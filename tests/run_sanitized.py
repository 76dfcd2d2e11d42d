"""Run the CPU test suite (-m "not gpu") against builds of the oracle, the host
code of libbq and the plain-C example made with AddressSanitizer and
UndefinedBehaviorSanitizer (clang, the ROCm toolchain's runtime preloaded).
Any report aborts the test process, so a green run means no report.

    python tests/run_sanitized.py [extra pytest arguments]

CPU only: the device code of the sanitize build of libbq is the ordinary one,
and nothing here touches a GPU.
"""
from __future__ import annotations

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main() -> int:
    from paper_2110_02861_amd import build as hip_build
    import oracle
    from tests.c import build_example

    hip_build.build(sanitize=True)
    oracle.build(sanitize=True)
    build_example.build(sanitize=True)
    env = dict(os.environ, **hip_build.sanitize_env())
    # --capture=sys: reports written by the sanitizer runtime reach the terminal
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "--capture=sys", "-m", "not gpu",
           os.path.join(ROOT, "tests"), *sys.argv[1:]]
    return subprocess.run(cmd, env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    sys.exit(main())
