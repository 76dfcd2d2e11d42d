"""The C ABI from plain C (tests/c/bq_c_example.c, built by
__graft_entry__.build()): host-only calls and argument errors here, and a
quantize round trip and 8-bit Adam steps (call and plan) on the GPU, checked
by the program itself against properties that hold at any size."""
import os
import subprocess

import pytest

from tests.gpu_helpers import needs_gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c",
                   "bq_c_example_san" if os.environ.get("BQ_SANITIZE") == "1" else "bq_c_example")


def _run(*args):
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built: run __graft_entry__.build() first")
    return subprocess.run([EXE, *args], capture_output=True, text=True, timeout=120)


def test_c_example_host_calls():
    r = _run()
    assert r.returncode == 0, r.stdout + r.stderr
    assert "bq_c_example ok" in r.stdout


@pytest.mark.gpu
@needs_gpu
def test_c_example_on_gpu():
    r = _run("gpu")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "bq_c_example ok" in r.stdout
