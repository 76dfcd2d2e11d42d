"""Host logic of bench.py: the algorithmic byte model and the one-GPU guard."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import bench
from paper_2110_02861_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_byte_model_of_the_lists():
    # 1.5B list, Adam, fp16 grads, B = 2048: 14 B per param + 16 B per block
    c5 = [s.numel for s in workloads.lm_1p5b_specs()]
    assert sum(c5) == 1_557_611_200
    assert bench.step_bytes(c5, 2048, 2, 2) == 21_818_727_840
    # ResNet-50 list, Momentum, fp32 grads: 4 + 4 + 4 + 2 B per param + 8 B per block
    c3 = [s.numel for s in workloads.resnet50_specs()]
    nb = sum((k + 2047) // 2048 for k in c3)
    assert nb == 12_560
    assert bench.step_bytes(c3, 2048, 4, 1) == 14 * sum(c3) + 8 * nb


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_recorded_counter_traffic_matches_the_byte_model():
    """The FETCH / WRITE counters recorded for each dominant kernel read within
    2 % of its algorithmic bytes (every byte moved once)."""
    c5 = [s.numel for s in workloads.lm_1p5b_specs()]
    c4 = [s.numel for s in workloads.SPECS["c4"]()]
    c3 = [s.numel for s in workloads.SPECS["c3"]()]
    quant = bench.QUANT_N * 5 + bench.QUANT_N // 2048 * 4
    algorithmic = {
        ("lm1p5b-adam", 2048, "plan"): bench.step_bytes(c5, 2048, 2, 2),
        ("lm1p5b-adam", 2048, "static"): bench.step_bytes(c5, 2048, 2, 2),
        ("lm1p5b-adam", 2048, "call"): bench.step_bytes(c5, 2048, 2, 2),
        ("gpt2m-adamw", 2048, "plan"): bench.step_bytes(c4, 2048, 2, 2),
        ("resnet50-momentum", 2048, "prepared"): bench.step_bytes(c3, 2048, 4, 1),
        ("resnet50-momentum", 2048, "plan"): bench.step_bytes(c3, 2048, 4, 1),
        ("quantize", 2048, "plan"): quant,
        ("quantize", 2048, "call"): quant,
        ("dequantize", 2048, "call"): quant,
    }
    assert set(algorithmic) == set(bench.MEASURED_TRAFFIC)
    for key, m in bench.MEASURED_TRAFFIC.items():
        t = m["fetch_kib"] * 1024 * bench.FETCH_SCALE + m["write_kib"] * 1024 * bench.WRITE_SCALE
        assert 0.99 < t / algorithmic[key] < 1.02, key


def test_byte_model_of_the_norm_pass():
    c5 = [s.numel for s in workloads.lm_1p5b_specs()]
    n = sum(c5)
    nb = sum((k + 2047) // 2048 for k in c5)
    # LAMB: Adam's step plus a read of w, g, both codes and both absmax
    assert bench.workload_bytes("lm1p5b-lamb", c5, 2048, 2) == 22 * n + 24 * nb
    # LARS: a one-state step (4+4+2+1+1 B, 8 B per block) plus a read of w and g
    assert bench.workload_bytes("lm1p5b-lars", c5, 2048, 2) == 18 * n + 8 * nb
    assert bench.workload_bytes("lm1p5b-adagrad", c5, 2048, 2) == 12 * n + 8 * nb
    assert bench.workload_bytes("lm1p5b-adam", c5, 2048, 2) == bench.step_bytes(c5, 2048, 2, 2)


def test_byte_model_of_the_paper_setup():
    """One tensor of 10^9 params with fp32 grads: Adam 16 B/param (the paper's
    setup), LAMB's norm pass reads w, the fp32 grad and both codes again."""
    p = [s.numel for s in workloads.paper_1b_specs()]
    n = 10 ** 9
    nb = (n + 2047) // 2048
    assert p == [n]
    assert bench.workload_bytes("paper1b-adam", p, 2048, 4) == 16 * n + 16 * nb
    assert bench.workload_bytes("paper1b-momentum", p, 2048, 4) == 14 * n + 8 * nb
    assert bench.workload_bytes("paper1b-lamb", p, 2048, 4) == (16 + 10) * n + 24 * nb
    assert bench.workload_bytes("paper1b-lars", p, 2048, 4) == (14 + 8) * n + 8 * nb


def test_cpu_model_is_read_from_proc_cpuinfo():
    m = bench.cpu_model()
    if os.path.exists("/proc/cpuinfo"):
        assert isinstance(m, str) and m


def test_stream_library_describes_its_variants_and_refuses_bad_arguments():
    """libbq_stream.so (the benchmark's stream ceilings and the access-shape
    study): variant descriptions and argument checks, which return before any
    HIP call."""
    import ctypes
    from paper_2110_02861_amd import build as pkg_build
    if not os.path.exists(pkg_build.STREAM_LIB):
        pytest.skip("libbq_stream.so is not built")
    L = ctypes.CDLL(pkg_build.STREAM_LIB)
    P = ctypes.c_void_p
    L.bq_stream_study_info.restype = ctypes.c_char_p
    L.bq_stream_study_info.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    L.bq_stream_study.argtypes = [ctypes.c_int, ctypes.POINTER(P), ctypes.POINTER(P),
                                  ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, P, ctypes.c_int,
                                  P]
    L.bq_stream_ceiling.argtypes = [ctypes.c_int] + [P] * 6 + [ctypes.c_int64, ctypes.c_int32,
                                                               ctypes.c_uint32, P, P]
    assert L.bq_stream_variants() == 9
    nv = L.bq_stream_study_variants()
    assert nv >= 28
    names = set()
    for v in range(nv):
        info = (ctypes.c_int * 3)()
        name = L.bq_stream_study_info(v, info).decode()
        assert name and name not in names
        names.add(name)
        assert info[0] in (256, 512, 1024) and info[1] in (1, 2, 4) and info[2] in (0, 1, 2)
        assert info[0] * info[1] * 4 >= 2048
    assert L.bq_stream_study_info(nv, None) == b"" and L.bq_stream_study_info(-1, None) == b""
    fake = 1 << 20  # never dereferenced: every call below fails its argument checks
    good = (P * 6)(*[fake] * 6)
    n = 8192 * 4
    assert L.bq_stream_study(-1, good, good, n, 2048, 0, P(fake), 0, None) == -1
    assert L.bq_stream_study(nv, good, good, n, 2048, 0, P(fake), 0, None) == -1
    assert L.bq_stream_study(0, good, good, n + 4096, 2048, 0, P(fake), 0, None) == -1
    assert L.bq_stream_study(0, good, good, n, 3000, 0, P(fake), 0, None) == -1
    assert L.bq_stream_study(0, good, good, n, 2048, 0, P(fake + 4), 0, None) == -1
    assert L.bq_stream_study(0, good, good, n, 2048, 0, P(fake), 5, None) == -1
    assert L.bq_stream_study(0, good, good, n, 2048, 0, P(fake), 1, None) == -1
    bad = (P * 6)(*([fake] * 5 + [fake + 8]))
    assert L.bq_stream_study(0, bad, good, n, 2048, 0, P(fake), 0, None) == -1
    nul = (P * 6)(*([fake] * 5 + [None]))
    assert L.bq_stream_study(0, good, nul, n, 2048, 0, P(fake), 0, None) == -1
    assert L.bq_stream_ceiling(9, *[P(fake)] * 6, n, 2048, 0, P(fake), None) == -1
    assert L.bq_stream_ceiling(0, *[P(fake)] * 6, n + 100, 2048, 0, P(fake), None) == -1
