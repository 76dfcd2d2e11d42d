"""GPU parity: standalone block-wise quantize / dequantize vs the oracle.

Codes and absmax must be bit-exact, and so must dequantized values (one fp32
multiply of the looked-up code by the block absmax, Section 2.2).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2110_02861_amd import bq, workloads
from tests.gpu_helpers import codebooks_on_device, dev, host, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]

BLOCKSIZES = [256, 512, 1024, 2048, 4096]


def run_pair(qmap_h, qmap_d, x, B):
    say(f"quantize n={x.size} B={B}")
    x_d = dev(x)
    c_d, a_d = bq.bq_quantize_blockwise(qmap_d, x_d, B)
    prep = bq.bq_prepare_codebook(qmap_d)
    c_p, a_p = bq.bq_quantize_blockwise_prepared(prep, x_d, B)
    torch.cuda.synchronize()
    c_ref, a_ref = oracle.quantize_blockwise(qmap_h, x, B)
    for c, a in ((c_d, a_d), (c_p, a_p)):
        np.testing.assert_array_equal(host(a).view(np.uint32), a_ref.view(np.uint32))
        np.testing.assert_array_equal(host(c), c_ref)
    say(f"dequantize n={x.size} B={B}")
    out = bq.bq_dequantize_blockwise(qmap_d, c_d, a_d, B)
    torch.cuda.synchronize()
    ref = oracle.dequantize_blockwise(qmap_h, c_ref, a_ref, B)
    np.testing.assert_array_equal(host(out).view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("B", BLOCKSIZES)
def test_ragged_multi_tile(B):
    qs, qu, qs_d, qu_d = codebooks_on_device()
    # several tiles of every kernel (2048 / 4096 / 8192 elements) and a
    # ragged tail ending in the first, second and last chunk of a tile
    for n in (7 * max(B, 2048) + 1234, 5 * 8192 + 2048 + 777, 3 * 8192 + 6144 + 3):
        x = workloads.student_t_host(n, seed=B + n)
        run_pair(qs, qs_d, x, B)
        run_pair(qu, qu_d, np.abs(x), B)


@pytest.mark.parametrize("n", [1, 7, 255, 256, 257, 2047, 2048, 2049, 4095, 4097, 8191, 8192,
                               8193, 10000, 16383, 16385])
def test_edge_lengths(n):
    qs, _, qs_d, _ = codebooks_on_device()
    x = workloads.student_t_host(n, seed=n)
    for B in (256, 2048, 4096):
        run_pair(qs, qs_d, x, B)


def test_ties_and_neighbours_exact():
    """Values whose quotient by the absmax lands exactly on a midpoint of two
    codes, and one ulp either side: ties go to the lower code (Eq. 3)."""
    qs, qu, qs_d, qu_d = codebooks_on_device()
    for q, q_d in ((qs, qs_d), (qu, qu_d)):
        ys = []
        for j in range(255):
            m = np.float32((float(q[j]) + float(q[j + 1])) / 2.0)
            ys += [np.nextafter(m, np.float32(-np.inf), dtype=np.float32), m,
                   np.nextafter(m, np.float32(np.inf), dtype=np.float32)]
        ys = np.array(ys, np.float32)
        B = 2048
        # block absmax 1 (and a scaled copy): one element fixes the absmax
        for N in (np.float32(1.0), np.float32(0.375), np.float32(3.0e-3)):
            blocks = []
            for s in range(0, ys.size, B - 1):
                chunk = (ys[s:s + B - 1] * N).astype(np.float32)
                blk = np.zeros(B, np.float32)
                blk[:chunk.size] = chunk
                blk[-1] = N
                blocks.append(blk)
            run_pair(q, q_d, np.concatenate(blocks), B)


def test_zero_blocks_and_signed_zero():
    qs, qu, qs_d, qu_d = codebooks_on_device()
    x = np.zeros(3 * 2048 + 5, np.float32)
    x[2048:4096] = workloads.student_t_host(2048, seed=3)
    x[100] = -0.0
    for q, q_d in ((qs, qs_d), (qu, qu_d)):
        run_pair(q, q_d, x, 2048)


@pytest.mark.parametrize("scale", [2.0 ** -120, 2.0 ** -70, 2.0 ** -30, 1.0, 2.0 ** 40, 2.0 ** 90])
def test_extreme_block_scales(scale):
    """Blocks whose absmax needs the power-of-two rescaling of the divisor."""
    qs, _, qs_d, _ = codebooks_on_device()
    x = (workloads.student_t_host(3 * 2048, seed=5).astype(np.float64) * scale).astype(np.float32)
    run_pair(qs, qs_d, x, 2048)


def test_round_trip_every_code():
    qs, qu, qs_d, qu_d = codebooks_on_device()
    B = 256
    codes = np.tile(np.arange(256, dtype=np.uint8), 8)
    absmax = np.array([1.0, 0.37, 3e-5, 12345.678, 2.0 ** -70, 2.0 ** 70, 7.0, 1e-3], np.float32)
    for q_d in (qs_d, qu_d):
        say("round trip")
        x = bq.bq_dequantize_blockwise(q_d, dev(codes), dev(absmax), B)
        c2, a2 = bq.bq_quantize_blockwise(q_d, x, B)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(c2), codes)
        np.testing.assert_array_equal(host(a2), absmax)


@pytest.mark.parametrize("B", [2048, 4096])
def test_full_size_student_t(B):
    """67,108,864 Student-t(3) values scaled 1e-2, every code and absmax compared."""
    qs, _, qs_d, _ = codebooks_on_device()
    n = 67_108_864
    x = workloads.student_t_host(n, seed=0)
    say(f"full-size quantize n={n} B={B}")
    x_d = dev(x)
    c_d, a_d = bq.bq_quantize_blockwise(qs_d, x_d, B)
    out_d = bq.bq_dequantize_blockwise(qs_d, c_d, a_d, B)
    c_p, a_p = bq.bq_quantize_blockwise_prepared(bq.bq_prepare_codebook(qs_d), x_d, B)
    torch.cuda.synchronize()
    c_ref, a_ref = oracle.quantize_blockwise(qs, x, B)
    for c, a in ((c_d, a_d), (c_p, a_p)):
        np.testing.assert_array_equal(host(a).view(np.uint32), a_ref.view(np.uint32))
        np.testing.assert_array_equal(host(c), c_ref)
    ref = oracle.dequantize_blockwise(qs, c_ref, a_ref, B)
    np.testing.assert_array_equal(host(out_d).view(np.uint32), ref.view(np.uint32))


def test_non_default_stream_ordering():
    qs, _, qs_d, _ = codebooks_on_device()
    x = workloads.student_t_host(5 * 2048 + 3, seed=9)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        x_d = dev(x)
        say("quantize on a side stream")
        c_d, a_d = bq.bq_quantize_blockwise(qs_d, x_d, 2048, stream=s)
        out = bq.bq_dequantize_blockwise(qs_d, c_d, a_d, 2048, stream=s)
    s.synchronize()
    c_ref, a_ref = oracle.quantize_blockwise(qs, x, 2048)
    np.testing.assert_array_equal(host(c_d), c_ref)
    np.testing.assert_array_equal(host(out), oracle.dequantize_blockwise(qs, c_ref, a_ref, 2048))


# --- other codebooks (App. F): the same kernels with any sorted 256-entry map ---

def _other_maps():
    """name -> (host map from the oracle, signed input?)."""
    normal = workloads.host_rng(0, "c2", 1, 0).standard_normal(200_001).astype(np.float32)
    heavy = np.abs(workloads.student_t_host(200_001, seed=11))
    return {
        "inverse_signed": (oracle.codebook(2), True),
        "inverse_unsigned": (oracle.codebook(3), False),
        "linear_signed": (oracle.codebook(4), True),
        "linear_unsigned": (oracle.codebook(5), False),
        "quantile_normal": (oracle.quantile_codebook(normal), True),
        "quantile_abs_t": (oracle.quantile_codebook(heavy), False),
    }


OTHER = ["inverse_signed", "inverse_unsigned", "linear_signed", "linear_unsigned",
         "quantile_normal", "quantile_abs_t"]


@pytest.mark.parametrize("B", [256, 2048, 4096])
@pytest.mark.parametrize("name", OTHER)
def test_other_codebooks_ragged(name, B):
    q, signed = _other_maps()[name]
    n = 3 * max(B, 2048) + 1234
    x = workloads.student_t_host(n, seed=B + 1)
    run_pair(q, dev(q), x if signed else np.abs(x), B)


@pytest.mark.parametrize("name", OTHER)
def test_other_codebooks_ties_and_round_trip(name):
    """Midpoints of adjacent codes and one ulp either side (ties to the lower
    code), and dequantize -> quantize returns every code."""
    q, _ = _other_maps()[name]
    q_d = dev(q)
    ys = []
    for j in range(255):
        m = np.float32((float(q[j]) + float(q[j + 1])) / 2.0)
        ys += [np.nextafter(m, np.float32(-np.inf), dtype=np.float32), m,
               np.nextafter(m, np.float32(np.inf), dtype=np.float32)]
    ys = np.array(ys, np.float32)
    B = 2048
    amax = np.float32(np.max(np.abs(q)))
    blocks = []
    for s0 in range(0, ys.size, B - 1):
        chunk = ys[s0:s0 + B - 1]
        blk = np.zeros(B, np.float32)
        blk[:chunk.size] = chunk
        blk[-1] = amax           # absmax = max |q|: the quotients stay as built
        blocks.append(blk)
    run_pair(q, q_d, np.concatenate(blocks), B)
    codes = np.tile(np.arange(256, dtype=np.uint8), 4)
    absmax = np.array([1.0, 0.37, 3e-5, 12345.678], np.float32)
    say(f"round trip {name}")
    x = bq.bq_dequantize_blockwise(q_d, dev(codes), dev(absmax), 256)
    c2, _ = bq.bq_quantize_blockwise(q_d, x, 256)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(c2), codes)


def test_exact_thresholds_for_uneven_maps():
    """Maps with adjacent codes of very different magnitude (where a double
    midpoint is inexact): decisions at and around those midpoints stay exact."""
    q = oracle.codebook(4).copy()
    q2 = q.copy()
    q2[127] = np.float32(-1e-43)
    q3 = q2.copy()
    q3[128] = np.float32(0.5)
    q3[129:] = np.linspace(0.5, 1.0, 128, dtype=np.float32)[1:]
    for qm in (q, q2, q3):
        assert np.all(np.diff(qm) > 0)
        ys = [np.float32(0.0), np.float32(2.0 ** -149), np.float32(-2.0 ** -149)]
        for j in range(255):
            m = np.float32((float(qm[j]) + float(qm[j + 1])) / 2.0)
            for k in range(-2, 3):
                y = m
                for _ in range(abs(k)):
                    y = np.nextafter(y, np.float32(np.sign(k)), dtype=np.float32)
                ys.append(y)
        x = np.array(ys, np.float32)
        B = 2048
        blocks = []
        for s0 in range(0, x.size, B - 1):
            blk = np.zeros(B, np.float32)
            chunk = x[s0:s0 + B - 1]
            blk[:chunk.size] = chunk
            blk[-1] = 1.0
            blocks.append(blk)
        run_pair(qm, dev(qm), np.concatenate(blocks), B)


def test_dense_bucket_map():
    """150 codes one ulp apart inside one bucket (just above 0.5): the bucket
    table leaves up to 149 thresholds to compare, so the search loop runs far
    beyond the dynamic maps' single compare, in the per-workgroup tables of
    the raw-map call and in the prepared tables alike."""
    low = np.linspace(-1.0, 0.49, 105).astype(np.float32)
    dense = np.float32(0.5) + np.arange(150, dtype=np.float32) * np.float32(2.0 ** -24)
    q = np.concatenate([low, dense, [np.float32(1.0)]]).astype(np.float32)
    assert q.size == 256 and np.all(np.diff(q.astype(np.float64)) > 0)
    rng = np.random.default_rng(21)
    B = 2048
    nblk = 6
    x = np.empty(nblk * B, np.float32)
    for b in range(nblk):
        blk = np.float32(0.5) + rng.integers(-5, 160, B).astype(np.float32) * np.float32(2.0 ** -24)
        spread = rng.random(B) < 0.2
        blk[spread] = rng.uniform(-1, 1, int(spread.sum())).astype(np.float32)
        blk[0] = 1.0
        x[b * B:(b + 1) * B] = blk * np.float32(2.0 ** (b - 3))
    run_pair(q, dev(q), x, B)


@pytest.mark.parametrize("B", [256, 2048])
def test_block_isolation_on_gpu(B):
    """Changing one block's values changes only that block's codes and absmax
    (each block is normalized by its own absmax, Section 3.1)."""
    qs, _, qs_d, _ = codebooks_on_device()
    n = 9 * 8192 + 333
    x = workloads.student_t_host(n, seed=77)
    prep = bq.bq_prepare_codebook(qs_d)
    say(f"block isolation B={B}")
    c0, a0 = bq.bq_quantize_blockwise_prepared(prep, dev(x), B)
    r0, s0 = bq.bq_quantize_blockwise(qs_d, dev(x), B)
    nb = (n + B - 1) // B
    for b in (0, nb // 2, nb - 1):
        y = x.copy()
        s = slice(b * B, min((b + 1) * B, n))
        y[s] = y[s] * np.float32(-3.0) + np.float32(1e-3)
        c1, a1 = bq.bq_quantize_blockwise_prepared(prep, dev(y), B)
        r1, s1 = bq.bq_quantize_blockwise(qs_d, dev(y), B)
        torch.cuda.synchronize()
        for (ca, aa), (cb, ab) in (((c0, a0), (c1, a1)), ((r0, s0), (r1, s1))):
            ca, cb, aa, ab = host(ca), host(cb), host(aa), host(ab)
            keep = np.ones(n, bool)
            keep[s] = False
            np.testing.assert_array_equal(ca[keep], cb[keep])
            others = np.arange(nb) != b
            np.testing.assert_array_equal(aa[others], ab[others])
            assert aa[b] != ab[b]
            ref_c, ref_a = oracle.quantize_blockwise(qs, np.ascontiguousarray(y[s]), B)
            np.testing.assert_array_equal(cb[s], ref_c)
            assert ab[b] == ref_a[0]
