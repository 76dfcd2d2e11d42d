"""Pins of the oracle's nearest-code search and block-wise (de)quantization.

Eq. 3 defines the code as the argmin of |q_j - T_i / N| (found in the paper by
a binary search); Section 3.1 / Eq. 4 applies it per block of B elements with
N_b = max |T_b|; dequantization is q[code] * N_b (Section 2.2).  The checks
below use exact rational arithmetic (fractions.Fraction) and IEEE binary32
division from numpy, neither of which shares code with the oracle.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def maps():
    return {"signed": oracle.dynamic_codebook(0), "unsigned": oracle.dynamic_codebook(1)}


def exact_nearest(qmap: np.ndarray, y: np.float32) -> int:
    """argmin_j |q_j - y| in exact rationals, lowest index on ties."""
    return int(exact_nearest_many(qmap, np.array([y], np.float32))[0])


def exact_nearest_many(qmap: np.ndarray, ys: np.ndarray) -> np.ndarray:
    """Vectorised exact argmin: a float64 screen picks every code within a
    relative 1e-9 of the best distance, and exact rationals decide among them
    (lowest index on ties)."""
    q64 = qmap.astype(np.float64)
    out = np.empty(ys.size, np.int64)
    for s in range(0, ys.size, 4096):
        y = ys[s:s + 4096].astype(np.float64)
        d = np.abs(y[:, None] - q64[None, :])
        best = d.min(axis=1, keepdims=True)
        cand = d <= best * (1 + 1e-9) + 1e-300
        for i in range(y.size):
            idx = np.nonzero(cand[i])[0]
            if idx.size == 1:
                out[s + i] = idx[0]
                continue
            fy = Fraction(float(ys[s + i]))
            ds = [abs(Fraction(float(qmap[j])) - fy) for j in idx]
            out[s + i] = idx[min(range(len(ds)), key=lambda k: (ds[k], idx[k]))]
    return out


def ulp_neighbours(v: np.float32, k: int):
    out = [v]
    a = b = v
    for _ in range(k):
        a = np.nextafter(a, np.float32(-np.inf), dtype=np.float32)
        b = np.nextafter(b, np.float32(np.inf), dtype=np.float32)
        out += [a, b]
    return out


def midpoint_probes(qmap):
    """Every midpoint of adjacent codes (rounded to binary32) and 2 ulps around it."""
    probes = []
    for j in range(255):
        m = (float(qmap[j]) + float(qmap[j + 1])) / 2.0   # exact in double
        probes += ulp_neighbours(np.float32(m), 2)
    return probes


@pytest.mark.parametrize("name", ["signed", "unsigned"])
def test_brute_and_bsearch_equal_exact_argmin_on_midpoints(maps, name):
    q = maps[name]
    ties = 0
    for y in midpoint_probes(q):
        e = exact_nearest(q, y)
        assert oracle.nearest_brute(q, y) == e, (name, float(y))
        assert oracle.nearest_bsearch(q, y) == e, (name, float(y))
    # exact ties exist: a midpoint representable in binary32 goes to the lower index
    for j in range(255):
        m = (float(q[j]) + float(q[j + 1])) / 2.0
        if float(np.float32(m)) == m:
            ties += 1
            assert oracle.nearest_bsearch(q, np.float32(m)) == j
    assert ties > 0


@pytest.mark.parametrize("name", ["signed", "unsigned"])
def test_every_code_maps_to_itself(maps, name):
    q = maps[name]
    for j in range(256):
        assert oracle.nearest_brute(q, q[j]) == j
        assert oracle.nearest_bsearch(q, q[j]) == j


@pytest.mark.parametrize("name", ["signed", "unsigned"])
def test_random_values_exact_argmin(maps, name):
    q = maps[name]
    rng = np.random.default_rng(1)
    ys = np.concatenate([
        rng.uniform(-1, 1, 300),
        np.sign(rng.standard_normal(300)) * 10.0 ** rng.uniform(-9, 0, 300),
        np.array([0.0, -0.0, 1.0, -1.0, 1e-30, -1e-30, 5e-8, -5e-7]),
    ]).astype(np.float32)
    for y in ys:
        e = exact_nearest(q, y)
        assert oracle.nearest_brute(q, y) == e
        assert oracle.nearest_bsearch(q, y) == e


def test_nearest_exact_on_maps_spanning_the_binary32_range():
    """The exact midpoint decision holds for any finite map, not only the
    dynamic ones: strictly increasing maps whose magnitudes span 2^-149
    (subnormal) to 2^100, with symmetric pairs (a + b == 0) and neighbours
    many binades apart; probes at every binary32 midpoint +-2 ulps."""
    rng = np.random.default_rng(7)
    for trial in range(6):
        mags = 2.0 ** rng.uniform(-149, 100, 300)
        vals = np.concatenate([mags, -mags[:120], [0.0, 2.0 ** -149, -(2.0 ** -149)]])
        q = np.unique(vals.astype(np.float32))
        q = np.sort(rng.choice(q, 256, replace=False)).astype(np.float32)
        assert np.all(np.diff(q.astype(np.float64)) > 0)
        probes = midpoint_probes(q) + list(q) + [np.float32(0.0), np.float32(-0.0)]
        ys = np.array(probes, np.float32)
        exact = exact_nearest_many(q, ys)
        for y, e in zip(ys, exact):
            assert oracle.nearest_brute(q, y) == e, (trial, float(y))
            assert oracle.nearest_bsearch(q, y) == e, (trial, float(y))


@pytest.mark.parametrize("name", ["signed", "unsigned"])
def test_nearest_property(maps, name):
    q = maps[name].astype(np.float64)
    rng = np.random.default_rng(2)
    for y in rng.uniform(q[0], q[255], 2000).astype(np.float32):
        c = oracle.nearest_bsearch(maps[name], y)
        d = abs(float(y) - q[c])
        if c > 0:
            assert d <= abs(float(y) - q[c - 1])
        if c < 255:
            assert d <= abs(float(y) - q[c + 1])


def exact_quantize_blockwise(qmap, x, B):
    """Independent definition: N_b = max|x|, y = fl32(x / N_b), exact argmin."""
    n = x.size
    nb = (n + B - 1) // B
    codes = np.empty(n, np.uint8)
    absmax = np.empty(nb, np.float32)
    zero = exact_nearest(qmap, np.float32(0))
    for b in range(nb):
        blk = x[b * B:(b + 1) * B]
        N = np.float32(np.max(np.abs(blk)))
        absmax[b] = N
        if N == 0:
            codes[b * B:(b + 1) * B] = zero
            continue
        y = (blk / N).astype(np.float32)  # IEEE binary32 division
        codes[b * B:(b + 1) * B] = exact_nearest_many(qmap, y)
    return codes, absmax


@pytest.mark.parametrize("B,n", [(256, 1000), (512, 512), (256, 1), (1024, 700)])
def test_quantize_blockwise_matches_exact_definition(maps, B, n):
    rng = np.random.default_rng(B + n)
    x = (rng.standard_t(3, n) * 1e-2).astype(np.float32)
    x[::97] = 0.0
    for name in ("signed", "unsigned"):
        q = maps[name]
        xe = x if name == "signed" else np.abs(x)
        c_ref, a_ref = exact_quantize_blockwise(q, xe, B)
        for brute in (False, True):
            c, a = oracle.quantize_blockwise(q, xe, B, brute=brute)
            np.testing.assert_array_equal(a, a_ref)
            np.testing.assert_array_equal(c, c_ref)


def test_dequantize_is_lookup_times_absmax(maps):
    q = maps["signed"]
    rng = np.random.default_rng(3)
    n, B = 3000, 256
    codes = rng.integers(0, 256, n).astype(np.uint8)
    absmax = rng.uniform(0, 2, (n + B - 1) // B).astype(np.float32)
    out = oracle.dequantize_blockwise(q, codes, absmax, B)
    for i in rng.integers(0, n, 200):
        assert out[i] == np.float32(q[codes[i]] * absmax[i // B])


@pytest.mark.parametrize("N", [1.0, 0.37, 3.0e-5, 12345.678, 2.0 ** -70])
@pytest.mark.parametrize("name", ["signed", "unsigned"])
def test_round_trip_every_code(maps, name, N):
    """quantize(dequantize(c)) == c for all 256 codes in one block (absmax = N)."""
    q = maps[name]
    B = 256
    codes = np.arange(256, dtype=np.uint8)
    absmax = np.array([N], np.float32)
    x = oracle.dequantize_blockwise(q, codes, absmax, B)
    c2, a2 = oracle.quantize_blockwise(q, x, B)
    assert a2[0] == np.float32(N)
    np.testing.assert_array_equal(c2, codes)


def test_absmax_element_reconstructed_exactly(maps):
    """Section 3.1: the block's absmax element is quantized without error."""
    q = maps["signed"]
    rng = np.random.default_rng(4)
    B = 512
    x = rng.standard_normal(4 * B).astype(np.float32)
    c, a = oracle.quantize_blockwise(q, x, B)
    xd = oracle.dequantize_blockwise(q, c, a, B)
    for b in range(4):
        blk = x[b * B:(b + 1) * B]
        i = int(np.argmax(np.abs(blk)))
        assert xd[b * B + i] == blk[i]


def test_block_isolation(maps):
    """Section 3.1: blocks are normalized independently; an outlier stays in its block."""
    q = maps["signed"]
    rng = np.random.default_rng(5)
    B, nb = 256, 6
    x = rng.standard_normal(B * nb).astype(np.float32)
    c0, a0 = oracle.quantize_blockwise(q, x, B)
    x2 = x.copy()
    x2[3 * B + 17] = 1e4
    c1, a1 = oracle.quantize_blockwise(q, x2, B)
    changed = np.nonzero(a0 != a1)[0]
    assert changed.tolist() == [3]
    diff_blocks = np.unique(np.nonzero(c0 != c1)[0] // B)
    assert diff_blocks.tolist() == [3]


def test_zero_block(maps):
    for name, zero_code in (("signed", 127), ("unsigned", 0)):
        q = maps[name]
        x = np.zeros(700, np.float32)
        x[600] = -0.0
        c, a = oracle.quantize_blockwise(q, x, 256)
        assert np.all(c == zero_code) and np.all(a == 0)
        assert np.all(oracle.dequantize_blockwise(q, c, a, 256) == 0)


def test_thread_count_does_not_change_results(maps):
    q = maps["signed"]
    x = (np.random.default_rng(6).standard_t(3, 200_000) * 1e-2).astype(np.float32)
    r1 = oracle.quantize_blockwise(q, x, 2048, nthreads=1)
    r4 = oracle.quantize_blockwise(q, x, 2048, nthreads=4)
    np.testing.assert_array_equal(r1[0], r4[0])
    np.testing.assert_array_equal(r1[1], r4[1])


def test_quantization_error_bound(maps):
    """|x - dequant(quant(x))| <= N_b * (largest code gap) / 2."""
    q = maps["signed"]
    B = 2048
    x = (np.random.default_rng(7).standard_t(3, 8 * B) * 1e-2).astype(np.float32)
    c, a = oracle.quantize_blockwise(q, x, B)
    xd = oracle.dequantize_blockwise(q, c, a, B)
    gap = float(np.diff(q.astype(np.float64)).max())
    bound = np.repeat(a.astype(np.float64), B) * (gap / 2) * (1 + 1e-6)
    assert np.all(np.abs(x.astype(np.float64) - xd) <= bound)


def test_half_to_float_all_patterns():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.half_to_float(h)
    ref = h.view(np.float16).astype(np.float32)
    finite = np.isfinite(ref)
    np.testing.assert_array_equal(got[finite].view(np.uint32), ref[finite].view(np.uint32))
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(np.isinf(got), np.isinf(ref))
