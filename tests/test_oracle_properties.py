"""Property tests of the oracle's block-wise quantize / dequantize over shapes
and value mixes drawn by hypothesis (Section 3.1, Eq. 3 / Eq. 4, Section 2.2).

Hypothesis draws the shape (n, B), a seed and the mix of values (scale,
share of zeros and signed zeros, exact-midpoint ties, blocks scaled into the
subnormal range); numpy builds the array.  Every block is checked against
definitions that share no code with the oracle: absmax = max |x| over the
block, the code of each element is the exact-rational argmin of |q_j - y| with
y = x / N_b in binary32 (numpy), lowest index on ties; dequantization is
q[code] * N_b; the largest element maps to +-1 and comes back exactly.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
from tests.test_oracle_quant import exact_nearest_many

BLOCKS = [256, 512, 1024, 2048, 4096]


@pytest.fixture(scope="module")
def maps():
    return {"signed": oracle.dynamic_codebook(0), "unsigned": oracle.dynamic_codebook(1)}


def build_values(n, seed, log2_scale, zero_frac, tie_frac, tiny_block, qmap, signed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_t(3, n) * np.exp2(log2_scale)).astype(np.float32)
    if not signed:
        x = np.abs(x)
    zeros = rng.random(n) < zero_frac
    x[zeros] = np.float32(0.0)
    if signed:
        # signed zeros too
        x[zeros & (rng.random(n) < 0.5)] = np.float32(-0.0)
    # exact midpoints of adjacent codes, times a power of two: y = x / N is
    # then the midpoint itself whenever the block's absmax is that power of two
    mids = [(float(qmap[j]) + float(qmap[j + 1])) / 2 for j in range(255)]
    mids = np.array([m for m in mids if float(np.float32(m)) == m], np.float32)
    ties = rng.random(n) < tie_frac
    if ties.any() and mids.size:
        x[ties] = rng.choice(mids, ties.sum()) * np.float32(2.0 ** log2_scale)
    if tiny_block:
        # one stretch far below the normal range of fp32 quotients
        s = rng.integers(0, n)
        x[s:s + 300] = (x[s:s + 300].astype(np.float64) * 2.0 ** -130).astype(np.float32)
    return np.ascontiguousarray(x)


def check_blocks(qmap, x, B, codes, absmax):
    n = x.size
    nb = (n + B - 1) // B
    assert absmax.size == nb
    zero_code = int(np.flatnonzero(qmap == 0.0)[0])
    for b in range(nb):
        s = slice(b * B, min((b + 1) * B, n))
        xb = x[s]
        N = np.float32(np.max(np.abs(xb)))
        assert absmax[b].view(np.uint32) == N.view(np.uint32), b
        if N == 0:
            assert np.all(codes[s] == zero_code)
            continue
        y = (xb / N).astype(np.float32)            # one binary32 division each
        want = exact_nearest_many(qmap, y)
        np.testing.assert_array_equal(codes[s].astype(np.int64), want)
        # the absmax element is +-1 exactly and dequantizes to +-N exactly
        k = int(np.argmax(np.abs(xb)))
        assert abs(float(qmap[codes[s][k]])) == 1.0
        assert abs(np.float32(qmap[codes[s][k]] * N)) == N


@settings(max_examples=60, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow])
@given(n=st.integers(1, 9000), B=st.sampled_from(BLOCKS), seed=st.integers(0, 2**31 - 1),
       log2_scale=st.integers(-60, 60), zero_frac=st.sampled_from([0.0, 0.01, 0.5, 1.0]),
       tie_frac=st.sampled_from([0.0, 0.05, 0.5]), tiny_block=st.booleans(),
       name=st.sampled_from(["signed", "unsigned"]))
def test_blockwise_quantize_properties(maps, n, B, seed, log2_scale, zero_frac, tie_frac,
                                       tiny_block, name):
    q = maps[name]
    x = build_values(n, seed, log2_scale, zero_frac, tie_frac, tiny_block, q,
                     signed=(name == "signed"))
    codes, absmax = oracle.quantize_blockwise(q, x, B)
    check_blocks(q, x, B, codes, absmax)
    # the brute-force search is the same function
    cb, ab = oracle.quantize_blockwise(q, x, B, brute=True)
    np.testing.assert_array_equal(cb, codes)
    np.testing.assert_array_equal(ab.view(np.uint32), absmax.view(np.uint32))
    # dequantize: q[code] * N_b in binary32, and within half the largest gap of x
    out = oracle.dequantize_blockwise(q, codes, absmax, B)
    blk = np.arange(n) // B
    want = (q[codes] * absmax[blk]).astype(np.float32)
    np.testing.assert_array_equal(out.view(np.uint32), want.view(np.uint32))
    gap = float(np.max(np.diff(q.astype(np.float64))))
    err = np.abs(out.astype(np.float64) - x.astype(np.float64))
    bound = absmax[blk].astype(np.float64) * (gap / 2) * (1 + 2.0 ** -20) + 2.0 ** -149
    assert np.all(err <= bound)
    # a second round trip is a fixed point wherever q_j * N_b stays a normal
    # number for every code (N_b >= 2^-100; below that q[code] * N_b loses bits
    # or underflows, and the dequantized values need not quantize back)
    c2, a2 = oracle.quantize_blockwise(q, out, B)
    big = absmax >= np.float32(2.0 ** -100)
    np.testing.assert_array_equal(c2[big[blk]], codes[big[blk]])
    np.testing.assert_array_equal(a2.view(np.uint32), absmax.view(np.uint32))
