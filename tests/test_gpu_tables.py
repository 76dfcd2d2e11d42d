"""GPU: the decision tables of a prepared codebook against their definition.

Eq. 3's nearest code is #{j : y >= T_j} with T_j the smallest binary32 above
the exact midpoint of codes j and j + 1 (T_255 = +inf).  The prepared buffer
holds q, T, and per bucket of the fp32 bit pattern (bits 30..16 of |y|,
clamped to the binades [2^-25, 2)) the count of thresholds at or below the
bucket's smallest value, for both signs, plus the largest number of thresholds
strictly inside one bucket.  Every entry is recomputed here from that
definition (exact rationals for the midpoints, IEEE binary32 comparisons for
the counts) and compared byte for byte, for the library's maps and for maps
built to put thresholds on bucket edges, at +-0 and across the whole binary32
range.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

from paper_2110_02861_amd import bq
from tests.gpu_helpers import dev, host, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]

SHIFT = 16
LO = (127 - 25) << 7
HI = (127 << 7) + 127
NB = HI - LO + 1
OFF_T, OFF_BASE = 1024, 2048
OFF_KMAX = OFF_BASE + 2 * NB


def f32(bits):
    return np.array(bits, np.uint32).view(np.float32)


def bucket_edges():
    b = np.arange(NB, dtype=np.int64)
    lo = np.where(b == 0, 0, (LO + b) << SHIFT).astype(np.uint32)
    hi = np.where(b == NB - 1, 0x7F7FFFFF, ((LO + b + 1) << SHIFT) - 1).astype(np.uint32)
    return f32(lo), f32(hi)


def thresholds(q):
    t = np.full(256, np.inf, np.float32)
    for j in range(255):
        m = (Fraction(float(q[j])) + Fraction(float(q[j + 1]))) / 2
        f = np.float32(float(m))
        while Fraction(float(f)) <= m:
            f = np.nextafter(f, np.float32(np.inf), dtype=np.float32)
        while True:
            g = np.nextafter(f, np.float32(-np.inf), dtype=np.float32)
            if Fraction(float(g)) > m:
                f = g
            else:
                break
        t[j] = f
    return t


def count_le(t, v):
    """#{j : t_j <= v_i} for each v_i, in binary32 comparisons."""
    return (t[None, :] <= v[:, None]).sum(axis=1)


def expected_tables(q):
    t = thresholds(q)
    lo, hi = bucket_edges()
    pos = count_le(t, lo)
    neg = count_le(t, -hi)
    inside = np.maximum(count_le(t, hi) - pos, count_le(t, -lo) - neg)
    return t, np.concatenate([pos, neg]).astype(np.uint8), int(inside.max())


def check_map(q, what):
    q = np.asarray(q, np.float32)
    assert np.all(np.diff(q.astype(np.float64)) > 0), what
    say(f"prepare {what}")
    prep = bq.bq_prepare_codebook(dev(q))
    torch.cuda.synchronize()
    got = host(prep)
    t, base, kmax = expected_tables(q)
    np.testing.assert_array_equal(got[:1024].view(np.uint32), q.view(np.uint32), err_msg=what)
    np.testing.assert_array_equal(got[OFF_T:OFF_T + 1024].view(np.uint32), t.view(np.uint32),
                                  err_msg=what)
    np.testing.assert_array_equal(got[OFF_BASE:OFF_KMAX], base, err_msg=what)
    assert int(got[OFF_KMAX:OFF_KMAX + 4].view(np.int32)[0]) == kmax, what


@pytest.mark.parametrize("kind", range(6))
def test_library_maps(kind):
    check_map(bq.bq_make_codebook(kind), f"codebook kind {kind}")


def test_quantile_map():
    rng = np.random.default_rng(3)
    check_map(bq.bq_make_quantile_codebook(rng.standard_t(3, 100_000).astype(np.float32)),
              "quantile of Student-t")


@pytest.mark.parametrize("seed", range(4))
def test_random_maps(seed):
    rng = np.random.default_rng(100 + seed)
    uni = np.unique(rng.uniform(-1, 1, 400).astype(np.float32))
    check_map(np.sort(rng.choice(uni, 256, replace=False)), f"uniform seed {seed}")
    mags = (10.0 ** rng.uniform(-7, 0, 400)) * np.sign(rng.standard_normal(400))
    u = np.unique(mags.astype(np.float32))
    check_map(np.sort(rng.choice(u, 256, replace=False)), f"log-uniform seed {seed}")
    wide = (2.0 ** rng.uniform(-140, 100, 400)) * np.sign(rng.standard_normal(400))
    u = np.unique(np.concatenate([wide, [0.0]]).astype(np.float32))
    check_map(np.sort(rng.choice(u, 256, replace=False)), f"wide range seed {seed}")


def edge_pairs(v):
    """Two codes whose threshold is exactly v: the midpoint of v - 2 ulp and v
    lies one ulp below v."""
    a = np.nextafter(np.nextafter(v, np.float32(-np.inf), dtype=np.float32), np.float32(-np.inf),
                     dtype=np.float32)
    return [a, v]


def test_thresholds_on_bucket_edges_and_at_zero():
    """Thresholds equal to a bucket's smallest value (positive half) or to
    -(a bucket's largest value) (negative half) count for that bucket and lie
    inside none; thresholds of +-0 lie inside the first negative bucket."""
    lo, hi = bucket_edges()
    rng = np.random.default_rng(9)
    picks = np.sort(rng.choice(np.arange(1, NB - 1), 40, replace=False))
    vals = []
    for b in picks[:20]:
        vals += edge_pairs(lo[b])
    for b in picks[20:]:
        vals += edge_pairs(-hi[b])
    # a threshold of -0.0: codes -2^-148 and 0 (midpoint -2^-149)
    vals += [np.float32(-(2.0 ** -148)), np.float32(0.0)]
    vals += [np.float32(1.5), np.float32(3.0), np.float32(-3.0), np.float32(1e-9)]
    u = np.unique(np.array(vals, np.float32))
    fill = np.unique(np.linspace(-0.9, 0.9, 300).astype(np.float32))
    rest = np.setdiff1d(fill, u)
    q = np.sort(np.concatenate([u, rng.choice(rest, 256 - u.size, replace=False)]))
    t, _, _ = expected_tables(q)
    assert np.any(t == 0.0) and np.any(np.signbit(t[t == 0.0]))
    assert np.isin(lo[picks[:20]], t).all() and np.isin(-hi[picks[20:]], t).all()
    check_map(q, "bucket edges and -0")


def test_many_thresholds_in_one_bucket():
    """The unsigned inverse dynamic map puts many thresholds into the first
    bucket; a map with 200 codes inside one bucket of [1, 1 + 2^-7) pushes the
    largest count far up."""
    check_map(bq.bq_make_codebook(bq.BQ_INVERSE_UNSIGNED), "inverse unsigned")
    base = np.float32(1.0)
    dense = [base]
    for _ in range(199):
        dense.append(np.nextafter(dense[-1], np.float32(2.0), dtype=np.float32))
    low = np.linspace(-1.0, 0.5, 56).astype(np.float32)
    q = np.sort(np.concatenate([low, np.array(dense, np.float32)]))
    _, _, kmax = expected_tables(q)
    assert kmax >= 150
    check_map(q, "200 codes in one bucket")
