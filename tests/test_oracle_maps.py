"""Pins of the oracle's further codebooks (App. F) against what the paper fixes.

Inverse dynamic quantization (App. F.1) keeps the dynamic layout but counts the
exponent run from the other end: the base is 10^-7 and each zero bit raises
the decade by 10x, up to a maximum of 1.  Linear quantization is the uniform
256-level baseline.  Quantile quantization (App. F.2, Eq. 5) takes midpoints
of 2^k + 1 = 257 equally spaced sample quantiles.  The library builds the same
maps independently; both must agree bit for bit.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2110_02861_amd import workloads


def _to_f32(fr: Fraction) -> np.float32:
    return np.float32(float(fr))


def _decode_inverse_byte(byte: int, signed: bool) -> Fraction:
    """The dynamic bit layout (sign, E zero bits, indicator, F fraction bits),
    with E zero bits selecting decade 10^-(Emax - E) and F = Emax - E."""
    nbits = 7 if signed else 8
    emax = nbits - 1
    neg = signed and bool(byte & 0x80)
    mag = byte & ((1 << nbits) - 1)
    if mag == 0:
        if signed and not neg:
            return Fraction(1, 10 ** 7)      # the base
        return Fraction(0)
    E = nbits - mag.bit_length()
    F = mag.bit_length() - 1
    assert F == emax - E
    k = emax - E
    j = (mag & ((1 << F) - 1)) + 1
    val = Fraction(1, 10 ** k) * (Fraction(1, 10) + Fraction(9, 10) * Fraction(j, 2 ** F))
    return -val if neg else val


@pytest.mark.parametrize("signed,kind", [(True, 2), (False, 3)])
def test_inverse_dynamic_bit_layout(signed, kind):
    q = oracle.codebook(kind)
    decoded = sorted(_to_f32(_decode_inverse_byte(b, signed)) for b in range(256))
    np.testing.assert_array_equal(np.array(decoded, np.float32), q)


def test_inverse_dynamic_structure():
    s, u = oracle.codebook(2), oracle.codebook(3)
    for q in (s, u):
        assert np.all(np.diff(q) > 0) and q[-1] == 1.0
    assert s[0] == -1.0 and np.count_nonzero(s == 0) == 1 and u[0] == 0.0
    # decade 10^-k holds 2^k values: the most values at the small end
    for q, kmax in ((s[s > 0], 6), (u[u > 0], 7)):
        for k in range(kmax + 1):
            hi, lo = 10.0 ** (-k), 10.0 ** (-(k + 1))
            cnt = np.count_nonzero((q > np.float32(lo) * (1 + 1e-6)) & (q <= np.float32(hi)))
            assert cnt == 2 ** k, (k, cnt)
    # the base 10^-7 (signed), the smallest decade's bottom (unsigned)
    assert np.min(s[s > 0]) == np.float32(1e-7)
    assert np.min(u[u > 0]) == _to_f32(Fraction(1, 10 ** 7) * (Fraction(1, 10) + Fraction(9, 1280)))
    # the dynamic map's largest gap is at the top; the inverse map's there is 0.9
    assert np.diff(s.astype(np.float64)).max() == pytest.approx(0.9, abs=1e-7)


@pytest.mark.parametrize("kind,signed", [(4, True), (5, False)])
def test_linear_exact(kind, signed):
    q = oracle.codebook(kind)
    ref = [_to_f32(Fraction(2 * i - 255, 255) if signed else Fraction(i, 255)) for i in range(256)]
    np.testing.assert_array_equal(q, np.array(ref, np.float32))
    step = 2.0 / 255 if signed else 1.0 / 255
    np.testing.assert_allclose(np.diff(q.astype(np.float64)), step, rtol=0, atol=2.0 ** -23)
    if signed:
        np.testing.assert_array_equal(q, -q[::-1])


def test_quantile_closed_form():
    """For the sample 0, 1, ..., 257 m - 1 the quantiles are exact:
    Q(i / 257) = i m, q_i = (i + 1/2) m, normalized q_i = (2 i + 1) / 511."""
    for m in (1, 3, 40):
        x = np.arange(257 * m, dtype=np.float32)
        q = oracle.quantile_codebook(x)
        ref = np.array([_to_f32(Fraction(2 * i + 1, 511)) for i in range(256)], np.float32)
        np.testing.assert_array_equal(q, ref)
        # order of the sample does not matter
        rng = workloads.host_rng(0, "c2", m, 0)
        np.testing.assert_array_equal(oracle.quantile_codebook(rng.permutation(x)), ref)


def test_quantile_sign_and_scale():
    rng = workloads.host_rng(0, "c2", 9, 0)
    x = rng.standard_normal(50_000).astype(np.float32)
    q = oracle.quantile_codebook(x)
    assert np.max(np.abs(q)) == 1.0 and np.all(np.diff(q) > 0)
    # a scaled sample gives the same map (normalized by max |q|)
    np.testing.assert_array_equal(oracle.quantile_codebook(x * np.float32(8.0)), q)
    # a non-negative sample gives a map in [0, 1]
    qa = oracle.quantile_codebook(np.abs(x))
    assert qa[0] >= 0.0 and qa[-1] == 1.0
    # about n / 257 sample values fall between consecutive quantiles: the middle
    # map entries sit inside the sample's central range
    s = np.sort(x.astype(np.float64))
    scale = max(abs(0.5 * (s[0] + s[(x.size) // 257])), abs(q[-1]))
    assert np.all(np.abs(q) <= 1.0)
    assert scale > 0


def test_quantile_ties_and_small_samples():
    # fewer values than quantiles: repeated entries are moved up by one ulp
    for x in (np.array([5.0], np.float32), np.array([-1.0, 2.0, 2.0], np.float32),
              np.round(workloads.host_rng(0, "c2", 3, 0).standard_normal(1000)).astype(np.float32)):
        q = oracle.quantile_codebook(x)
        assert np.all(np.diff(q) > 0)
        assert np.max(np.abs(q)) >= 1.0
    with pytest.raises(ValueError):
        oracle.quantile_codebook(np.zeros(10, np.float32))
    with pytest.raises(ValueError):
        oracle.quantile_codebook(np.array([1.0, np.nan], np.float32))
    with pytest.raises(ValueError):
        oracle.quantile_codebook(np.zeros(0, np.float32))


def test_nearest_code_on_new_maps_brute_equals_search():
    """The oracle's two nearest-code routines agree on every midpoint +-1 ulp of
    each new map (ties to the lower index)."""
    rng = workloads.host_rng(0, "c2", 4, 0)
    maps = [oracle.codebook(k) for k in (2, 3, 4, 5)]
    maps.append(oracle.quantile_codebook(rng.standard_normal(10_000).astype(np.float32)))
    for q in maps:
        for j in range(255):
            m = np.float32((float(q[j]) + float(q[j + 1])) / 2.0)
            for y in (np.nextafter(m, np.float32(-np.inf), dtype=np.float32), m,
                      np.nextafter(m, np.float32(np.inf), dtype=np.float32)):
                assert oracle.nearest_brute(q, float(y)) == oracle.nearest_bsearch(q, float(y))


def test_library_builds_the_same_maps():
    from paper_2110_02861_amd import bq
    for k in range(6):
        np.testing.assert_array_equal(bq.bq_make_codebook(k), oracle.codebook(k))
    rng = workloads.host_rng(0, "c2", 5, 0)
    for x in (rng.standard_normal(30_001).astype(np.float32),
              np.abs(workloads.student_t_host(5000, seed=2)),
              np.round(rng.standard_normal(700)).astype(np.float32),
              np.array([3.0], np.float32)):
        np.testing.assert_array_equal(bq.bq_make_quantile_codebook(x), oracle.quantile_codebook(x))


def _exact_nearest(q, y):
    """Eq. 3 in exact rational arithmetic, ties to the lower index."""
    fy = Fraction(float(y))
    best, bestd = 0, abs(fy - Fraction(float(q[0])))
    for j in range(1, q.size):
        d = abs(fy - Fraction(float(q[j])))
        if d < bestd:
            best, bestd = j, d
    return best


def test_nearest_code_exact_where_double_rounding_would_tie():
    """Adjacent codes of very different magnitude, or symmetric about 0: the
    distances y - q are not exact in double there, the oracle's decision is."""
    q = oracle.codebook(4).copy()                       # linear: codes -1/255, +1/255 around 0
    ys = [np.float32(2.0 ** -149), np.float32(-2.0 ** -149), np.float32(0.0)]
    q2 = q.copy()
    q2[127] = np.float32(-1e-43)                        # a tiny code next to 1/255
    m = (Fraction(float(q2[127])) + Fraction(float(q2[128]))) / 2
    f = np.float32(float(m))
    ys += [f, np.nextafter(f, np.float32(-1)), np.nextafter(f, np.float32(1))]
    q3 = q.copy()
    q3[127], q3[128] = np.float32(-1e-43), np.float32(0.5)
    q3[129:] = np.linspace(0.5, 1.0, 128, dtype=np.float32)[1:]
    ys += [np.float32(0.25), np.nextafter(np.float32(0.25), np.float32(0)),
           np.nextafter(np.float32(0.25), np.float32(1))]
    for qm in (q, q2, q3):
        assert np.all(np.diff(qm) > 0)
        for y in ys:
            want = _exact_nearest(qm, y)
            assert oracle.nearest_brute(qm, float(y)) == want, (y, want)
            assert oracle.nearest_bsearch(qm, float(y)) == want, (y, want)


# --- chunked quantile estimate (App. G) ---

def test_chunked_quantiles_single_chunk_is_eq5():
    """With n <= chunk the estimate is the sample's own quantile map (Eq. 5)."""
    rng = workloads.host_rng(0, "c2", 6, 0)
    for n in (1, 7, 300, 4096):
        x = rng.standard_normal(n).astype(np.float32)
        if n == 1:
            x[0] = 2.5
        q = oracle.chunked_quantile_codebook(x)
        np.testing.assert_array_equal(q, oracle.quantile_codebook(x))


def test_chunked_quantiles_identical_chunks():
    """Chunks holding the same values (in any order) average to those values'
    quantile map, which is also the whole tensor's (each value repeated)."""
    rng = workloads.host_rng(0, "c2", 7, 0)
    base = rng.standard_normal(4096).astype(np.float32)
    x = np.concatenate([rng.permutation(base) for _ in range(5)])
    q = oracle.chunked_quantile_codebook(x)
    np.testing.assert_array_equal(q, oracle.quantile_codebook(base))
    np.testing.assert_array_equal(q, oracle.quantile_codebook(x))


def test_chunked_quantiles_converge_and_scale():
    rng = workloads.host_rng(0, "c2", 8, 0)
    x = rng.standard_normal(1_000_003).astype(np.float32)
    q = oracle.chunked_quantile_codebook(x)
    exact = oracle.quantile_codebook(x)
    assert np.all(np.diff(q) > 0)
    # away from the extreme tails the average of chunk quantiles is close to
    # the tensor's quantiles; the maps differ in scale, since the first entry
    # (the sample minimum: of each 4096-chunk, or of the whole tensor) sets
    # the normalization
    ratio = float(exact[240]) / float(q[240])
    np.testing.assert_allclose(q[8:-8].astype(np.float64) * ratio, exact[8:-8], atol=0.01)
    np.testing.assert_array_equal(oracle.chunked_quantile_codebook(x * np.float32(4.0)), q)
    z = oracle.chunked_quantile_codebook(np.zeros(5000, np.float32))
    assert z[0] == 0.0 and np.all(np.diff(z) > 0) and z[-1] < 1e-42


def _exact_chunked_map(x, chunk=4096):
    """App. G's estimate with exact rationals: per chunk a numpy sort and the
    sample quantiles sorted_c[floor(i L_c / 257)], their length-weighted
    average, Eq. 5's midpoints and the division by the largest magnitude, all
    as Fractions; one rounding to fp32 at the end (through double)."""
    from fractions import Fraction
    n = x.size
    S = [Fraction(0)] * 257
    for c0 in range(0, n, chunk):
        s = np.sort(x[c0:c0 + chunk].astype(np.float64))
        L = s.size
        for i in range(257):
            S[i] += L * Fraction(float(s[i * L // 257]))
    Q = [v / n for v in S]
    q = [(Q[i] + Q[i + 1]) / 2 for i in range(256)]
    amax = max(abs(v) for v in q)
    return np.array([float(v / amax) for v in q], np.float64).astype(np.float32)


def test_chunked_quantiles_equal_exact_weighted_average():
    """The double sums of the oracle equal App. G's average computed exactly,
    within one fp32 ulp (the oracle rounds its double sums; the exact form
    rounds once): a ragged last chunk, weighted by its length."""
    x = workloads.student_t_host(5 * 4096 + 1234, seed=11)
    q = oracle.chunked_quantile_codebook(x)
    ref = _exact_chunked_map(x)
    ulp = np.spacing(np.abs(ref))
    assert np.all(np.abs(q.astype(np.float64) - ref) <= ulp), \
        np.max(np.abs(q.astype(np.float64) - ref) / ulp)
    # an unweighted mean of the chunk quantiles is a different estimate here
    # (the short last chunk would count as much as a full one)
    sorted_chunks = [np.sort(x[c0:c0 + 4096]) for c0 in range(0, x.size, 4096)]
    unweighted = np.mean([[s[i * s.size // 257] for i in range(257)] for s in sorted_chunks],
                         axis=0)
    mid = (unweighted[:-1] + unweighted[1:]) / 2
    alt = (mid / np.max(np.abs(mid))).astype(np.float32)
    assert np.max(np.abs(alt.astype(np.float64) - ref) / ulp) > 4
