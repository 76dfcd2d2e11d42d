"""Pins of the oracle's codebooks against what the paper fixes.

Section 2.3: dynamic tree quantization = sign bit, a run of zero bits giving a
decimal exponent, an indicator one bit, then linear fraction bits; range
[-1, 1] with magnitudes down to 10^-7.  Section 3.2: the unsigned variant turns
the sign bit into one more fraction bit.  Appendix F.1: base exponent 10^0,
each zero bit divides by 10, minimum 10^-7.

The exact values depend on a reading of the missing layout figure ("parity
unpinned" for the values themselves); the structure below is pinned.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def maps():
    return oracle.dynamic_codebook(oracle.SIGNED), oracle.dynamic_codebook(oracle.UNSIGNED)


def test_shape_sorted_distinct(maps):
    for q in maps:
        assert q.dtype == np.float32 and q.shape == (256,)
        assert np.all(np.diff(q) > 0)  # strictly increasing: code = rank
        assert len(set(q.tolist())) == 256


def test_endpoints_and_zero(maps):
    s, u = maps
    assert s[0] == -1.0 and s[255] == 1.0 and s[127] == 0.0
    assert u[0] == 0.0 and u[255] == 1.0
    # exactly one zero in each map
    assert np.count_nonzero(s == 0) == 1 and np.count_nonzero(u == 0) == 1


def _decade_counts(vals):
    counts = {}
    for E in range(8):
        hi, lo = 10.0 ** (-E), 10.0 ** (-(E + 1))
        counts[E] = int(np.count_nonzero((vals > np.float32(lo) * (1 + 1e-6)) &
                                         (vals <= np.float32(hi))))
    return counts


def test_bits_per_decade_signed(maps):
    s, _ = maps
    # E zero bits after the sign leave 6 - E fraction bits: 2^(6-E) values
    pos = _decade_counts(s[s > 0])
    neg = _decade_counts(-s[s < 0])
    for E in range(7):
        assert pos[E] == 2 ** (6 - E), (E, pos)
        assert neg[E] == 2 ** (6 - E), (E, neg)
    assert pos[7] == 1 and neg[7] == 0  # the single 10^-7 magnitude


def test_bits_per_decade_unsigned(maps):
    _, u = maps
    c = _decade_counts(u[u > 0])
    for E in range(8):
        assert c[E] == 2 ** (7 - E), (E, c)


def test_range_seven_orders_of_magnitude(maps):
    for q in maps:
        nz = np.abs(q[q != 0])
        assert nz.min() == np.float32(1e-7)
        assert nz.max() == 1.0
        assert round(float(np.log10(nz.max() / nz.min()))) == 7


def _decode_tree_byte(byte: int, signed: bool) -> Fraction:
    """Decode one 8-bit pattern following the bit layout of Section 2.3, exactly.

    signed: bit 7 = sign, then the 7 remaining bits; unsigned: all 8 bits.  A run
    of E leading zero bits is the exponent 10^-E; the following one bit is the
    indicator; the F bits after it are a linear fraction j-1 in [0, 2^F), mapped
    into the decade (10^-(E+1), 10^-E] as 10^-E * (0.1 + 0.9 * j / 2^F).
    A pattern with no indicator bit is 0, except the positive signed all-zero
    magnitude, which is the 10^-7 end of the range.
    """
    nbits = 7 if signed else 8
    neg = signed and bool(byte & 0x80)
    mag = byte & ((1 << nbits) - 1)
    if mag == 0:
        if signed and not neg:
            return Fraction(1, 10 ** 7)
        return Fraction(0)
    E = nbits - mag.bit_length()      # leading zero bits
    F = mag.bit_length() - 1          # bits after the indicator
    j = (mag & ((1 << F) - 1)) + 1
    val = Fraction(1, 10 ** E) * (Fraction(1, 10) + Fraction(9, 10) * Fraction(j, 2 ** F))
    return -val if neg else val


def _to_f32(fr: Fraction) -> np.float32:
    # correctly rounded via exact integer scaling: float(Fraction) is RN to double;
    # from a 53-bit RN value of a short rational the float32 rounding is exact
    return np.float32(float(fr))


@pytest.mark.parametrize("signed", [True, False])
def test_bit_layout_decode_matches(maps, signed):
    q = maps[0] if signed else maps[1]
    decoded = sorted(_to_f32(_decode_tree_byte(b, signed)) for b in range(256))
    np.testing.assert_array_equal(np.array(decoded, np.float32), q)


def test_linear_fraction_inside_decades(maps):
    s, u = maps
    for q, fbits in ((s, 6), (u, 7)):
        pos = q[q > 0].astype(np.float64)
        for E in range(fbits + 1):
            hi, lo = 10.0 ** (-E), 10.0 ** (-(E + 1))
            d = pos[(pos > lo * (1 + 1e-6)) & (pos <= hi * (1 + 1e-6))]
            if d.size < 2:
                continue
            step = 0.9 * 10.0 ** (-E) / 2 ** (fbits - E)
            # each value is rounded once to binary32: a difference is off by <= 1 ulp
            np.testing.assert_allclose(np.diff(d), step, rtol=0, atol=2.0 ** -23 * hi)


def test_largest_gap(maps):
    s, u = maps
    # one code step of the top decade: 0.9 / 64 and 0.9 / 128
    assert abs(np.diff(s.astype(np.float64)).max() - 0.9 / 64) <= 2.0 ** -23
    assert abs(np.diff(u.astype(np.float64)).max() - 0.9 / 128) <= 2.0 ** -23


def test_unknown_kind_rejected():
    with pytest.raises(ValueError):
        oracle.dynamic_codebook(7)
