// Dynamic (tree) quantization codebooks, built on the host.
//
// Section 2.3: after the sign bit, a run of E zero bits gives the decimal
// exponent 10^-E, a one bit marks the end of the run, and the F bits after it
// are a linear fraction.  Section 3.2: for unsigned data the sign bit becomes
// one more fraction bit.  Each decade (10^-(E+1), 10^-E] holds 2^F values
//     10^-E * (0.1 + 0.9 j / 2^F) = (2^F + 9 j) / (10^(E+1) 2^F),  j = 1..2^F,
// so the top of every decade, and in particular 1.0, is exactly representable.
// Signed map: E = 0..6 (F = 6 - E) for each sign, plus 0 and +1e-7 from the two
// patterns without an indicator bit.  Unsigned map: E = 0..7 (F = 7 - E) plus 0.
//
// Every value is the exact rational rounded once to fp32 (round to nearest,
// ties to even), done here with integer long division.
#include <algorithm>
#include <cmath>
#include <cstdint>

#include "bq_internal.h"

namespace bq {
namespace {

// Round num / den (positive integers, value in [1e-7, 1], num < 2^11,
// den < 2^34) to the nearest fp32.  num * 2^k stays below 2^11 * 2^48.
float round_rational_to_f32(uint64_t num, uint64_t den)
{
    // Smallest k with floor(num * 2^k / den) >= 2^23; then that quotient is
    // below 2^24 because doubling from below 2^23 cannot pass 2^24.
    int k = 0;
    while ((num << k) / den < (1u << 23))
        ++k;
    uint64_t scaled = num << k;
    uint64_t mant = scaled / den, rem = scaled % den;
    if (2 * rem > den || (2 * rem == den && (mant & 1)))
        ++mant;
    if (mant == (1u << 24)) {
        mant >>= 1;
        --k;
    }
    return std::ldexp(static_cast<float>(mant), -k);
}

float decade_entry(int E, int F, int j)
{
    uint64_t num = (1ull << F) + 9ull * static_cast<uint64_t>(j);
    uint64_t den = 1ull << F;
    for (int i = 0; i <= E; ++i)
        den *= 10;
    return round_rational_to_f32(num, den);
}

}  // namespace

int build_dynamic_codebook(int kind, float out[256])
{
    int n = 0;
    if (kind == 0) {
        for (int E = 0; E <= 6; ++E) {
            int F = 6 - E;
            for (int j = 1; j <= (1 << F); ++j) {
                float v = decade_entry(E, F, j);
                out[n++] = -v;
                out[n++] = v;
            }
        }
        out[n++] = 0.0f;
        out[n++] = decade_entry(7, 0, 1);  // 1e-7
    } else if (kind == 1) {
        out[n++] = 0.0f;
        for (int E = 0; E <= 7; ++E) {
            int F = 7 - E;
            for (int j = 1; j <= (1 << F); ++j)
                out[n++] = decade_entry(E, F, j);
        }
    } else {
        return -1;
    }
    std::sort(out, out + 256);
    return n == 256 ? 0 : -1;
}

}  // namespace bq
