// Quantization codebooks, built on the host: dynamic (tree) maps, their
// inverse, linear maps, and quantile maps from a sample.
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
//
// Inverse dynamic maps (App. F.1) swap the roles of the exponent run and the
// base: with E zero bits the value lies in decade 10^-(Emax-E) and keeps the
// same F fraction bits, so the most fraction bits go to the smallest decade.
// Signed: decades 10^-k with F = k bits for k = 0..6, both signs, plus 0 and
// +1e-7; unsigned: k = 0..7 plus 0.  Both reach exactly 1.
// Linear maps: (2i - 255) / 255 (signed) or i / 255 (unsigned), i = 0..255.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <vector>

#include "bq_internal.h"

namespace bq {
namespace {

// Round num / den (positive integers, value in [1e-8, 1], num < 2^11,
// den < 2^34) to the nearest fp32.  num * 2^k stays below 2^11 * 2^52.
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
    if (kind == 0 || kind == 2) {
        // dynamic: decade E with 6 - E fraction bits; inverse: decade k with k bits
        for (int E = 0; E <= 6; ++E) {
            const int F = 6 - E;
            const int decade = kind == 0 ? E : F;
            for (int j = 1; j <= (1 << F); ++j) {
                const float v = decade_entry(decade, F, j);
                out[n++] = -v;
                out[n++] = v;
            }
        }
        out[n++] = 0.0f;
        out[n++] = decade_entry(7, 0, 1);  // 1e-7
    } else if (kind == 1 || kind == 3) {
        out[n++] = 0.0f;
        for (int E = 0; E <= 7; ++E) {
            const int F = 7 - E;
            const int decade = kind == 1 ? E : F;
            for (int j = 1; j <= (1 << F); ++j)
                out[n++] = decade_entry(decade, F, j);
        }
    } else if (kind == 4 || kind == 5) {
        for (int i = 0; i < 256; ++i) {
            const int num = kind == 4 ? 2 * i - 255 : i;
            const float mag = num == 0 ? 0.0f : round_rational_to_f32((uint64_t)std::abs(num), 255);
            out[n++] = num < 0 ? -mag : mag;
        }
    } else {
        return -1;
    }
    std::sort(out, out + 256);
    return n == 256 ? 0 : -1;
}

int build_quantile_codebook(const float *sample, int64_t n, float out[256])
{
    if (!sample || n < 1)
        return -1;
    std::vector<double> s((size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        if (!std::isfinite(sample[i]))
            return -1;
        s[(size_t)i] = sample[i];
    }
    std::sort(s.begin(), s.end());
    // App. F.2: q_i = (Q(i / 257) + Q((i + 1) / 257)) / 2, i = 0..255, with the
    // sample quantile Q(p) = sorted[floor(p n)]; then scaled into [-1, 1]
    double Q[257];
    for (int i = 0; i <= 256; ++i) {
        const int64_t idx = (int64_t)(((__int128)i * n) / 257);
        Q[i] = s[(size_t)std::min<int64_t>(idx, n - 1)];
    }
    double q[256], amax = 0.0;
    for (int i = 0; i < 256; ++i) {
        q[i] = 0.5 * (Q[i] + Q[i + 1]);
        amax = std::max(amax, std::fabs(q[i]));
    }
    if (!(amax > 0.0))
        return -1;
    for (int i = 0; i < 256; ++i)
        out[i] = static_cast<float>(q[i] / amax);
    // repeated sample values can give equal entries: separate them by one ulp
    for (int i = 1; i < 256; ++i)
        if (!(out[i] > out[i - 1]))
            out[i] = std::nextafter(out[i - 1], INFINITY);
    return 0;
}

}  // namespace bq
