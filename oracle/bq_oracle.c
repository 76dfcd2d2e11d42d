/*
 * Plain, slow CPU oracle for 8-bit block-wise optimizers
 * (Dettmers et al., "8-bit Optimizers via Block-wise Quantization", ICLR 2022).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference the HIP library is
 * checked against.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it; the product path never does.  It shares no
 * code, header, table or constant generator with the HIP library.
 *
 * Arithmetic rules: IEEE binary32 with round-to-nearest-even, no contraction of
 * a*b+c into an fma (build with -ffp-contract=off), no fast-math, denormals kept.
 * The paper fixes the precision of the optimizer update at 32 bits (Section 3:
 * states are dequantized to 32 bits, updated, requantized), so the update is
 * written in float, in the operation order stated next to each function.
 *
 * Readings of points the paper leaves open are marked "Reading:" below.
 *
 * Parity unpinned: the exact values of the dynamic and inverse dynamic maps.
 * The paper's figure of the bit layout is missing, so the values below are a
 * reading of its text; the tests pin their structure (values per decade, the
 * 10^-7 .. 1 range, 0 and +-1 present, strictly increasing), not the values.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_API __attribute__((visibility("default")))

/* ------------------------------------------------------------------------- */
/* Codebooks: Section 2.3 (dynamic tree quantization), Section 3.2 (dynamic   */
/* quantization for unsigned data), Appendix F.1 (10^-7 .. 1 range).          */
/* ------------------------------------------------------------------------- */

/*
 * One "decade" of the dynamic data type.  After the sign bit, E zero bits set
 * the decimal exponent 10^-E, a one bit ends the run, and the remaining F bits
 * are a linear fraction (Section 2.3).  Reading: the 2^F fraction values split
 * the decade (10^-(E+1), 10^-E] into equal steps, j = 1..2^F, so
 *     value(E, F, j) = 10^-E * (0.1 + 0.9 * j / 2^F)
 *                    = (2^F + 9 j) / (10^(E+1) * 2^F).
 * The top value of each decade is 10^-E itself, so +-1 is in the map and the
 * block absmax element is reconstructed exactly (Section 3.1).
 *
 * The rational form has a numerator below 2^11 and a denominator 5^(E+1) *
 * 2^(E+1+F) whose odd part is below 2^24, so both are exact binary32 values and
 * one double division followed by a float conversion is the correctly rounded
 * binary32 value of the rational (double rounding is innocuous for a single
 * division when 53 >= 2*24 + 2).
 */
static float decade_value(int E, int F, int j)
{
    double num = (double)((1 << F) + 9 * j);
    double den = (double)(1 << F);
    for (int k = 0; k <= E; ++k)
        den *= 10.0; /* exact: 10^8 * 2^7 < 2^53 */
    return (float)(num / den);
}

static int cmp_float(const void *a, const void *b)
{
    float x = *(const float *)a, y = *(const float *)b;
    return (x > y) - (x < y);
}

/*
 * kind 0 = signed dynamic tree map (state 1 of Adam, the Momentum state).
 *   Reading: per sign, E = 0..6 zero bits leave F = 6 - E fraction bits,
 *   giving 64 + 32 + ... + 1 = 127 magnitudes; the two all-zero magnitude
 *   patterns are 0 (negative sign) and the smallest magnitude 10^-7 (positive
 *   sign), the "10^-7" end of the range.  127 + 127 + 2 = 256 values.
 * kind 1 = unsigned dynamic map (state 2 of Adam, Section 3.2): the sign bit
 *   becomes one more fraction bit, so E = 0..7 zero bits leave F = 7 - E
 *   fraction bits: 128 + 64 + ... + 1 = 255 magnitudes, plus 0.
 * The result is sorted ascending so that code = rank.  Returns 0 on success,
 * -1 for an unknown kind.
 */
ORACLE_API int oracle_dynamic_codebook(int kind, float out[256])
{
    int k = 0;
    if (kind == 0) {
        for (int E = 0; E <= 6; ++E)
            for (int j = 1; j <= (1 << (6 - E)); ++j) {
                float v = decade_value(E, 6 - E, j);
                out[k++] = v;
                out[k++] = -v;
            }
        out[k++] = 0.0f;
        out[k++] = decade_value(7, 0, 1); /* 1e-7 */
    } else if (kind == 1) {
        for (int E = 0; E <= 7; ++E)
            for (int j = 1; j <= (1 << (7 - E)); ++j)
                out[k++] = decade_value(E, 7 - E, j);
        out[k++] = 0.0f;
    } else {
        return -1;
    }
    qsort(out, 256, sizeof(float), cmp_float);
    return 0;
}

/*
 * Further fixed maps (App. F):
 * kind 2 / 3 = inverse dynamic, signed / unsigned (App. F.1).  Reading: the
 *   exponent run is counted from the small end -- with E zero bits the value
 *   lies in decade 10^-(Emax - E) (Emax = 6 signed, 7 unsigned) and keeps
 *   F = Emax - E fraction bits, so decade 10^-k holds 2^k values:
 *   signed: +-10^-k (0.1 + 0.9 j / 2^k), j = 1..2^k, k = 0..6, plus 0 and
 *   +1e-7 (the base); unsigned: k = 0..7, plus 0.
 * kind 4 / 5 = linear, signed / unsigned (the ablation baseline): 256 evenly
 *   spaced values, (2i - 255) / 255 or i / 255, i = 0..255.
 * kinds 0 and 1 are the dynamic maps above.  Sorted ascending.  Returns 0, or
 * -1 for an unknown kind.
 */
ORACLE_API int oracle_codebook(int kind, float out[256])
{
    int k = 0;
    if (kind == 0 || kind == 1)
        return oracle_dynamic_codebook(kind, out);
    if (kind == 2) {
        for (int dec = 0; dec <= 6; ++dec)
            for (int j = 1; j <= (1 << dec); ++j) {
                float v = decade_value(dec, dec, j);
                out[k++] = v;
                out[k++] = -v;
            }
        out[k++] = 0.0f;
        out[k++] = decade_value(7, 0, 1); /* 1e-7 */
    } else if (kind == 3) {
        for (int dec = 0; dec <= 7; ++dec)
            for (int j = 1; j <= (1 << dec); ++j)
                out[k++] = decade_value(dec, dec, j);
        out[k++] = 0.0f;
    } else if (kind == 4 || kind == 5) {
        for (int i = 0; i < 256; ++i)
            out[k++] = (float)((kind == 4 ? (double)(2 * i - 255) : (double)i) / 255.0);
    } else {
        return -1;
    }
    qsort(out, 256, sizeof(float), cmp_float);
    return 0;
}

static int cmp_double(const void *a, const void *b)
{
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/*
 * Quantile map of a sample (App. F.2, Eq. 5): with the sample quantile
 * Q(p) = sorted[floor(p n)] (the value at index p n of the sorted sample),
 *   q_i = (Q(i / (2^k + 1)) + Q((i + 1) / (2^k + 1))) / 2,  i = 0..2^k - 1,
 * k = 8, in double; then divided by max |q_i| so the map spans [-1, 1]
 * (Fig. of the data types normalizes the map that way) and rounded to fp32.
 * Reading: equal entries (ties in the sample) are moved up by one ulp in
 * order, keeping code = rank well defined.  Returns 0, or -1 for n < 1, a
 * non-finite value or an all-zero map.
 */
ORACLE_API int oracle_quantile_codebook(const float *x, int64_t n, float out[256])
{
    if (n < 1)
        return -1;
    double *s = (double *)malloc(sizeof(double) * (size_t)n);
    if (!s)
        return -1;
    for (int64_t i = 0; i < n; ++i) {
        if (!isfinite(x[i])) {
            free(s);
            return -1;
        }
        s[i] = x[i];
    }
    qsort(s, (size_t)n, sizeof(double), cmp_double);
    double q[256], amax = 0.0;
    for (int i = 0; i < 256; ++i) {
        int64_t a = (int64_t)((__int128)i * n / 257);
        int64_t b = (int64_t)((__int128)(i + 1) * n / 257);
        if (a > n - 1)
            a = n - 1;
        if (b > n - 1)
            b = n - 1;
        q[i] = (s[a] + s[b]) / 2.0;
        if (fabs(q[i]) > amax)
            amax = fabs(q[i]);
    }
    free(s);
    if (!(amax > 0.0))
        return -1;
    for (int i = 0; i < 256; ++i) {
        out[i] = (float)(q[i] / amax);
        if (i > 0 && !(out[i] > out[i - 1]))
            out[i] = nextafterf(out[i - 1], INFINITY);
    }
    return 0;
}

/*
 * Chunked quantile estimate (App. G): the sample is cut into chunks of
 * `chunk` values (the last one shorter, length L_c); each chunk's sample
 * quantiles Q_c(i / 257) = sorted_c[floor(i L_c / 257)], i = 0..256, are
 * averaged over the chunks.
 * Reading: App. G averages the per-chunk quantiles; weighting each by its
 * length L_c makes a short last chunk count for what it holds.  The weighted
 * sum is accumulated in double in plain chunk order and divided by n (App. G
 * accumulates atomically, i.e. in no fixed order; any order is the same
 * average up to rounding).  The map then follows Eq. 5 as in
 * oracle_quantile_codebook, except that an all-zero map is kept (0, then
 * successive subnormals after the tie separation) instead of rejected.
 * Returns 0, or -1 for n < 1, chunk < 1 or a non-finite value.
 */
ORACLE_API int oracle_chunked_quantile_codebook(const float *x, int64_t n, int64_t chunk,
                                               float out[256])
{
    if (n < 1 || chunk < 1)
        return -1;
    double S[257];
    for (int i = 0; i <= 256; ++i)
        S[i] = 0.0;
    double *s = (double *)malloc(sizeof(double) * (size_t)chunk);
    if (!s)
        return -1;
    for (int64_t c0 = 0; c0 < n; c0 += chunk) {
        int64_t L = n - c0 < chunk ? n - c0 : chunk;
        for (int64_t i = 0; i < L; ++i) {
            if (!isfinite(x[c0 + i])) {
                free(s);
                return -1;
            }
            s[i] = x[c0 + i];
        }
        qsort(s, (size_t)L, sizeof(double), cmp_double);
        for (int i = 0; i <= 256; ++i)
            S[i] += (double)L * s[(int64_t)i * L / 257];
    }
    free(s);
    double Q[257], q[256], amax = 0.0;
    for (int i = 0; i <= 256; ++i)
        Q[i] = S[i] / (double)n;
    for (int i = 0; i < 256; ++i) {
        q[i] = (Q[i] + Q[i + 1]) * 0.5;
        if (fabs(q[i]) > amax)
            amax = fabs(q[i]);
    }
    for (int i = 0; i < 256; ++i) {
        out[i] = (float)(amax > 0.0 ? q[i] / amax : q[i]);
        if (i > 0 && !(out[i] > out[i - 1]))
            out[i] = nextafterf(out[i - 1], INFINITY);
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Nearest code: Eq. 3 / Eq. 4 argmin over the 256 map entries.               */
/* ------------------------------------------------------------------------- */

/*
 * Exact sign of 2y - (a + b) for binary32 y, a, b.  For a < b,
 * |y - a| < |y - b|  <=>  (y - a)^2 < (y - b)^2  <=>  2y (b - a) < b^2 - a^2
 *                    <=>  2y < a + b,
 * so this decides which of two codes is nearer.  It is evaluated in integers,
 * with no rounding at all: every finite binary32 is an integer multiple of
 * 2^-149 of magnitude below 2^128, so 2y, a and b are integers in units of
 * 2^-149 below 2^279 and their signed sum fits a 320-bit two's-complement
 * integer (five 64-bit limbs, least significant first).
 */
enum { WIDE_LIMBS = 5 };

/* acc += sign * m * 2^shift, for m < 2^24 and 0 <= shift <= 255 */
static void wide_add(uint64_t acc[WIDE_LIMBS], int negative, uint64_t m, int shift)
{
    uint64_t t[WIDE_LIMBS] = {0, 0, 0, 0, 0};
    const int limb = shift / 64, off = shift % 64;
    t[limb] = m << off;
    if (off > 40 && limb + 1 < WIDE_LIMBS)
        t[limb + 1] = m >> (64 - off);
    if (negative) { /* two's complement: invert, then add one below */
        for (int i = 0; i < WIDE_LIMBS; ++i)
            t[i] = ~t[i];
    }
    uint64_t carry = negative ? 1u : 0u;
    for (int i = 0; i < WIDE_LIMBS; ++i) {
        const uint64_t x = acc[i] + carry;
        const uint64_t c1 = x < carry;
        const uint64_t y = x + t[i];
        const uint64_t c2 = y < x;
        acc[i] = y;
        carry = c1 + c2;
    }
}

/* acc += (twice ? 2 : 1) * v in units of 2^-149, v finite */
static void wide_add_float(uint64_t acc[WIDE_LIMBS], float v, int twice)
{
    uint32_t bits;
    memcpy(&bits, &v, sizeof bits);
    const int negative = (int)(bits >> 31);
    const int biased = (int)((bits >> 23) & 0xffu);
    uint64_t m = bits & 0x7fffffu;
    int shift = 0; /* subnormal or zero: m * 2^-149 */
    if (biased != 0) { /* normal: (2^23 + m) * 2^(biased - 150) */
        m |= 0x800000u;
        shift = biased - 1;
    }
    wide_add(acc, negative, m, shift + (twice ? 1 : 0));
}

static int sign_twice_y_minus_sum(float y, float a, float b)
{
    if (!isfinite(y) || !isfinite(a) || !isfinite(b)) { /* outside the contract */
        const double t = 2.0 * (double)y, s = (double)a + (double)b;
        return (t > s) - (t < s);
    }
    uint64_t acc[WIDE_LIMBS] = {0, 0, 0, 0, 0};
    wide_add_float(acc, y, 1);
    wide_add_float(acc, -a, 0);
    wide_add_float(acc, -b, 0);
    if (acc[WIDE_LIMBS - 1] >> 63)
        return -1;
    for (int i = 0; i < WIDE_LIMBS; ++i)
        if (acc[i] != 0)
            return 1;
    return 0;
}

/*
 * Definition of Eq. 3: argmin_j |q_j - y| over j = 0..255 (Reading: the
 * printed upper limit 2^n means the last index 2^k - 1).  Ties go to the lower
 * index (Reading: the paper is silent; exact ties happen because many
 * midpoints of adjacent codes are binary32 numbers).  A linear scan keeps the
 * nearest code so far and moves to a later (larger) code only when that one is
 * strictly nearer, decided exactly by sign_twice_y_minus_sum.  Requires a
 * strictly increasing map.
 */
ORACLE_API int oracle_nearest_brute(const float *qmap, float y)
{
    int best = 0;
    for (int j = 1; j < 256; ++j)
        if (sign_twice_y_minus_sum(y, qmap[best], qmap[j]) > 0)
            best = j;
    return best;
}

/*
 * The same argmin by binary search (Section 2.2 finds the closest value "via a
 * binary search"): locate i with q_i <= y < q_{i+1}, then take i + 1 when y
 * lies strictly above the midpoint of q_i and q_{i+1} (the exact predicate
 * above), else i.  Requires a strictly increasing map.
 */
ORACLE_API int oracle_nearest_bsearch(const float *qmap, float y)
{
    if (!(y > qmap[0]))
        return 0;
    if (y >= qmap[255])
        return 255;
    int lo = 0, hi = 255; /* invariant: qmap[lo] < y < qmap[hi] or y == qmap[lo] */
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (qmap[mid] <= y)
            lo = mid;
        else
            hi = mid;
    }
    return sign_twice_y_minus_sum(y, qmap[lo], qmap[lo + 1]) > 0 ? lo + 1 : lo;
}

/* ------------------------------------------------------------------------- */
/* Block-wise quantization: Section 3.1, Eq. 4; dequantization: Section 2.2.  */
/* ------------------------------------------------------------------------- */

/*
 * Quantize one block of len values against qmap.
 *   N_b = max |x_i| over the block (exact).
 *   Reading: y = x_i / N_b is one binary32 division (RN-even); if N_b == 0 the
 *   block is all zeros and every element takes the code nearest to 0.
 *   code_i = nearest(y).
 */
static float quantize_block(const float *qmap, const float *x, int64_t len,
                            uint8_t *codes, int brute)
{
    float N = 0.0f;
    for (int64_t i = 0; i < len; ++i) {
        float a = fabsf(x[i]);
        if (a > N)
            N = a;
    }
    for (int64_t i = 0; i < len; ++i) {
        float y = (N == 0.0f) ? 0.0f : x[i] / N;
        codes[i] = (uint8_t)(brute ? oracle_nearest_brute(qmap, y)
                                   : oracle_nearest_bsearch(qmap, y));
    }
    return N;
}

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/*
 * x[n] -> codes[n] (uint8) and absmax[ceil(n/B)] (fp32).  Block b covers the
 * flat elements [b*B, min((b+1)*B, n)); the last block may be partial
 * (Reading: ceil(n/B) blocks).  brute selects the brute-force argmin.
 * nthreads > 0 sets the OpenMP team size; results do not depend on it.
 */
ORACLE_API void oracle_quantize_blockwise(const float *qmap, const float *x, int64_t n,
                                          int32_t B, uint8_t *codes, float *absmax,
                                          int brute, int nthreads)
{
    int64_t nb = (n + B - 1) / B;
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < nb; ++b) {
        int64_t s = b * B, len = (n - s < B) ? n - s : B;
        absmax[b] = quantize_block(qmap, x + s, len, codes + s, brute);
    }
}

/* out_i = qmap[code_i] * N_b, one binary32 multiply (Section 2.2). */
ORACLE_API void oracle_dequantize_blockwise(const float *qmap, const uint8_t *codes,
                                            const float *absmax, int64_t n, int32_t B,
                                            float *out, int nthreads)
{
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = qmap[codes[i]] * absmax[i / B];
}

/* ------------------------------------------------------------------------- */
/* Gradients in binary16 (mixed-precision training, Section 4 setup).        */
/* ------------------------------------------------------------------------- */

/* Exact binary16 -> binary32 from the bit fields (IEEE 754-2008, 3.4). */
static float half_to_float(uint16_t h)
{
    int sign = (h >> 15) & 1, e = (h >> 10) & 0x1f, f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(f | 0x400), e - 25);
    return (float)(sign ? -v : v);
}

ORACLE_API void oracle_half_to_float(const uint16_t *h, float *out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = half_to_float(h[i]);
}

/* ------------------------------------------------------------------------- */
/* Optimizer update: Eq. 1 (Momentum), Eq. 2 (Adam), AdamW.                   */
/* ------------------------------------------------------------------------- */

enum { OR_ADAM = 0, OR_ADAMW = 1, OR_MOMENTUM = 2, OR_ADAGRAD = 3, OR_LAMB = 4, OR_LARS = 5 };

/* beta^t by square-and-multiply in double (t >= 0). */
static double pow_int(double beta, int64_t t)
{
    double r = 1.0, b = beta;
    while (t > 0) {
        if (t & 1)
            r *= b;
        b *= b;
        t >>= 1;
    }
    return r;
}

/*
 * Per-step scalars.  Each is formed in double from the binary32 inputs and
 * rounded once to binary32.
 * Reading (Eq. 2 omits "damping and scaling constants"): textbook Adam with
 * bias correction and t starting at 1, written as
 *     denom = sqrt(v') * (1 / sqrt(1 - beta2^t)) + eps
 *     w'    = w - (lr / (1 - beta1^t)) * (m' / denom),
 * which is w - lr * mhat / (sqrt(vhat) + eps) with eps outside the root.
 * Reading (AdamW is named but not written out): decoupled decay, w <- w * (1 -
 * lr * wd) before the Adam update.  Adam and Momentum apply weight decay as an
 * L2 term added to the gradient, g <- g + wd * w.
 */
typedef struct {
    float b1, omb1, b2, omb2, eps, lr, wd, step_size, inv_sqrt_bc2, decay;
    float bc1_inv; /* 1 / (1 - beta1^t), LAMB's first-moment correction */
} step_scalars;

static step_scalars make_scalars(float lr, float beta1, float beta2, float eps,
                                 float wd, int64_t t)
{
    step_scalars s;
    s.b1 = beta1;
    s.omb1 = (float)(1.0 - (double)beta1);
    s.b2 = beta2;
    s.omb2 = (float)(1.0 - (double)beta2);
    s.eps = eps;
    s.lr = lr;
    s.wd = wd;
    s.step_size = (float)((double)lr / (1.0 - pow_int((double)beta1, t)));
    s.inv_sqrt_bc2 = (float)(1.0 / sqrt(1.0 - pow_int((double)beta2, t)));
    s.decay = (float)(1.0 - (double)lr * (double)wd);
    s.bc1_inv = (float)(1.0 / (1.0 - pow_int((double)beta1, t)));
    return s;
}

/*
 * One element of the 32-bit update.  In: w, g (fp32), m, v (fp32 states).
 * Out: updated *w, *m, *v.  v is untouched for Momentum.
 *   Adam:     g += wd*w (if wd != 0); m' = b1*m + (1-b1)*g;
 *             v' = b2*v + (1-b2)*(g*g); w' = w - step_size*(m'/denom)
 *   AdamW:    w *= decay; then Adam with no L2 term
 *   Momentum: g += wd*w (if wd != 0); m' = b1*m + g; w' = w - lr*m'
 *             (with m = 0 at the first step this gives m_0 = g_0, Eq. 1)
 *   AdaGrad (App. H; reading: the textbook method, no learning-rate decay,
 *             zero initial accumulator): g += wd*w (if wd != 0);
 *             m' = m + g*g (m holds the sum of squares);
 *             w' = w - lr*(g/(sqrt(m') + eps))
 */
static void update_element(int opt, const step_scalars *s, float *w, float g, float *m,
                           float *v)
{
    float wv = *w;
    if (opt == OR_ADAGRAD) {
        if (s->wd != 0.0f)
            g = g + s->wd * wv;
        float mn = *m + g * g;
        *m = mn;
        *w = wv - s->lr * (g / (sqrtf(mn) + s->eps));
        return;
    }
    if (opt == OR_MOMENTUM) {
        if (s->wd != 0.0f)
            g = g + s->wd * wv;
        float mn = s->b1 * (*m) + g;
        *m = mn;
        *w = wv - s->lr * mn;
        return;
    }
    if (opt == OR_ADAMW)
        wv = wv * s->decay;
    else if (s->wd != 0.0f)
        g = g + s->wd * wv;
    float mn = s->b1 * (*m) + s->omb1 * g;
    float vn = s->b2 * (*v) + s->omb2 * (g * g);
    float denom = sqrtf(vn) * s->inv_sqrt_bc2 + s->eps;
    *m = mn;
    *v = vn;
    *w = wv - s->step_size * (mn / denom);
}

static float load_grad(const void *g, int grad_is_f16, int64_t i)
{
    return grad_is_f16 ? half_to_float(((const uint16_t *)g)[i]) : ((const float *)g)[i];
}

/*
 * LAMB and LARS (App. E times 8-bit versions of both; the paper gives no
 * equations).  Reading: the textbook methods, with a per-tensor trust ratio
 * from the norms of the whole tensor, computed before the update:
 *   LAMB: m' = b1*m + (1-b1)*g;  v' = b2*v + (1-b2)*(g*g);
 *         u = (m' * bc1_inv) / (sqrt(v') * inv_sqrt_bc2 + eps) + wd*w;
 *         ratio = |w| / |u|;  w' = w - (lr*ratio) * u
 *   LARS: ratio = trust * |w| / (|g| + wd*|w|)  (g before weight decay);
 *         g' = g + wd*w;  m' = b1*m + (lr*ratio) * g';  w' = w - m'
 * with ratio = 1 when either norm is zero.  Norms are sums of squares in
 * double; lr*ratio is formed in double and rounded once to fp32.
 */
static float lamb_direction(const step_scalars *s, float w, float mn, float vn)
{
    float mh = mn * s->bc1_inv;
    float denom = sqrtf(vn) * s->inv_sqrt_bc2 + s->eps;
    return mh / denom + s->wd * w;
}

static float trust_lr(int opt, const step_scalars *s, double nw2, double nx2, float trust)
{
    double a = sqrt(nw2), b = sqrt(nx2), ratio = 1.0;
    if (a > 0.0 && b > 0.0)
        ratio = (opt == OR_LAMB) ? a / b : (double)trust * a / (b + (double)s->wd * a);
    return (float)((double)s->lr * ratio);
}

/* One element of LAMB / LARS given the tensor's lr*ratio. */
static void trust_update_element(int opt, const step_scalars *s, float lr_r, float *w, float g,
                                 float *m, float *v)
{
    float wv = *w;
    if (opt == OR_LAMB) {
        float mn = s->b1 * (*m) + s->omb1 * g;
        float vn = s->b2 * (*v) + s->omb2 * (g * g);
        float u = lamb_direction(s, wv, mn, vn);
        *m = mn;
        *v = vn;
        *w = wv - lr_r * u;
    } else {
        if (s->wd != 0.0f)
            g = g + s->wd * wv;
        float mn = s->b1 * (*m) + lr_r * g;
        *m = mn;
        *w = wv - mn;
    }
}

/* Squared norms (of w, and of u for LAMB or g for LARS) of one element. */
static void trust_norm_terms(int opt, const step_scalars *s, float w, float g, float m, float v,
                             double *nw2, double *nx2)
{
    *nw2 += (double)w * (double)w;
    if (opt == OR_LAMB) {
        float mn = s->b1 * m + s->omb1 * g;
        float vn = s->b2 * v + s->omb2 * (g * g);
        float u = lamb_direction(s, w, mn, vn);
        *nx2 += (double)u * (double)u;
    } else {
        *nx2 += (double)g * (double)g;
    }
}

/*
 * 32-bit reference step with quantization bypassed: fp32 states m[n], v[n]
 * (v unused for Momentum).  This is the special case that reduces to the
 * textbook optimizers.
 */
ORACLE_API int oracle_step32(int opt, int64_t n, float *w, const void *g, int grad_is_f16,
                             float *m, float *v, float lr, float beta1, float beta2,
                             float eps, float wd, int64_t step, float trust)
{
    if (opt < OR_ADAM || opt > OR_LARS || step < 1)
        return -1;
    int two = (opt == OR_ADAM || opt == OR_ADAMW || opt == OR_LAMB);
    step_scalars s = make_scalars(lr, beta1, beta2, eps, wd, step);
    if (opt == OR_LAMB || opt == OR_LARS) {
        double nw2 = 0.0, nx2 = 0.0;
        for (int64_t i = 0; i < n; ++i)
            trust_norm_terms(opt, &s, w[i], load_grad(g, grad_is_f16, i), m[i],
                             two ? v[i] : 0.0f, &nw2, &nx2);
        float lr_r = trust_lr(opt, &s, nw2, nx2, trust);
        for (int64_t i = 0; i < n; ++i) {
            float vi = two ? v[i] : 0.0f;
            trust_update_element(opt, &s, lr_r, &w[i], load_grad(g, grad_is_f16, i), &m[i], &vi);
            if (two)
                v[i] = vi;
        }
        return 0;
    }
    for (int64_t i = 0; i < n; ++i) {
        float vi = two ? v[i] : 0.0f;
        update_element(opt, &s, &w[i], load_grad(g, grad_is_f16, i), &m[i], &vi);
        if (two)
            v[i] = vi;
    }
    return 0;
}

/*
 * The 8-bit step on one tensor (Section 3, Fig. 1 caption), block by block:
 *   1. dequantize: m = Q1[c1] * N1_old, v = Q2[c2] * N2_old;
 *   2. 32-bit update of w, m, v (update_element);
 *   3. after the update, new block absmax N1 = max|m'|, N2 = max|v'|;
 *   4. requantize m' with Q1 and v' with Q2 to the nearest code.
 * The param update uses the unquantized m', v'.  c2, a2, q2 are unused (may be
 * NULL) for Momentum.  Returns 0, or -1 on a bad argument.
 */
ORACLE_API int oracle_step8(int opt, int32_t B, int grad_is_f16, int64_t n, float *w,
                            const void *g, uint8_t *c1, uint8_t *c2, float *a1, float *a2,
                            const float *q1, const float *q2, float lr, float beta1,
                            float beta2, float eps, float wd, int64_t step, int nthreads,
                            float trust)
{
    if (opt < OR_ADAM || opt > OR_LARS || step < 1 || B <= 0)
        return -1;
    int two = (opt == OR_ADAM || opt == OR_ADAMW || opt == OR_LAMB);
    step_scalars s = make_scalars(lr, beta1, beta2, eps, wd, step);
    int64_t nb = (n + B - 1) / B;
    int trust_opt = (opt == OR_LAMB || opt == OR_LARS);
    float lr_r = 0.0f;
    if (trust_opt) {
        /* the tensor's norms, from the dequantized states, before any update */
        double nw2 = 0.0, nx2 = 0.0;
        for (int64_t e = 0; e < n; ++e) {
            int64_t b = e / B;
            float m = q1[c1[e]] * a1[b];
            float v = two ? q2[c2[e]] * a2[b] : 0.0f;
            trust_norm_terms(opt, &s, w[e], load_grad(g, grad_is_f16, e), m, v, &nw2, &nx2);
        }
        lr_r = trust_lr(opt, &s, nw2, nx2, trust);
    }
    set_threads(nthreads);
#pragma omp parallel
    {
        float *mt = (float *)malloc(sizeof(float) * (size_t)B);
        float *vt = (float *)malloc(sizeof(float) * (size_t)B);
#pragma omp for schedule(static)
        for (int64_t b = 0; b < nb; ++b) {
            int64_t st = b * B, len = (n - st < B) ? n - st : B;
            for (int64_t i = 0; i < len; ++i) {
                int64_t e = st + i;
                float m = q1[c1[e]] * a1[b];
                float v = two ? q2[c2[e]] * a2[b] : 0.0f;
                if (trust_opt)
                    trust_update_element(opt, &s, lr_r, &w[e], load_grad(g, grad_is_f16, e), &m,
                                         &v);
                else
                    update_element(opt, &s, &w[e], load_grad(g, grad_is_f16, e), &m, &v);
                mt[i] = m;
                vt[i] = v;
            }
            a1[b] = quantize_block(q1, mt, len, c1 + st, 0);
            if (two)
                a2[b] = quantize_block(q2, vt, len, c2 + st, 0);
        }
        free(mt);
        free(vt);
    }
    return 0;
}

ORACLE_API int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
