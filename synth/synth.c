/*
 * synth.c -- seeded, counter-based synthetic input generator.
 *
 * Serves both the oracle side and the HIP side with identical inputs.  It
 * holds none of the GEMV arithmetic: it only draws numbers and rounds them to
 * the storage types (fp32, binary16, block-quantised 8/4-bit codes).
 *
 * Generator: SplitMix64 (G. L. Steele, D. Lea, C. H. Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  The k-th output (k >= 0) of
 * the sequence seeded with s is mix(s + (k+1) * gamma), gamma = 0x9E3779B97F4A7C15,
 * with the published 64-bit finaliser "mix".  Because each output is a pure
 * function of (s, k), any element (e.g. one matrix row) can be regenerated on
 * its own, and the output does not depend on the thread count.
 *
 *   uniform u in [0,1):  top 53 bits * 2^-53
 *   U(a,b):              a + (b-a)*u in double, rounded to fp32 (RNE)
 *   N(0, sigma^2):       Box-Muller (G. E. P. Box, M. E. Muller, 1958) on the
 *                        pair (2p, 2p+1): u1 in (0,1], u2 in [0,1);
 *                        element 2p = sigma*r*cos(2 pi u2),
 *                        element 2p+1 = sigma*r*sin(2 pi u2), r = sqrt(-2 ln u1),
 *                        computed in double, rounded to fp32 (RNE)
 *   binary16 weights:    the fp32 value above, rounded to binary16 with
 *                        round-to-nearest-even (what a cast of an fp32 tensor
 *                        to fp16 does)
 *
 * Build: gcc -std=c99 -O2 -fopenmp -fPIC -shared.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define SM64_GAMMA 0x9E3779B97F4A7C15ULL
#define TWO_M53 (1.0 / 9007199254740992.0) /* 2^-53 */
#define TWO_PI 6.283185307179586476925286766559

static inline uint64_t sm64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* k-th output of the SplitMix64 sequence seeded with s. */
uint64_t synth_u64(uint64_t s, uint64_t k)
{
    return sm64_mix(s + (k + 1) * SM64_GAMMA);
}

/* Stream key from a root seed and a tuple of small integers
 * (e.g. config, layer, matrix id, kind, repetition): a chain of SplitMix64
 * steps, one per field. */
uint64_t synth_key(uint64_t root, const uint64_t *fields, int n)
{
    uint64_t h = sm64_mix(root + SM64_GAMMA);
    for (int i = 0; i < n; ++i)
        h = sm64_mix(h + (fields[i] + 1) * SM64_GAMMA);
    return h;
}

static inline double u53(uint64_t v) { return (double)(v >> 11) * TWO_M53; }

static inline double normal_at(uint64_t key, uint64_t idx)
{
    const uint64_t p = idx >> 1;
    const double u1 = ((double)(synth_u64(key, 2 * p) >> 11) + 1.0) * TWO_M53; /* (0,1] */
    const double u2 = u53(synth_u64(key, 2 * p + 1));                        /* [0,1) */
    const double r = sqrt(-2.0 * log(u1));
    return (idx & 1) ? r * sin(TWO_PI * u2) : r * cos(TWO_PI * u2);
}

/* fp32 -> binary16 bits, round to nearest, ties to even. */
uint16_t synth_f32_to_f16_bits(float f)
{
    uint32_t x;
    memcpy(&x, &f, 4);
    const uint32_t sign = (x >> 16) & 0x8000u;
    const uint32_t a = x & 0x7fffffffu;
    if (a >= 0x7f800000u) /* Inf or NaN (NaN keeps a quiet payload bit) */
        return (uint16_t)(sign | (a > 0x7f800000u ? 0x7e00u : 0x7c00u));
    if (a >= 0x477ff000u) /* >= 65520: rounds to Inf */
        return (uint16_t)(sign | 0x7c00u);
    if (a < 0x38800000u) { /* |f| < 2^-14: binary16 subnormal or zero */
        const uint32_t e = a >> 23;
        if (e < 102) /* |f| < 2^-25: below half the smallest subnormal */
            return (uint16_t)sign;
        const uint32_t m = (a & 0x7fffffu) | 0x800000u;
        const uint32_t shift = 126 - e; /* 14..24: q = m / 2^shift units of 2^-24 */
        uint32_t q = m >> shift;
        const uint32_t rem = m & ((1u << shift) - 1);
        const uint32_t half = 1u << (shift - 1);
        if (rem > half || (rem == half && (q & 1))) ++q;
        return (uint16_t)(sign | q);
    }
    uint32_t h = (a - 0x38000000u) >> 13; /* rebias exponent 127 -> 15 */
    const uint32_t rem = a & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1))) ++h;
    return (uint16_t)(sign | h);
}

void synth_f32_to_f16(const float *in, uint16_t *out, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = synth_f32_to_f16_bits(in[i]);
}

/* out[i] = U(a,b) element (offset + i) of stream key. */
void synth_uniform_f32(float *out, int64_t n, uint64_t key, uint64_t offset,
                       double a, double b)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(a + (b - a) * u53(synth_u64(key, offset + (uint64_t)i)));
}

/* out[i] = N(0, sigma^2) element (offset + i) of stream key, as fp32. */
void synth_normal_f32(float *out, int64_t n, uint64_t key, uint64_t offset,
                      double sigma)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(sigma * normal_at(key, offset + (uint64_t)i));
}

/* Same values as synth_normal_f32, then rounded to binary16 (RNE). */
void synth_normal_f16(uint16_t *out, int64_t n, uint64_t key, uint64_t offset,
                      double sigma)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = synth_f32_to_f16_bits((float)(sigma * normal_at(key, offset + (uint64_t)i)));
}

/* Integers uniform in [lo, hi], stored as fp32 (for exact-arithmetic cases). */
void synth_int_f32(float *out, int64_t n, uint64_t key, uint64_t offset,
                   int64_t lo, int64_t hi)
{
    const uint64_t span = (uint64_t)(hi - lo + 1);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(lo + (int64_t)(synth_u64(key, offset + (uint64_t)i) % span));
}

/* Same, as binary16 bit patterns (exact for |v| <= 2048). */
void synth_int_f16(uint16_t *out, int64_t n, uint64_t key, uint64_t offset,
                   int64_t lo, int64_t hi)
{
    const uint64_t span = (uint64_t)(hi - lo + 1);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = synth_f32_to_f16_bits(
            (float)(lo + (int64_t)(synth_u64(key, offset + (uint64_t)i) % span)));
}

/* ------------------------------------------------------------------------ */
/* Block quantisation of an fp32 matrix into the quantised format (a code   */
/* plane of M rows x ldw bytes, then the fp32 scale plane in blocks of 4   */
/* rows: group g of row i at (i/4)*4*ng + 4*g + i%4; see the library        */
/* header).                                                                 */
/* Symmetric: 8-bit s = max|w| / 127, q = round(w / s) in [-127, 127];      */
/* 4-bit s = max|w| / 7, q in [-7, 7].                                      */
/* codes stored in two's complement.  An all-zero group gets s = 0, q = 0.  */
/* Padding bytes of the code rows keep what the caller put in `out`.        */
/* ------------------------------------------------------------------------ */
int64_t synth_q_row_bytes(int64_t K, int bits)
{
    const int64_t b = (K * bits + 7) / 8;
    return (b + 127) / 128 * 128;
}

void synth_quantize_rows(const float *w, int64_t M, int64_t K, int bits, uint8_t *out,
                         int64_t ldw)
{
    const int64_t ng = (K + 63) / 64, Mp = (M + 3) / 4 * 4;
    const int qmax = bits == 8 ? 127 : 7;
    float *plane = (float *)(out + M * ldw);
    for (int64_t g = 0; g < ng; ++g) /* scale padding rows M .. Mp-1 */
        for (int64_t i = M; i < Mp; ++i)
            plane[(i / 4) * 4 * ng + 4 * g + i % 4] = 0.f;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < M; ++i) {
        const float *src = w + i * K;
        uint8_t *row = out + i * ldw;
        for (int64_t g = 0; g < ng; ++g) {
            const int64_t j0 = g * 64, j1 = (j0 + 64 < K) ? j0 + 64 : K;
            float amax = 0.f;
            for (int64_t j = j0; j < j1; ++j)
                amax = fabsf(src[j]) > amax ? fabsf(src[j]) : amax;
            const float s = amax / (float)qmax;
            plane[(i / 4) * 4 * ng + 4 * g + i % 4] = s;
            for (int64_t j = j0; j < j1; ++j) {
                int q = 0;
                if (s > 0.f) {
                    q = (int)lrintf(src[j] / s);
                    q = q > qmax ? qmax : (q < -qmax ? -qmax : q);
                }
                if (bits == 8) {
                    row[j] = (uint8_t)(int8_t)q;
                } else {
                    const uint8_t u = (uint8_t)(q & 0x0f);
                    if (j % 2 == 0)
                        row[j / 2] = (uint8_t)((row[j / 2] & 0xf0) | u);
                    else
                        row[j / 2] = (uint8_t)((row[j / 2] & 0x0f) | (u << 4));
                }
            }
        }
    }
}
