/*
 * oracle.c -- the plain CPU oracle for the TVL GEMV path.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load or call this file.  The product path
 * (the HIP library under paper_2601_03324_amd/) never includes, links or calls
 * it, and this file includes no HIP header and no product source.
 *
 * What it computes (Kilictas & Alpay, "Bare-Metal Tensor Virtualization",
 * arXiv 2601.03324):
 *
 *   y = W x, W row-major with row i at W + i*ldw  (Sec. 6.1, the naive loop
 *   y[i] += W[i][j] * x[j] and the GEMV listing xout = W @ x with the weight
 *   for (i, j) at w + i*n + j; Sec. 3.1 Roofline: one product and one add per
 *   weight).
 *
 * The paper's NEON kernel only reorders this sum (Sec. 5.2 says reordered
 * fused multiply-add accumulation drifts from scalar accumulation and that
 * this drift is accepted).  So the oracle is the plain definition, written as
 * the naive loop, in double precision:
 *
 *   - each product w*x of an fp32 (24-bit significand) or fp16 (11-bit) weight
 *     and an fp32 x is exact in double (at most 48 significand bits < 53);
 *   - the only rounding is the sequential double sum over ascending j, so
 *     |acc - exact| <= (K-1) * 2^-53 * S_i, with S_i = sum_j |W_ij x_j|.
 *
 * The oracle also returns S_i, the normaliser of the parity norm
 * err_i = |y_gpu_i - y_ref_i| / S_i (the textbook forward error bound of a
 * dot product is a multiple of S_i).
 *
 * Readings of the paper taken here (each listed in the design notes):
 *   - layout is row-major with a row stride ldw >= K; entries j >= K of a row
 *     are padding and never read;
 *   - the output is overwritten (xout = W @ x), not accumulated into;
 *   - all K terms are included (the printed vector loop has no remainder loop;
 *     the result here is the mathematical one over every column);
 *   - fp16 weights are decoded exactly (binary16 definition, subnormals kept)
 *     and accumulated in double; x stays fp32.
 *
 * Build: gcc -std=c99 -O2 -ffp-contract=off -fPIC -shared (no -ffast-math).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

/* ------------------------------------------------------------------------ */
/* IEEE 754 binary16 -> double, exact (IEEE 754-2008 Sec. 3.4 definition).   */
/* ------------------------------------------------------------------------ */
double oracle_f16_to_f64(uint16_t h)
{
    const int sign = (h >> 15) & 1;
    const int e = (h >> 10) & 0x1f;
    const int m = h & 0x3ff;
    double v;
    if (e == 0) {
        /* zero or subnormal: m * 2^-24 */
        v = ldexp((double)m, -24);
    } else if (e == 31) {
        v = (m == 0) ? INFINITY : NAN;
    } else {
        /* normal: (1 + m/1024) * 2^(e-15) = (1024 + m) * 2^(e-25) */
        v = ldexp((double)(1024 + m), e - 25);
    }
    return sign ? -v : v;
}

/* ------------------------------------------------------------------------ */
/* y_i = sum_{j<K} W[i*ldw + j] * x[j], in double, j ascending (Sec. 6.1).   */
/* S_i = sum_{j<K} |W[i*ldw + j] * x[j]|.  S may be NULL.                    */
/* ------------------------------------------------------------------------ */
void oracle_gemv_f32(const float *W, int64_t ldw, const float *x,
                     int64_t M, int64_t K, double *y, double *S)
{
    for (int64_t i = 0; i < M; ++i) {
        const float *row = W + i * ldw;
        double acc = 0.0, s = 0.0;
        for (int64_t j = 0; j < K; ++j) {
            const double p = (double)row[j] * (double)x[j]; /* exact */
            acc += p;
            s += fabs(p);
        }
        y[i] = acc;
        if (S) S[i] = s;
    }
}

/* Same definition with binary16 weights (bit patterns), fp32 x. */
void oracle_gemv_f16(const uint16_t *W, int64_t ldw, const float *x,
                     int64_t M, int64_t K, double *y, double *S)
{
    for (int64_t i = 0; i < M; ++i) {
        const uint16_t *row = W + i * ldw;
        double acc = 0.0, s = 0.0;
        for (int64_t j = 0; j < K; ++j) {
            const double p = oracle_f16_to_f64(row[j]) * (double)x[j]; /* exact */
            acc += p;
            s += fabs(p);
        }
        y[i] = acc;
        if (S) S[i] = s;
    }
}

/* ------------------------------------------------------------------------ */
/* Parity norm.  err_i = |y_i - ref_i| / S_i; a non-finite y_i, or a nonzero */
/* y_i where S_i == 0 (zero row or zero x), counts as an infinite error.     */
/* Returns the number of outputs with err_i > tol.                           */
/* ------------------------------------------------------------------------ */
int64_t oracle_check(const float *y, const double *ref, const double *S,
                     int64_t M, double tol, double *max_err,
                     int64_t *argmax, double *mean_err)
{
    double worst = 0.0, sum = 0.0;
    int64_t where = -1, bad = 0;
    for (int64_t i = 0; i < M; ++i) {
        const double yi = (double)y[i];
        double e;
        if (!isfinite(yi)) {
            e = INFINITY;
        } else if (S[i] == 0.0) {
            e = (yi == 0.0) ? 0.0 : INFINITY;
        } else {
            e = fabs(yi - ref[i]) / S[i];
        }
        if (e > tol) ++bad;
        if (where < 0 || e > worst) {
            worst = e;
            where = i;
        }
        sum += e;
    }
    if (max_err) *max_err = worst;
    if (argmax) *argmax = where;
    if (mean_err) *mean_err = (M > 0) ? sum / (double)M : 0.0;
    return bad;
}

/* ------------------------------------------------------------------------ */
/* RMSNorm (Sec. 2.1: pre-normalisation; Sec. 6.2 and the Sec. 11.2 listing): */
/*   ms = (1/K) sum_j x_j^2 ;  inv = 1 / sqrt(ms + eps) ;  o_j = x_j g_j inv  */
/* in double; epsilon is added to the mean square inside the root, as in the */
/* listing.  Output in double (the GEMV below takes it as its x).            */
/* ------------------------------------------------------------------------ */
void oracle_rmsnorm(const float *x, const float *g, int64_t K, double eps, double *out)
{
    double ss = 0.0;
    for (int64_t j = 0; j < K; ++j)
        ss += (double)x[j] * (double)x[j];
    const double ms = ss / (double)K;
    const double inv = 1.0 / sqrt(ms + eps);
    for (int64_t j = 0; j < K; ++j)
        out[j] = (double)x[j] * (double)g[j] * inv;
}

/* y = W xd with x given in double (e.g. an RMSNorm output), fp32 or binary16
 * weights; same loop as oracle_gemv_f32/_f16.  S_i = sum_j |W_ij xd_j|. */
void oracle_gemv_dx(const void *W, int32_t is_f16, int64_t ldw, const double *xd,
                    int64_t M, int64_t K, double *y, double *S)
{
    for (int64_t i = 0; i < M; ++i) {
        double acc = 0.0, s = 0.0;
        for (int64_t j = 0; j < K; ++j) {
            const double w = is_f16 ? oracle_f16_to_f64(((const uint16_t *)W)[i * ldw + j])
                                    : (double)((const float *)W)[i * ldw + j];
            const double p = w * xd[j];
            acc += p;
            s += fabs(p);
        }
        y[i] = acc;
        if (S) S[i] = s;
    }
}

/* ------------------------------------------------------------------------ */
/* SwiGLU gate (Sec. 2.1: the FFN uses three matrices W1, W2, W3; with the   */
/* gated linear unit of Shazeer, "GLU Variants Improve Transformer", 2020):  */
/*   h_i = silu(a_i) * b_i,  silu(z) = z / (1 + e^-z),                      */
/* where a = W1 xn and b = W3 xn are given (e.g. from oracle_gemv_dx).       */
/* ------------------------------------------------------------------------ */
void oracle_swiglu(const double *a, const double *b, int64_t M, double *h)
{
    for (int64_t i = 0; i < M; ++i)
        h[i] = a[i] / (1.0 + exp(-a[i])) * b[i];
}

/* ------------------------------------------------------------------------ */
/* Block-quantised weights (Sec. 8.2 proposes 4-bit weights unpacked on the  */
/* fly; Sec. 2.2 names 4/8-bit quantisation; the paper fixes no format).     */
/* Format of this library for an M x K matrix:                               */
/*   code plane: M rows of ldw bytes; column j of a row at byte j (8-bit) or */
/*               in nibble j of byte j/2, low nibble first (4-bit);          */
/*   codes are two's complement: q in [-128, 127] (8-bit), [-8, 7] (4-bit);  */
/*   scale plane: right after the code plane (byte M*ldw), fp32, in blocks   */
/*               of 4 rows: s_{i,g} (columns 64g .. 64g+63 of row i) at      */
/*               index (i/4)*4*ng + 4*g + i%4, ng = ceil(K/64) groups, rows  */
/*               padded to Mp = M rounded up to 4 (entries of rows i >= M    */
/*               are padding);                                               */
/*   w_ij = s_{i, j/64} * q_ij.                                              */
/* The products and sums are done exactly as in oracle_gemv_f32, in double.  */
/* ------------------------------------------------------------------------ */
static double q_weight(const uint8_t *W, int64_t ldw, int64_t M, int64_t K, int bits,
                       int64_t i, int64_t j)
{
    const float *scales = (const float *)(W + M * ldw);
    const int64_t ng = (K + 63) / 64;
    const double s = (double)scales[(i / 4) * 4 * ng + 4 * (j / 64) + i % 4];
    const uint8_t *row = W + i * ldw;
    double q;
    if (bits == 8) {
        q = (double)(int8_t)row[j];
    } else {
        const uint8_t byte = row[j / 2];
        const int u = (j % 2 == 0) ? (byte & 0x0f) : (byte >> 4);
        q = (double)(u >= 8 ? u - 16 : u); /* 4-bit two's complement */
    }
    return s * q; /* exact: 24-bit scale times a code of at most 8 bits */
}

void oracle_gemv_q(const uint8_t *W, int32_t bits, int64_t ldw, const float *x,
                   int64_t M, int64_t K, double *y, double *S)
{
    for (int64_t i = 0; i < M; ++i) {
        double acc = 0.0, s = 0.0;
        for (int64_t j = 0; j < K; ++j) {
            const double p = q_weight(W, ldw, M, K, bits, i, j) * (double)x[j];
            acc += p;
            s += fabs(p);
        }
        y[i] = acc;
        if (S) S[i] = s;
    }
}

/* Decoded fp64 weight of row i, column j (for tests). */
double oracle_q_weight(const uint8_t *W, int32_t bits, int64_t ldw, int64_t M, int64_t K,
                       int64_t i, int64_t j)
{
    return q_weight(W, ldw, M, K, bits, i, j);
}
