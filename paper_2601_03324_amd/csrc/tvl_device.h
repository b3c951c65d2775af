// tvl_device.h -- device code shared by the gfx950 (MI355X) kernel families
// of the TVL GEMV path: vector types, weight and x loads, the per-lane
// multiply-accumulate forms, the joint cross-lane reduction, the direct-x row
// streamer and the direct-x tile of one item (plain GEMV, RMSNorm-fused,
// SwiGLU pair).
//
// y = W x over row-major weights (Kilictas & Alpay, arXiv 2601.03324,
// Sec. 6.1).  A GEMV moves |W| + |x| + |y| bytes for 2|W| flops (Sec. 3.1):
// 0.5 flop per byte at fp32, far below the fp32 vector ridge of MI355X, so
// these kernels are built around HBM streaming, not arithmetic:
//
//   * every weight byte is read exactly once, with 16-byte per-lane loads
//     (one wavefront load = 1 KB contiguous = 8 full 128-byte lines, the
//     GPU form of the paper's "one vector load touches one cache line",
//     Sec. 3.2); rows start on 128-byte boundaries (TVL layout);
//   * x is either staged once per workgroup in LDS (tvl_gemv.hip) or read
//     by each wavefront next to its weights, and every x vector a lane holds
//     is reused for the R rows of its wavefront;
//   * each lane keeps 4 independent fp32 accumulators per row (the paper's
//     four-accumulator ILP, Sec. 11.1) and U loads per row in flight, so a
//     wavefront has R*U KB of weights outstanding;
//   * a wavefront reduces its R rows jointly: R values per lane are halved
//     across lanes in log2(R) exchange steps, then summed over the rest (the
//     horizontal add at the end of the GEMV listing, Sec. 6.1, done across
//     64 lanes); the order is fixed, so results are bitwise reproducible.
//
// No MFMA: a GEMV is not a dense contraction.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvl_internal.h"

namespace tvl {
namespace {

typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

template <typename T>
struct Vec;
template <>
struct Vec<float> {
    using type = f4;
    static constexpr int N = 4;
};
template <>
struct Vec<_Float16> {
    using type = h8;
    static constexpr int N = 8;
};

// Global (address space 1) pointers: the weights and x arrive as generic
// pointers inside descriptors, and a generic access would compile to a flat
// load, which shares its wait counter with LDS reads and serialises the
// stream.  A global load keeps its own in-order counter.
#define TVL_GLOBAL __attribute__((address_space(1)))

// Weights are streamed with non-temporal loads: every byte is used once, and
// on MI355X these read ~13% faster than default-policy loads.
template <typename T>
__device__ __forceinline__ typename Vec<T>::type load_w(const T *p)
{
    using V = typename Vec<T>::type;
    return __builtin_nontemporal_load((const TVL_GLOBAL V *)(p));
}

// x is read by every wavefront of a matrix: default (cached) policy.
__device__ __forceinline__ f4 load_x4(const float *p)
{
    return *(const TVL_GLOBAL f4 *)(p);
}

__device__ __forceinline__ void fma4(f4 &a, const f4 w, const f4 x)
{
    a.x = __builtin_fmaf(w.x, x.x, a.x);
    a.y = __builtin_fmaf(w.y, x.y, a.y);
    a.z = __builtin_fmaf(w.z, x.z, a.z);
    a.w = __builtin_fmaf(w.w, x.w, a.w);
}

// One 16-byte weight vector times its x values from LDS.
// fp32: vector v holds columns 4v..4v+3, x at xs4[v].
// fp16: vector v holds columns 8v..8v+7; LDS keeps x in two planes so that
//       both reads are unit-stride across lanes: xs4[v] = 8v..8v+3 and
//       xs4[plane + v] = 8v+4..8v+7.  The conversion is exact.
__device__ __forceinline__ void mac(f4 &a, const f4 w, const f4 *xs4, int v, int)
{
    fma4(a, w, xs4[v]);
}
__device__ __forceinline__ void mac(f4 &a, const h8 w, const f4 *xs4, int v, int plane)
{
    const f8 wf = __builtin_convertvector(w, f8);
    const f4 lo = {wf[0], wf[1], wf[2], wf[3]};
    const f4 hi = {wf[4], wf[5], wf[6], wf[7]};
    fma4(a, lo, xs4[v]);
    fma4(a, hi, xs4[plane + v]);
}

// The same products with x already in registers (direct-x mode).
__device__ __forceinline__ void mac_x(f4 &a, const f4 w, const f4 xa, const f4)
{
    fma4(a, w, xa);
}
__device__ __forceinline__ void mac_x(f4 &a, const h8 w, const f4 xa, const f4 xb)
{
    const f8 wf = __builtin_convertvector(w, f8);
    const f4 lo = {wf[0], wf[1], wf[2], wf[3]};
    const f4 hi = {wf[4], wf[5], wf[6], wf[7]};
    fma4(a, lo, xa);
    fma4(a, hi, xb);
}

// Two accumulators per (row, vector) for the several-vector kernel: half
// the registers of four, and each still sums only K/128 products.
__device__ __forceinline__ void mac2(f2 &a, const f4 w, const f4 xa, const f4)
{
    a.x = __builtin_fmaf(w.x, xa.x, a.x);
    a.y = __builtin_fmaf(w.y, xa.y, a.y);
    a.x = __builtin_fmaf(w.z, xa.z, a.x);
    a.y = __builtin_fmaf(w.w, xa.w, a.y);
}
__device__ __forceinline__ void mac2(f2 &a, const h8 w, const f4 xa, const f4 xb)
{
    const f8 wf = __builtin_convertvector(w, f8);
    a.x = __builtin_fmaf(wf[0], xa.x, a.x);
    a.y = __builtin_fmaf(wf[1], xa.y, a.y);
    a.x = __builtin_fmaf(wf[2], xa.z, a.x);
    a.y = __builtin_fmaf(wf[3], xa.w, a.y);
    a.x = __builtin_fmaf(wf[4], xb.x, a.x);
    a.y = __builtin_fmaf(wf[5], xb.y, a.y);
    a.x = __builtin_fmaf(wf[6], xb.z, a.x);
    a.y = __builtin_fmaf(wf[7], xb.w, a.y);
}

template <typename V, int N>
__device__ __forceinline__ V mask_from(V w, int valid)
{
#pragma unroll
    for (int e = 0; e < N; ++e)
        if (e >= valid) w[e] = 0;
    return w;
}
// Row results: plain stores for y; for K-split partials, agent-scope
// (device-coherent) stores, which bypass the XCD-local L2 so that the
// workgroup that combines them, on any XCD, reads what was written.
template <bool COHERENT>
__device__ __forceinline__ void store_out(float *p, float v)
{
    if constexpr (COHERENT)
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        *p = v;
}

// Exchange step of the joint reduction: lanes with bit O set keep the upper
// H values, the others the lower H, each adding its partner's copy.
template <int H, int O>
__device__ __forceinline__ void halve(float *v, int lane)
{
    const bool up = (lane & O) != 0;
#pragma unroll
    for (int i = 0; i < H; ++i) {
        const float send = up ? v[i] : v[i + H];
        const float keep = up ? v[i + H] : v[i];
        v[i] = keep + __shfl_xor(send, O);
    }
}

// Apply the exchange steps for N values: offsets 32, 16, ... (log2 N steps).
template <int N, int O>
__device__ __forceinline__ void halve_all(float *v, int lane)
{
    if constexpr (N > 1) {
        halve<N / 2, O>(v, lane);
        halve_all<N / 2, O / 2>(v, lane);
    }
}

// Reduce N values per lane over the wavefront (N a power of two <= 64).  On
// return every lane holds the total of value lane / (64 / N).
template <int N>
__device__ __forceinline__ float reduce_vals(float *v, int lane)
{
    static_assert(N >= 1 && N <= 64 && (N & (N - 1)) == 0, "N must be a power of two <= 64");
    halve_all<N, 32>(v, lane);
#pragma unroll
    for (int o = 32 / N; o >= 1; o >>= 1)
        v[0] += __shfl_xor(v[0], o);
    return v[0];
}

// Reduce R rows of per-lane float4 partials over the wavefront.  On return
// every lane holds the total of row lane / (64 / R).
template <int R>
__device__ __forceinline__ float reduce_rows(const f4 (&acc)[R], int lane)
{
    float v[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        v[r] = (acc[r].x + acc[r].y) + (acc[r].z + acc[r].w);
    return reduce_vals<R>(v, lane);
}
// Direct-x mode: each wavefront reads its x vectors straight from global
// memory (cached: every wavefront of the matrix reads the same x) together
// with the weights.  No LDS, no barrier: wavefronts are independent, so none
// waits for a staging round trip before its first weight load.
//
// NORM (fused RMSNorm, Sec. 2.1 / Sec. 11.2 listing): the RMSNorm weight g is
// read next to x, the products use x*g, and each lane also accumulates x^2
// over its columns.  The scalar 1/sqrt(mean(x^2) + eps) factors out of the
// dot product, so it is applied to the row sums at the end: the normalised
// vector is never materialised and the fusion costs no extra pass over x.
template <typename T, int R, int U, bool NORM = false>
struct DirectRows {
    using V = typename Vec<T>::type;
    static constexpr int N = Vec<T>::N;
    static constexpr int CH = kWave * N;
    const T *rows[R];
    const float *xl; // x at this lane's first column
    const float *gl; // RMSNorm weight at this lane's first column (NORM)
    int kn, nv, nfull;

    __device__ __forceinline__ DirectRows(const T *w0, int64_t ldw, int nrows, const float *x,
                                          int kn_, int lane, const float *g = nullptr)
        : xl(x + lane * N), gl(g + lane * N), kn(kn_), nv((kn_ + N - 1) / N), nfull(kn_ / CH)
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            rows[r] = w0 + (int64_t)(r < nrows ? r : nrows - 1) * ldw + lane * N;
    }
    // explicit row starts (column 0 of each row, this lane's offset added here)
    __device__ __forceinline__ DirectRows(const T *const (&starts)[R], const float *x, int kn_,
                                          int lane, const float *g = nullptr)
        : xl(x + lane * N), gl(g + lane * N), kn(kn_), nv((kn_ + N - 1) / N), nfull(kn_ / CH)
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            rows[r] = starts[r] + lane * N;
    }

    __device__ __forceinline__ void xg(f4 &xa, f4 &xb, f4 &ssq, const f4 ga, const f4 gb) const
    {
        if constexpr (NORM) {
            fma4(ssq, xa, xa);
            xa *= ga;
            if constexpr (N == 8) {
                fma4(ssq, xb, xb);
                xb *= gb;
            }
        }
    }

    __device__ __forceinline__ void run(f4 (&acc)[R], int lane, f4 &ssq) const
    {
        int c = 0;
        for (; c + U <= nfull; c += U) {
            V w[U][R];
            f4 xa[U], xb[U], ga[U], gb[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                xa[u] = load_x4(xl + (c + u) * CH);
                xb[u] = (N == 8) ? load_x4(xl + (c + u) * CH + 4) : xa[u];
                if constexpr (NORM) {
                    ga[u] = load_x4(gl + (c + u) * CH);
                    gb[u] = (N == 8) ? load_x4(gl + (c + u) * CH + 4) : ga[u];
                }
#pragma unroll
                for (int r = 0; r < R; ++r)
                    w[u][r] = load_w<T>(rows[r] + (c + u) * CH);
            }
            __builtin_amdgcn_sched_barrier(0); // all loads of the batch first
#pragma unroll
            for (int u = 0; u < U; ++u) {
                xg(xa[u], xb[u], ssq, ga[u], gb[u]);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    mac_x(acc[r], w[u][r], xa[u], xb[u]);
            }
        }
        for (; c < nfull; ++c) {
            V w[R];
            f4 xa = load_x4(xl + c * CH);
            f4 xb = (N == 8) ? load_x4(xl + c * CH + 4) : xa;
            f4 ga = xa, gb = xb;
            if constexpr (NORM) {
                ga = load_x4(gl + c * CH);
                gb = (N == 8) ? load_x4(gl + c * CH + 4) : ga;
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
                w[r] = load_w<T>(rows[r] + c * CH);
            xg(xa, xb, ssq, ga, gb);
#pragma unroll
            for (int r = 0; r < R; ++r)
                mac_x(acc[r], w[r], xa, xb);
        }
        if (c * kWave < nv) { // ragged last chunk: mask W, x and g past kn
            const int v = c * kWave + lane;
            if (v < nv) {
                const int valid = kn - v * N; // >= 1
                // an f4 of x (or g) is read only when it starts before kn; it
                // then lies in the same 16-byte block as a valid element
                f4 xa = mask_from<f4, 4>(load_x4(xl + c * CH), valid);
                f4 xb = xa, ga = xa, gb = xa;
                if constexpr (N == 8) {
                    xb = f4{0.f, 0.f, 0.f, 0.f};
                    if (valid > 4) xb = mask_from<f4, 4>(load_x4(xl + c * CH + 4), valid - 4);
                }
                if constexpr (NORM) {
                    ga = mask_from<f4, 4>(load_x4(gl + c * CH), valid);
                    gb = ga;
                    if constexpr (N == 8) {
                        gb = f4{0.f, 0.f, 0.f, 0.f};
                        if (valid > 4) gb = mask_from<f4, 4>(load_x4(gl + c * CH + 4), valid - 4);
                    }
                }
                V w[R];
#pragma unroll
                for (int r = 0; r < R; ++r)
                    w[r] = mask_from<V, N>(load_w<T>(rows[r] + c * CH), valid);
                xg(xa, xb, ssq, ga, gb);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    mac_x(acc[r], w[r], xa, xb);
            }
        }
    }
    __device__ __forceinline__ void run(f4 (&acc)[R], int lane) const
    {
        f4 unused = {0.f, 0.f, 0.f, 0.f};
        run(acc, lane, unused);
    }
};

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v += __shfl_xor(v, o);
    return v;
}

// silu(z) = z / (1 + e^-z) (the SwiGLU gate of the FFN, Sec. 2.1), fp32 with
// the accurate expf; z -> -inf gives -0, NaN stays NaN.
__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// One row tile of any item (GEMV or SwiGLU, with or without RMSNorm),
// direct-x.  A wavefront streams R weight rows: R output rows of a GEMV, or
// R/2 output rows of a SwiGLU item (R/2 rows of W1 and the same rows of W3;
// the pairs meet across lane halves after the joint reduction).
template <typename T, int R, int WV, int U, bool NORM, bool SWIGLU>
__device__ __forceinline__ void tile_fused(const DevItem &it, int row0)
{
    constexpr int RO = SWIGLU ? R / 2 : R; // output rows per wavefront
    static_assert(!SWIGLU || (R % 2 == 0), "SwiGLU pairs rows across lane halves");
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * RO;
    const int nrows = it.M - wrow0;
    if (nrows <= 0) return;
    const int nv = min(nrows, RO);
    const T *W = static_cast<const T *>(it.W);
    const T *W3 = static_cast<const T *>(it.W3);
    const T *starts[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int rr = r % RO;
        const T *base = (SWIGLU && r >= RO) ? W3 : W;
        starts[r] = base + (int64_t)(wrow0 + (rr < nv ? rr : nv - 1)) * it.ldw;
    }
    f4 acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = f4{0.f, 0.f, 0.f, 0.f};
    f4 ssq = {0.f, 0.f, 0.f, 0.f};
    const DirectRows<T, R, U, NORM> dr(starts, it.x, it.K, lane, it.g);
    dr.run(acc, lane, ssq);
    float v = reduce_rows<R>(acc, lane);
    if constexpr (NORM) {
        const float ss = wave_sum((ssq.x + ssq.y) + (ssq.z + ssq.w));
        const float inv = 1.0f / sqrtf(ss / (float)it.K + it.eps);
        v *= inv;
    }
    constexpr int G = kWave / R;
    if constexpr (SWIGLU) {
        const float b = __shfl_xor(v, 32); // row r + R/2 (W3) meets row r (W1)
        if (lane < 32 && (lane % G) == 0) {
            const int row = wrow0 + lane / G;
            if (row < it.M) it.y[row] = silu(v) * b;
        }
    } else {
        if ((lane % G) == 0) {
            const int row = wrow0 + lane / G;
            if (row < it.M) it.y[row] = v;
        }
    }
}

template <typename T, int R, int WV, int U>
__device__ __forceinline__ void tile_any(const DevItem &it, int row0)
{
    const bool norm = it.g != nullptr;
    if (it.op == kOpSwiglu) {
        if constexpr (R % 2 == 0) {
            if (norm)
                tile_fused<T, R, WV, U, true, true>(it, row0);
            else
                tile_fused<T, R, WV, U, false, true>(it, row0);
        }
    } else {
        if (norm)
            tile_fused<T, R, WV, U, true, false>(it, row0);
        else
            tile_fused<T, R, WV, U, false, false>(it, row0);
    }
}

// Output rows one tile of `it` covers.
template <int R, int WV>
__host__ __device__ __forceinline__ int tile_rows(int op)
{
    return (op == kOpSwiglu ? R / 2 : R) * WV;
}

}  // namespace
}  // namespace tvl
