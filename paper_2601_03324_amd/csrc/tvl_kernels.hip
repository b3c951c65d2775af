// tvl_kernels.hip -- gfx950 (MI355X) kernels of the TVL GEMV path.
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
//   * x is staged once per workgroup in LDS (in slices of up to 8192
//     elements) and each x vector read from LDS is reused for R rows held by
//     the same wavefront;
//   * each lane keeps 4 independent fp32 accumulators per row (the paper's
//     four-accumulator ILP, Sec. 11.1) and U loads per row in flight, so a
//     wavefront has R*U KB of weights outstanding;
//   * a wavefront reduces its R rows jointly: R values per lane are halved
//     across lanes in log2(R) exchange steps, then summed over the rest (the
//     horizontal add at the end of the GEMV listing, Sec. 6.1, done across
//     64 lanes); the order is fixed, so results are bitwise reproducible.
//
// No MFMA: a GEMV is not a dense contraction.
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

// Stage x[0..kn) of the current slice into LDS, zero-filled to a whole
// number of weight vectors (so masked tail products are exactly 0 * 0).
template <typename T>
__device__ __forceinline__ void stage_x(const float *__restrict__ xg, int kn, f4 *__restrict__ xs4,
                                        int plane)
{
    constexpr int N = Vec<T>::N;
    const int nq = (kn + N - 1) / N * (N / 4);
    for (int q = threadIdx.x; q < nq; q += blockDim.x) {
        const int j = q * 4;
        f4 val;
        if (j + 4 <= kn) {
            val = load_x4(xg + j);
        } else {
            val = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (j + e < kn) val[e] = *(const TVL_GLOBAL float *)(xg + j + e);
        }
        if constexpr (N == 4)
            xs4[q] = val;
        else
            xs4[(q & 1) * plane + (q >> 1)] = val;
    }
}

// The weights of one LDS slice for the R rows of one wavefront: columns
// [0, kn) of the slice, streamed in batches of U wavefront loads per row.
// w0 points at column 0 of the slice in the wavefront's first row; rows
// r >= nrows re-read row nrows-1 (their results are discarded).
template <typename T, int R, int U>
struct SliceRows {
    using V = typename Vec<T>::type;
    static constexpr int N = Vec<T>::N;
    static constexpr int CH = kWave * N; // elements per wavefront load
    const T *rows[R];
    int kn, nv, nfull;

    __device__ __forceinline__ SliceRows(const T *w0, int64_t ldw, int nrows, int kn_, int lane)
        : kn(kn_), nv((kn_ + N - 1) / N), nfull(kn_ / CH)
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            rows[r] = w0 + (int64_t)(r < nrows ? r : nrows - 1) * ldw + lane * N;
    }

    // issue the loads of chunks c .. c+U-1 (all full)
    __device__ __forceinline__ void load(V (&w)[U][R], int c) const
    {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r)
                w[u][r] = load_w<T>(rows[r] + (c + u) * CH);
    }

    __device__ __forceinline__ void mac_batch(const V (&w)[U][R], int c, const f4 *xs4, int plane,
                                              int lane, f4 (&acc)[R]) const
    {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r)
                mac(acc[r], w[u][r], xs4, (c + u) * kWave + lane, plane);
    }

    // chunks c .. end of the slice: whole batches, single chunks, then the
    // ragged last chunk (elements past kn masked to zero)
    __device__ __forceinline__ void run_from(int c, const f4 *xs4, int plane, int lane,
                                             f4 (&acc)[R]) const
    {
        for (; c + U <= nfull; c += U) {
            V w[U][R];
            load(w, c);
            // keep all U*R loads ahead of the first multiply: left alone, the
            // scheduler interleaves them with the FMAs to save registers and
            // only two or three loads stay in flight
            __builtin_amdgcn_sched_barrier(0);
            mac_batch(w, c, xs4, plane, lane, acc);
        }
        for (; c < nfull; ++c) {
            V w[R];
#pragma unroll
            for (int r = 0; r < R; ++r)
                w[r] = load_w<T>(rows[r] + c * CH);
#pragma unroll
            for (int r = 0; r < R; ++r)
                mac(acc[r], w[r], xs4, c * kWave + lane, plane);
        }
        if (c * kWave < nv) {
            const int v = c * kWave + lane;
            if (v < nv) {
                const int valid = kn - v * N;
                V w[R];
#pragma unroll
                for (int r = 0; r < R; ++r)
                    w[r] = load_w<T>(rows[r] + c * CH);
                if (valid < N) {
#pragma unroll
                    for (int r = 0; r < R; ++r)
                        w[r] = mask_from<V, N>(w[r], valid);
                }
#pragma unroll
                for (int r = 0; r < R; ++r)
                    mac(acc[r], w[r], xs4, v, plane);
            }
        }
    }
};

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

// One row tile, x staged in LDS: WV wavefronts x R rows, columns
// [kbeg, kend).  out[row] gets the tile's sum for each row < M.
template <typename T, int R, int WV, int U, bool COHERENT = false>
__device__ __forceinline__ void gemv_tile(const T *__restrict__ W, int64_t ldw,
                                          const float *__restrict__ x, int M, int row0, int kbeg,
                                          int kend, int ks_cap, f4 *__restrict__ xs4,
                                          float *__restrict__ out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * R;
    const int nrows = M - wrow0;
    const int plane = ks_cap / 8;
    f4 acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = f4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = kbeg; k0 < kend; k0 += ks_cap) {
        const int kn = min(ks_cap, kend - k0);
        __syncthreads(); // the previous slice (or tile) is no longer read
        stage_x<T>(x + k0, kn, xs4, plane);
        __syncthreads();
        if (nrows > 0) {
            const SliceRows<T, R, U> sr(W + (int64_t)wrow0 * ldw + k0, ldw, min(nrows, R), kn,
                                        lane);
            sr.run_from(0, xs4, plane, lane, acc);
        }
    }
    const float v = reduce_rows<R>(acc, lane);
    constexpr int G = kWave / R;
    if (nrows > 0 && (lane % G) == 0) {
        const int row = wrow0 + lane / G;
        if (row < M) store_out<COHERENT>(out + row, v);
    }
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

template <typename T, int R, int WV, int U, bool COHERENT = false>
__device__ __forceinline__ void gemv_tile_direct(const T *__restrict__ W, int64_t ldw,
                                                 const float *__restrict__ x, int M, int row0,
                                                 int kbeg, int kend, float *__restrict__ out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * R;
    const int nrows = M - wrow0;
    if (nrows <= 0) return; // direct-x tiles have no barrier to reach
    f4 acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = f4{0.f, 0.f, 0.f, 0.f};
    const DirectRows<T, R, U> dr(W + (int64_t)wrow0 * ldw + kbeg, ldw, min(nrows, R), x + kbeg,
                                 kend - kbeg, lane);
    dr.run(acc, lane);
    const float v = reduce_rows<R>(acc, lane);
    constexpr int G = kWave / R;
    if ((lane % G) == 0) {
        const int row = wrow0 + lane / G;
        if (row < M) store_out<COHERENT>(out + row, v);
    }
}

// ---------------------------------------------------------------- kernels
template <typename T, int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_gemv_rows(const T *__restrict__ W, int64_t ldw,
                                                          const float *__restrict__ x,
                                                          float *__restrict__ y, int M, int K,
                                                          int ks_cap)
{
    extern __shared__ f4 smem4[];
    gemv_tile<T, R, WV, U>(W, ldw, x, M, (int)blockIdx.x * (R * WV), 0, K, ks_cap, smem4, y);
}

template <typename T, int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_gemv_rows_direct(const T *__restrict__ W,
                                                                 int64_t ldw,
                                                                 const float *__restrict__ x,
                                                                 float *__restrict__ y, int M,
                                                                 int K)
{
    gemv_tile_direct<T, R, WV, U>(W, ldw, x, M, (int)blockIdx.x * (R * WV), 0, K, y);
}

// K split: workgroup b handles row tile b / S and K slice b % S.  Each
// slice's row sums go to partials[split * M + row] with device-coherent
// stores; every thread waits for its stores to be acknowledged, the
// workgroup meets at a barrier, and one thread bumps the tile's counter.  The
// workgroup that brings the counter to S adds the S partials in the order
// 0..S-1 (device-coherent loads) and resets the counter for the next launch.
//
// An agent-scope release/acquire fence would be the textbook way to publish
// the partials, but on a multi-XCD part it compiles to a write-back and an
// invalidation of the whole L2, once per workgroup: measured 20-100x slower
// than the row split.  Coherent stores plus the store wait give the same
// guarantee for exactly the data that needs it.
template <typename T, int R, int WV, int U, int XM>
__global__ __launch_bounds__(WV *kWave) void k_gemv_ksplit(
    const T *__restrict__ W, int64_t ldw, const float *__restrict__ x, float *__restrict__ y,
    int M, int K, int ks_cap, int S, int kspan, float *__restrict__ partials,
    int *__restrict__ counters)
{
    extern __shared__ f4 smem4[];
    __shared__ int is_last;
    const int tile = (int)blockIdx.x / S;
    const int split = (int)blockIdx.x - tile * S;
    const int row0 = tile * (R * WV);
    const int kbeg = split * kspan;
    const int kend = min(K, kbeg + kspan);
    if constexpr (XM == kXLds)
        gemv_tile<T, R, WV, U, true>(W, ldw, x, M, row0, kbeg, kend, ks_cap, smem4,
                                     partials + (int64_t)split * M);
    else
        gemv_tile_direct<T, R, WV, U, true>(W, ldw, x, M, row0, kbeg, kend,
                                            partials + (int64_t)split * M);
    __builtin_amdgcn_s_waitcnt(0x0F70); // this thread's partial stores acknowledged
    __syncthreads();
    if (threadIdx.x == 0) {
        const int prev =
            __hip_atomic_fetch_add(counters + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        is_last = (prev == S - 1);
    }
    __syncthreads();
    if (is_last) {
        const int rows = min(R * WV, M - row0);
        for (int r = threadIdx.x; r < rows; r += blockDim.x) {
            float s = 0.f;
            for (int p = 0; p < S; ++p)
                s += __hip_atomic_load(partials + (int64_t)p * M + row0 + r, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            y[row0 + r] = s;
        }
        if (threadIdx.x == 0)
            __hip_atomic_store(counters + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Grouped sweep: every GEMV of a decode token in one launch.  Workgroup b
// takes tiles b, b + grid, ... of the plan's tile table (grid = number of
// tiles gives one tile per workgroup and leaves the balancing to the
// hardware dispatcher).
template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_sweep(const DevItem *__restrict__ items,
                                                      const DevTile *__restrict__ tiles,
                                                      int ntiles, int ks_cap)
{
    extern __shared__ f4 smem4[];
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        if (it.dtype == 1)
            gemv_tile<_Float16, R, WV, U>(static_cast<const _Float16 *>(it.W), it.ldw, it.x, it.M,
                                          tl.row0, 0, it.K, ks_cap, smem4, it.y);
        else
            gemv_tile<float, R, WV, U>(static_cast<const float *>(it.W), it.ldw, it.x, it.M,
                                       tl.row0, 0, it.K, ks_cap, smem4, it.y);
        // Drain this tile's y stores before the next tile's loads.  With a
        // store still counted, the compiler's wait-count tracking treats the
        // memory counter as out of order and waits for *all* loads before
        // the first multiply of every chunk (vmcnt field 0; expcnt and
        // lgkmcnt fields at their maxima, i.e. not waited on).
        __builtin_amdgcn_s_waitcnt(0x0F70);
    }
}

template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_sweep_direct(const DevItem *__restrict__ items,
                                                             const DevTile *__restrict__ tiles,
                                                             int ntiles)
{
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        if (it.dtype == 1)
            gemv_tile_direct<_Float16, R, WV, U>(static_cast<const _Float16 *>(it.W), it.ldw,
                                                 it.x, it.M, tl.row0, 0, it.K, it.y);
        else
            gemv_tile_direct<float, R, WV, U>(static_cast<const float *>(it.W), it.ldw, it.x,
                                              it.M, tl.row0, 0, it.K, it.y);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

// Several x vectors against the same weights (beam search with B
// hypotheses, Sec. 9.1: each extra hypothesis would otherwise stream every
// weight again).  Y[b][i] = sum_j W_ij X[b][j] for b < nb <= B: the weights
// are loaded once per wavefront and multiplied into R x B accumulators; the
// x vectors come straight from global memory (L1/L2-cached).  Vectors
// b >= nb re-read vector 0 and their results are dropped.
template <typename T, int R, int U, int B>
struct MultiRows {
    using V = typename Vec<T>::type;
    static constexpr int N = Vec<T>::N;
    static constexpr int CH = kWave * N;
    const T *rows[R];
    const float *xl[B]; // vector b at this lane's first column
    int kn, nv, nfull;

    __device__ __forceinline__ MultiRows(const T *w0, int64_t ldw, int nrows, const float *x,
                                         int64_t ldx, int nb, int kn_, int lane)
        : kn(kn_), nv((kn_ + N - 1) / N), nfull(kn_ / CH)
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            rows[r] = w0 + (int64_t)(r < nrows ? r : nrows - 1) * ldw + lane * N;
#pragma unroll
        for (int b = 0; b < B; ++b)
            xl[b] = x + (int64_t)(b < nb ? b : 0) * ldx + lane * N;
    }

    __device__ __forceinline__ void run(f2 (&acc)[R][B], int lane) const
    {
        int c = 0;
        for (; c + U <= nfull; c += U) {
            V w[U][R];
            f4 xa[U][B], xb[U][B];
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    w[u][r] = load_w<T>(rows[r] + (c + u) * CH);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    xa[u][b] = load_x4(xl[b] + (c + u) * CH);
                    xb[u][b] = (N == 8) ? load_x4(xl[b] + (c + u) * CH + 4) : xa[u][b];
                }
            }
            __builtin_amdgcn_sched_barrier(0); // all loads of the batch first
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int r = 0; r < R; ++r)
#pragma unroll
                    for (int b = 0; b < B; ++b)
                        mac2(acc[r][b], w[u][r], xa[u][b], xb[u][b]);
        }
        for (; c < nfull; ++c) {
            V w[R];
            f4 xa[B], xb[B];
#pragma unroll
            for (int r = 0; r < R; ++r)
                w[r] = load_w<T>(rows[r] + c * CH);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                xa[b] = load_x4(xl[b] + c * CH);
                xb[b] = (N == 8) ? load_x4(xl[b] + c * CH + 4) : xa[b];
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int b = 0; b < B; ++b)
                    mac2(acc[r][b], w[r], xa[b], xb[b]);
        }
        if (c * kWave < nv) { // ragged last chunk: mask W and x past kn
            const int v = c * kWave + lane;
            if (v < nv) {
                const int valid = kn - v * N;
                V w[R];
                f4 xa[B], xb[B];
#pragma unroll
                for (int r = 0; r < R; ++r)
                    w[r] = mask_from<V, N>(load_w<T>(rows[r] + c * CH), valid);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    xa[b] = mask_from<f4, 4>(load_x4(xl[b] + c * CH), valid);
                    xb[b] = xa[b];
                    if constexpr (N == 8) {
                        xb[b] = f4{0.f, 0.f, 0.f, 0.f};
                        if (valid > 4)
                            xb[b] = mask_from<f4, 4>(load_x4(xl[b] + c * CH + 4), valid - 4);
                    }
                }
#pragma unroll
                for (int r = 0; r < R; ++r)
#pragma unroll
                    for (int b = 0; b < B; ++b)
                        mac2(acc[r][b], w[r], xa[b], xb[b]);
            }
        }
    }
};

template <typename T, int R, int WV, int U, int B>
__device__ __forceinline__ void tile_multi(const DevItem &it, int row0)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * R;
    const int nrows = it.M - wrow0;
    if (nrows <= 0) return;
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f2 acc[R][B];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < B; ++b)
            acc[r][b] = f2{0.f, 0.f};
    const MultiRows<T, R, U, B> mr(static_cast<const T *>(it.W) + (int64_t)wrow0 * it.ldw, it.ldw,
                                   min(nrows, R), it.x, it.ldx, nb, it.K, lane);
    mr.run(acc, lane);
    float v[R * B];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int b = 0; b < B; ++b)
            v[r * B + b] = acc[r][b].x + acc[r][b].y;
    const float t = reduce_vals<R * B>(v, lane);
    constexpr int G = kWave / (R * B);
    if ((lane % G) == 0) {
        const int q = lane / G;
        const int r = q / B, b = q % B;
        const int row = wrow0 + r;
        if (b < nb && r < nrows) it.y[(int64_t)b * it.ldy + row] = t;
    }
}

template <int R, int WV, int U, int B>
__global__ __launch_bounds__(WV *kWave) void k_sweep_multi(const DevItem *__restrict__ items,
                                                            const DevTile *__restrict__ tiles,
                                                            int ntiles)
{
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        if (it.dtype == 1)
            tile_multi<_Float16, R, WV, U, B>(it, tl.row0);
        else
            tile_multi<float, R, WV, U, B>(it, tl.row0);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int R, int WV, int U, int B>
__global__ __launch_bounds__(WV *kWave) void k_item_multi(const DevItem it)
{
    const int row0 = (int)blockIdx.x * (R * WV);
    if (it.dtype == 1)
        tile_multi<_Float16, R, WV, U, B>(it, row0);
    else
        tile_multi<float, R, WV, U, B>(it, row0);
}

// Block-quantised weights (8- or 4-bit two's-complement codes in M rows of
// ldw bytes; fp32 scale per 64 columns in a row-major plane after the code
// rows).  A 16-byte load brings N = 16 (8-bit) or 32 (4-bit) codes of one
// row, all in one 64-column scale group, so each load is dotted with x first
// and scaled once.
//
// Decoding costs VALU work per code (a 4-bit row streams two codes per byte),
// so every code converts with ONE sign-extending SDWA conversion of a byte
// (v_cvt_f32_i32 with a byte select) and one FMA, exactly:
//   8-bit: the bytes are the codes;
//   4-bit: (v << 4) & 0xF0F0F0F0 and v & 0xF0F0F0F0 put 16 * q of the low
//          and of the high nibbles in the top of each byte; the factor 16
//          is folded into the scale (a power of two, exact).
//
// Short rows: a wavefront splits into 64 / G groups of G lanes, one row per
// group (G from quant_lanes), so a 384-byte row still fills its lanes.
__device__ __forceinline__ float sbyte(unsigned v, int b) { return (float)(int)(signed char)(v >> (8 * b)); }

// 8-bit: sum_j q_j x_j over the 16 columns of one 16-byte weight vector
__device__ __forceinline__ float qdot8(const u4 w, const f4 (&xv)[4])
{
    float ta = 0.f, tb = 0.f;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const unsigned v = w[d];
        ta = fmaf(sbyte(v, 0), xv[d].x, ta);
        tb = fmaf(sbyte(v, 1), xv[d].y, tb);
        ta = fmaf(sbyte(v, 2), xv[d].z, ta);
        tb = fmaf(sbyte(v, 3), xv[d].w, tb);
    }
    return ta + tb;
}

// 4-bit: 16 * sum_j q_j x_j over the 32 columns of one 16-byte vector.  Dword
// d holds columns 8d .. 8d+7, column 8d + 2b in the low nibble of byte b and
// 8d + 2b + 1 in its high nibble.
__device__ __forceinline__ float qdot4(const u4 w, const f4 (&xv)[8])
{
    float ta = 0.f, tb = 0.f; // even columns; odd columns
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        // lo = (w << 4) & 0xF0F0F0F0, hi = w & 0xF0F0F0F0, formed here and
        // only here: written plainly, the optimiser moves each mask past the
        // byte sign extension (an AND per code instead of per dword) and
        // hoists every row's masks together (registers)
        unsigned lo, hi;
        asm volatile("v_lshlrev_b32 %0, 4, %2\n\t"
                     "v_and_b32 %0, 0xf0f0f0f0, %0\n\t"
                     "v_and_b32 %1, 0xf0f0f0f0, %2"
                     : "=&v"(lo), "=v"(hi)
                     : "v"(w[d]));
        const f4 x0 = xv[2 * d], x1 = xv[2 * d + 1];
        ta = fmaf(sbyte(lo, 0), x0.x, ta);
        tb = fmaf(sbyte(hi, 0), x0.y, tb);
        ta = fmaf(sbyte(lo, 1), x0.z, ta);
        tb = fmaf(sbyte(hi, 1), x0.w, tb);
        ta = fmaf(sbyte(lo, 2), x1.x, ta);
        tb = fmaf(sbyte(hi, 2), x1.y, tb);
        ta = fmaf(sbyte(lo, 3), x1.z, ta);
        tb = fmaf(sbyte(hi, 3), x1.w, tb);
    }
    return ta + tb;
}

// Buffer descriptor (CDNA V#) over [base, base + bytes): raw addressing, the
// gfx9-family default format word.  Loads through it take a 32-bit per-lane
// offset and a scalar offset, so R rows cost R offset registers instead of
// R 64-bit pointers, and the chunk advance is one scalar add.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes)
{
    const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, n, 0x00020000);
}
constexpr int kBufNT = 2; // cache policy: non-temporal (streamed once)

template <int BITS, int G, int R, int U>
struct QuantRows {
    static constexpr int N = 128 / BITS;       // columns per 16-byte load
    static constexpr int NX = N / 4;           // float4 of x per load
    static constexpr int CH = G * N;           // columns per row per wavefront load
    static constexpr int CB = CH * BITS / 8;   // code bytes per row per chunk
    static constexpr int XB = CH * 4;          // x bytes per chunk
    static_assert(CH % 64 == 0, "a chunk spans whole scale groups");
    static_assert(R == 1 || R == 2 || R % 4 == 0, "scale loads of 1, 2 or 4k rows");
    static constexpr int SSTEP = CH / 64 * 16; // scale-plane bytes between chunks
    __amdgpu_buffer_rsrc_t wr, sr, xr; // codes from the wave's first row; scale plane; x
    int vw[R];                         // this lane's byte offset of each code row
    int vs;                            // byte offset of the lane's first scale in chunk 0
    int sblk;                          // bytes between 4-row blocks of the scale plane
    int vx;
    int kn, nv, nfull, seg;

    // lrow[r]: the lane's r-th row relative to the wave's first row (in range:
    // rows past M are clamped by the caller); srow0: the lane's first row in
    // the scale plane (rows past M read padding or, past the plane, zeros).
    // Scale of row i, group g: float (i/4)*4*ng + 4*g + i%4.
    __device__ __forceinline__ QuantRows(const unsigned char *codes0, int64_t code_bytes,
                                         const float *plane, int64_t plane_bytes, int64_t ldw,
                                         int ng, const int (&lrow)[R], int srow0, const float *x,
                                         int K, int seg_)
        : wr(make_rsrc(codes0, code_bytes)), sr(make_rsrc(plane, plane_bytes)),
          xr(make_rsrc(x, ((int64_t)K * 4 + 15) & ~(int64_t)15)),
          vs(16 * ((srow0 / 4) * ng + seg_ * N / 64) + 4 * (srow0 % 4)), sblk(16 * ng),
          vx(seg_ * N * 4), kn(K), nv((K + N - 1) / N), nfull(K / CH), seg(seg_)
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            vw[r] = (int)(lrow[r] * ldw) + seg_ * 16;
    }

    __device__ __forceinline__ u4 wload(int r, int c) const
    {
        return __builtin_amdgcn_raw_buffer_load_b128(wr, vw[r], c * CB, kBufNT);
    }
    // the scales of the lane's R consecutive rows for chunk c: one 16-byte
    // load per 4-row block when R >= 4, the whole offset range-checked
    __device__ __forceinline__ void sload(int c, float (&sc)[R]) const
    {
        const int off = vs + c * SSTEP;
        if constexpr (R < 4) {
            // (the 64-bit raw buffer load builtin is lowered to a single
            // dword load by this compiler, so R = 2 takes two dword loads)
#pragma unroll
            for (int r = 0; r < R; ++r)
                sc[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sr, off + 4 * r, 0, 0));
        } else {
#pragma unroll
            for (int q = 0; q < R / 4; ++q) {
                const f4 v = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(sr, off + sblk * q, 0, 0));
                sc[4 * q] = v.x;
                sc[4 * q + 1] = v.y;
                sc[4 * q + 2] = v.z;
                sc[4 * q + 3] = v.w;
            }
        }
    }
    __device__ __forceinline__ f4 xload(int c, int k) const
    {
        return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(xr, vx + 16 * k, c * XB, 0));
    }
    // The same load with the whole offset in the range-checked VGPR part:
    // past the end of x (rounded to 16 bytes) it returns zeros, no branch.
    __device__ __forceinline__ f4 xload_checked(int c, int k) const
    {
        return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(xr, vx + 16 * k + c * XB, 0, 0));
    }

    __device__ __forceinline__ void accumulate(float &acc, const u4 w, float sc, const f4 (&xv)[NX]) const
    {
        if constexpr (BITS == 4)
            acc = fmaf(sc * 0.0625f, qdot4(w, xv), acc);
        else
            acc = fmaf(sc, qdot8(w, xv), acc);
    }

    __device__ __forceinline__ void load_codes(int c, u4 (&w)[R], float (&sc)[R]) const
    {
#pragma unroll
        for (int r = 0; r < R; ++r)
            w[r] = wload(r, c);
        sload(c, sc);
    }
    __device__ __forceinline__ void load_x(int c, f4 (&xv)[NX]) const
    {
#pragma unroll
        for (int k = 0; k < NX; ++k)
            xv[k] = xload(c, k);
    }
    __device__ __forceinline__ void compute(float (&acc)[R], const u4 (&w)[R], const float (&sc)[R],
                                            const f4 (&xv)[NX]) const
    {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            accumulate(acc[r], w[r], sc[r], xv);
            // decode one row at a time: only its masked dwords stay live
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // Full chunks in batches of U (all loads of a batch issued first).
    __device__ __forceinline__ void run_batched(float (&acc)[R]) const
    {
        int c = 0;
        for (; c + U <= nfull; c += U) {
            u4 w[U][R];
            float sc[U][R];
            f4 xv[U][NX];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                load_codes(c + u, w[u], sc[u]);
                load_x(c + u, xv[u]);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < U; ++u)
                compute(acc, w[u], sc[u], xv[u]);
        }
        for (; c < nfull; ++c) {
            u4 w[R];
            float sc[R];
            f4 xv[NX];
            load_codes(c, w, sc);
            load_x(c, xv);
            compute(acc, w, sc, xv);
        }
    }

    __device__ __forceinline__ void run(float (&acc)[R]) const
    {
        run_batched(acc);
        const int c = nfull;
        if (c * G < nv) { // ragged last chunk: x past kn is zero (codes are finite)
            const int v = c * G + seg;
            if (v < nv) {
                const int valid = kn - v * N;
                f4 xv[NX];
#pragma unroll
                for (int k = 0; k < NX; ++k)
                    xv[k] = mask_from<f4, 4>(xload_checked(c, k), valid - 4 * k);
                u4 w[R];
                float sc[R];
                load_codes(c, w, sc);
                compute(acc, w, sc, xv);
            }
        }
    }
};

// Reduce R values per lane over each group of G consecutive lanes (R <= G,
// both powers of two).  On return lane l holds the group total of value
// (l % G) / (G / R).
template <int R, int G>
__device__ __forceinline__ float reduce_group(float (&v)[R], int lane)
{
    static_assert(R <= G && G <= kWave, "R <= G <= 64");
    halve_all<R, G / 2>(v, lane);
#pragma unroll
    for (int o = G / (2 * R); o >= 1; o >>= 1)
        v[0] += __shfl_xor(v[0], o);
    return v[0];
}

// One quantised row tile: WV wavefronts, each 64 / G row groups x R rows.
// Group p of a wavefront takes the R consecutive rows wrow0 + p * R + r, so
// its R scales of a group sit side by side in the scale plane's 4-row blocks.
template <int BITS, int G, int R, int WV, int U>
__device__ __forceinline__ void tile_quant_g(const DevItem &it, int row0)
{
    constexpr int P = kWave / G;
    int lane = threadIdx.x & (kWave - 1);
    // lane-derived values (group, masks of the reduction) are cheap to form
    // per tile; hiding the lane index from the optimiser keeps it from
    // hoisting them for every (bits, G) branch out of a sweep's tile loop,
    // where they would stay live and cost occupancy
    asm volatile("" : "+v"(lane));
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (P * R);
    if (wrow0 >= it.M) return;
    const int sub = lane / G, seg = lane % G;
    const unsigned char *codes = static_cast<const unsigned char *>(it.W);
    const int Mp = (it.M + 3) / 4 * 4;
    const float *plane = reinterpret_cast<const float *>(codes + (int64_t)it.M * it.ldw);
    const int rows_left = it.M - wrow0; // >= 1
    int lrow[R];
#pragma unroll
    for (int r = 0; r < R; ++r) // rows past M: computed from row M - 1, not stored
        lrow[r] = min(sub * R + r, rows_left - 1);
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.f;
    const int ng = (it.K + 63) / 64;
    const QuantRows<BITS, G, R, U> qr(codes + (int64_t)wrow0 * it.ldw, (int64_t)rows_left * it.ldw,
                                      plane, (int64_t)4 * Mp * ng, it.ldw, ng, lrow,
                                      wrow0 + sub * R, it.x, it.K, seg);
    qr.run(acc);
    const float v = reduce_group<R, G>(acc, lane);
    constexpr int S = G / R; // lanes holding each row's total
    if (seg % S == 0) {
        const int row = wrow0 + sub * R + seg / S;
        if (row < it.M) it.y[row] = v;
    }
}

template <int BITS, int R, int WV, int U>
__device__ __forceinline__ void tile_quant(const DevItem &it, int row0)
{
    switch (it.lanes) {
    case 8: tile_quant_g<BITS, 8, R, WV, U>(it, row0); break;
    case 16: tile_quant_g<BITS, 16, R, WV, U>(it, row0); break;
    case 32: tile_quant_g<BITS, 32, R, WV, U>(it, row0); break;
    default: tile_quant_g<BITS, 64, R, WV, U>(it, row0); break;
    }
}

// Any plain item (fp32, fp16, 8-bit or 4-bit weights), direct-x.
template <int R, int WV, int U>
__device__ __forceinline__ void tile_plain_any(const DevItem &it, int row0)
{
    switch (it.dtype) {
    case 3: tile_quant<4, R, WV, U>(it, row0); break;
    case 2: tile_quant<8, R, WV, U>(it, row0); break;
    case 1: tile_fused<_Float16, R, WV, U, false, false>(it, row0); break;
    default: tile_fused<float, R, WV, U, false, false>(it, row0); break;
    }
}

template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_sweep_quant(const DevItem *__restrict__ items,
                                                            const DevTile *__restrict__ tiles,
                                                            int ntiles)
{
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_plain_any<R, WV, U>(it, tl.row0);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_item_quant(const DevItem it)
{
    tile_plain_any<R, WV, U>(it, (int)blockIdx.x * (R * WV * (kWave / it.lanes)));
}

// Grouped sweep whose items may carry a fused RMSNorm and/or be SwiGLU
// pairs: the same tile loop, with the item's kind chosen per tile.
template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_sweep_fused(const DevItem *__restrict__ items,
                                                            const DevTile *__restrict__ tiles,
                                                            int ntiles)
{
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        if (it.dtype == 1)
            tile_any<_Float16, R, WV, U>(it, tl.row0);
        else
            tile_any<float, R, WV, U>(it, tl.row0);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

// One item passed by value: workgroup b computes its row tile b.
template <int R, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_item(const DevItem it)
{
    const int row0 = (int)blockIdx.x * tile_rows<R, WV>(it.op);
    if (it.dtype == 1)
        tile_any<_Float16, R, WV, U>(it, row0);
    else
        tile_any<float, R, WV, U>(it, row0);
}

template <typename E>
__global__ __launch_bounds__(256) void k_pack(E *__restrict__ dst, int64_t ldw,
                                              const E *__restrict__ src, int64_t M, int64_t K)
{
    for (int64_t row = blockIdx.x; row < M; row += gridDim.x)
        for (int64_t j = threadIdx.x; j < ldw; j += blockDim.x)
            dst[row * ldw + j] = (j < K) ? src[row * K + j] : E(0);
}

__global__ __launch_bounds__(256) void k_zero_i32(int *p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// Read-only streaming with the GEMV's load kind: workgroup b reads the
// contiguous span [b*per, (b+1)*per) of 16-byte vectors, eight loads in
// flight per lane, and writes one float so the loads cannot be optimised away.
__global__ __launch_bounds__(256) void k_read_stream(const f4 *__restrict__ src, int64_t nvec,
                                                     int64_t per, float *__restrict__ sink)
{
    __shared__ float red[4];
    const int64_t beg = (int64_t)blockIdx.x * per;
    const int64_t end = min(beg + per, nvec);
    const TVL_GLOBAL f4 *g = (const TVL_GLOBAL f4 *)(src);
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    int64_t i = beg + threadIdx.x;
    for (; i + 7 * 256 < end; i += 8 * 256) {
        f4 a[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            a[u] = __builtin_nontemporal_load(g + i + u * 256);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            acc += a[u];
    }
    for (; i < end; i += 256)
        acc += __builtin_nontemporal_load(g + i);
    float v = (acc.x + acc.y) + (acc.z + acc.w);
    for (int o = 32; o >= 1; o >>= 1)
        v += __shfl_xor(v, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x / 64] = v;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(256) void k_copy(f4 *__restrict__ dst, const f4 *__restrict__ src,
                                              int64_t nvec)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec;
         i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = __builtin_nontemporal_load(src + i);
}

// ------------------------------------------------------ shape dispatch
// (R, waves per block, U) triples the library instantiates, per x mode.
#define TVL_LDS_SHAPES(X)                                                                         \
    X(1, 4, 4) X(1, 4, 8) X(2, 4, 2) X(2, 4, 3) X(2, 4, 4) X(2, 4, 8) X(4, 4, 1) X(4, 4, 2)       \
    X(4, 4, 3) X(4, 4, 4) X(8, 4, 1) X(8, 4, 2) X(2, 8, 4) X(2, 8, 8) X(4, 8, 2) X(1, 2, 8)       \
    X(2, 2, 8) X(4, 2, 4) X(8, 2, 2)
#define TVL_DIRECT_SHAPES(X)                                                                      \
    X(1, 1, 4) X(1, 1, 8) X(2, 1, 2) X(2, 1, 3) X(2, 1, 4) X(2, 1, 8) X(4, 1, 1) X(4, 1, 2)       \
    X(4, 1, 3) X(4, 1, 4) X(8, 1, 1) X(8, 1, 2) X(1, 4, 4) X(1, 4, 8) X(2, 4, 2) X(2, 4, 3)       \
    X(2, 4, 4) X(2, 4, 8) X(4, 4, 1) X(4, 4, 2) X(4, 4, 3) X(4, 4, 4) X(8, 4, 1) X(8, 4, 2)

// (R, waves per block, U) triples with fused RMSNorm / SwiGLU support.
#define TVL_FUSED_SHAPES(X)                                                                       \
    X(2, 4, 2) X(2, 4, 3) X(2, 4, 4) X(2, 1, 4) X(4, 1, 2) X(4, 1, 4) X(4, 4, 2) X(2, 1, 8)

template <int R, int WV, int U>
struct InstFused {
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_fused<R, WV, U>), dim3(grid), dim3(WV * kWave), 0, st, items,
                           tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const int rows = tile_rows<R, WV>(it.op);
        const dim3 grid((it.M + rows - 1) / rows), block(WV * kWave);
        hipLaunchKernelGGL((k_item<R, WV, U>), grid, block, 0, st, it);
        return hipGetLastError();
    }
};

// (R, waves per block, U, B) with B x vectors per launch (B >= nrhs).
#define TVL_MULTI_SHAPES(X)                                                                       \
    X(2, 4, 2, 2) X(2, 4, 4, 2) X(4, 4, 2, 2) X(2, 4, 1, 4) X(2, 4, 2, 4) X(4, 4, 1, 4)          \
        X(4, 4, 2, 4) X(2, 4, 1, 8) X(2, 4, 2, 8) X(4, 4, 1, 8)

template <int R, int WV, int U, int B>
struct InstMulti {
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_multi<R, WV, U, B>), dim3(grid), dim3(WV * kWave), 0, st,
                           items, tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        hipLaunchKernelGGL((k_item_multi<R, WV, U, B>), grid, block, 0, st, it);
        return hipGetLastError();
    }
};

// (R, waves per block, U) for plans holding block-quantised weights.
#define TVL_QUANT_SHAPES(X)                                                                       \
    X(2, 4, 2) X(4, 4, 1) X(4, 4, 2) X(4, 1, 2) X(8, 4, 1) X(8, 2, 1)

template <int R, int WV, int U>
struct InstQuant {
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_quant<R, WV, U>), dim3(grid), dim3(WV * kWave), 0, st, items,
                           tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const int rows = R * WV * (kWave / it.lanes);
        const dim3 grid((it.M + rows - 1) / rows), block(WV * kWave);
        hipLaunchKernelGGL((k_item_quant<R, WV, U>), grid, block, 0, st, it);
        return hipGetLastError();
    }
};

template <int R, int WV, int U, int XM>
hipError_t launch_ksplit(int dtype, const void *W, int64_t ldw, const float *x, float *y, int M,
                         int K, int S, float *partials, int *counters, hipStream_t st)
{
    // slice width: a whole number of LDS chunks, S' = ceil(K / kspan) <= S
    const int per = (K + S - 1) / S;
    const int kspan = (per + kChunkElems - 1) / kChunkElems * kChunkElems;
    const int Se = (K + kspan - 1) / kspan;
    const int ks = XM == kXLds ? slice_cap(kspan) : 0;
    const int tiles = (M + R * WV - 1) / (R * WV);
    const dim3 grid(tiles * Se), block(WV * kWave);
    if (dtype == 1)
        hipLaunchKernelGGL((k_gemv_ksplit<_Float16, R, WV, U, XM>), grid, block, ks * 4, st,
                           static_cast<const _Float16 *>(W), ldw, x, y, M, K, ks, Se, kspan,
                           partials, counters);
    else
        hipLaunchKernelGGL((k_gemv_ksplit<float, R, WV, U, XM>), grid, block, ks * 4, st,
                           static_cast<const float *>(W), ldw, x, y, M, K, ks, Se, kspan,
                           partials, counters);
    return hipGetLastError();
}

template <int R, int WV, int U>
struct Inst {
    static hipError_t rows(int dtype, const void *W, int64_t ldw, const float *x, float *y, int M,
                           int K, hipStream_t st)
    {
        const int ks = slice_cap(K);
        const dim3 grid((M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (dtype == 1)
            hipLaunchKernelGGL((k_gemv_rows<_Float16, R, WV, U>), grid, block, ks * 4, st,
                               static_cast<const _Float16 *>(W), ldw, x, y, M, K, ks);
        else
            hipLaunchKernelGGL((k_gemv_rows<float, R, WV, U>), grid, block, ks * 4, st,
                               static_cast<const float *>(W), ldw, x, y, M, K, ks);
        return hipGetLastError();
    }
    static hipError_t ksplit(int dtype, const void *W, int64_t ldw, const float *x, float *y,
                             int M, int K, int S, float *partials, int *counters, hipStream_t st)
    {
        return launch_ksplit<R, WV, U, kXLds>(dtype, W, ldw, x, y, M, K, S, partials, counters,
                                              st);
    }
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            int ks_cap, hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep<R, WV, U>), dim3(grid), dim3(WV * kWave), ks_cap * 4, st,
                           items, tiles, ntiles, ks_cap);
        return hipGetLastError();
    }
};

template <int R, int WV, int U>
struct InstDirect {
    static hipError_t rows(int dtype, const void *W, int64_t ldw, const float *x, float *y, int M,
                           int K, hipStream_t st)
    {
        const dim3 grid((M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (dtype == 1)
            hipLaunchKernelGGL((k_gemv_rows_direct<_Float16, R, WV, U>), grid, block, 0, st,
                               static_cast<const _Float16 *>(W), ldw, x, y, M, K);
        else
            hipLaunchKernelGGL((k_gemv_rows_direct<float, R, WV, U>), grid, block, 0, st,
                               static_cast<const float *>(W), ldw, x, y, M, K);
        return hipGetLastError();
    }
    static hipError_t ksplit(int dtype, const void *W, int64_t ldw, const float *x, float *y,
                             int M, int K, int S, float *partials, int *counters, hipStream_t st)
    {
        return launch_ksplit<R, WV, U, kXDirect>(dtype, W, ldw, x, y, M, K, S, partials,
                                                 counters, st);
    }
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_direct<R, WV, U>), dim3(grid), dim3(WV * kWave), 0, st, items,
                           tiles, ntiles);
        return hipGetLastError();
    }
};

}  // namespace

bool shape_supported(const Shape &s)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return true;
    if (s.xmode == kXLds) {
        TVL_LDS_SHAPES(X)
    } else if (s.xmode == kXDirect) {
        TVL_DIRECT_SHAPES(X)
    }
#undef X
    return false;
}

hipError_t launch_gemv_rows(const Shape &s, int dtype, const void *W, int64_t ldw,
                            const float *x, float *y, int M, int K, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return Inst<R_, W_, U_>::rows(dtype, W, ldw, x, y, M, K, st);
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstDirect<R_, W_, U_>::rows(dtype, W, ldw, x, y, M, K, st);
    if (s.xmode == kXLds) {
        TVL_LDS_SHAPES(X)
    } else {
        TVL_DIRECT_SHAPES(Y)
    }
#undef X
#undef Y
    return hipErrorInvalidValue;
}

hipError_t launch_gemv_ksplit(const Shape &s, int dtype, const void *W, int64_t ldw,
                              const float *x, float *y, int M, int K, int S, float *partials,
                              int *counters, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return Inst<R_, W_, U_>::ksplit(dtype, W, ldw, x, y, M, K, S, partials, counters, st);
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstDirect<R_, W_, U_>::ksplit(dtype, W, ldw, x, y, M, K, S, partials, counters,   \
                                              st);
    if (s.xmode == kXLds) {
        TVL_LDS_SHAPES(X)
    } else {
        TVL_DIRECT_SHAPES(Y)
    }
#undef X
#undef Y
    return hipErrorInvalidValue;
}

hipError_t launch_sweep(const Shape &s, const DevItem *items, const DevTile *tiles, int ntiles,
                        int grid, int ks_cap, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return Inst<R_, W_, U_>::sweep(items, tiles, ntiles, grid, ks_cap, st);
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstDirect<R_, W_, U_>::sweep(items, tiles, ntiles, grid, st);
    if (s.xmode == kXLds) {
        TVL_LDS_SHAPES(X)
    } else {
        TVL_DIRECT_SHAPES(Y)
    }
#undef X
#undef Y
    return hipErrorInvalidValue;
}

bool fused_shape_supported(const Shape &s)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return s.xmode == kXDirect;
    TVL_FUSED_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_sweep_fused(const Shape &s, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstFused<R_, W_, U_>::sweep(items, tiles, ntiles, grid, st);
    TVL_FUSED_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_item(const Shape &s, const DevItem &item, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstFused<R_, W_, U_>::item(item, st);
    TVL_FUSED_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

bool multi_shape_supported(const Shape &s, int B)
{
#define X(R_, W_, U_, B_)                                                                         \
    if (s.R == R_ && s.W == W_ && s.U == U_ && B == B_) return s.xmode == kXDirect;
    TVL_MULTI_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_sweep_multi(const Shape &s, int B, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, hipStream_t st)
{
#define X(R_, W_, U_, B_)                                                                         \
    if (s.R == R_ && s.W == W_ && s.U == U_ && B == B_)                                          \
        return InstMulti<R_, W_, U_, B_>::sweep(items, tiles, ntiles, grid, st);
    TVL_MULTI_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_item_multi(const Shape &s, int B, const DevItem &item, hipStream_t st)
{
#define X(R_, W_, U_, B_)                                                                         \
    if (s.R == R_ && s.W == W_ && s.U == U_ && B == B_)                                          \
        return InstMulti<R_, W_, U_, B_>::item(item, st);
    TVL_MULTI_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

bool quant_shape_supported(const Shape &s)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return s.xmode == kXDirect;
    TVL_QUANT_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_sweep_quant(const Shape &s, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstQuant<R_, W_, U_>::sweep(items, tiles, ntiles, grid, st);
    TVL_QUANT_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_item_quant(const Shape &s, const DevItem &item, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstQuant<R_, W_, U_>::item(item, st);
    TVL_QUANT_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_pack(int dtype, void *dst, int64_t ldw, const void *src, int64_t M, int64_t K,
                       hipStream_t st)
{
    const int grid = (int)(M < 65536 ? M : 65536);
    if (dtype == 1)
        hipLaunchKernelGGL(k_pack<uint16_t>, dim3(grid), dim3(256), 0, st,
                           static_cast<uint16_t *>(dst), ldw, static_cast<const uint16_t *>(src),
                           M, K);
    else
        hipLaunchKernelGGL(k_pack<uint32_t>, dim3(grid), dim3(256), 0, st,
                           static_cast<uint32_t *>(dst), ldw, static_cast<const uint32_t *>(src),
                           M, K);
    return hipGetLastError();
}

hipError_t launch_zero_i32(int *p, int64_t n, hipStream_t st)
{
    int64_t g = (n + 255) / 256;
    const int grid = (int)(g < 4096 ? (g > 0 ? g : 1) : 4096);
    hipLaunchKernelGGL(k_zero_i32, dim3(grid), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

hipError_t launch_read_stream(const void *src, int64_t bytes, float *sink, int grid,
                              hipStream_t st)
{
    const int64_t nvec = bytes / 16;
    const int64_t per = (nvec + grid - 1) / grid;
    hipLaunchKernelGGL(k_read_stream, dim3(grid), dim3(256), 0, st,
                       static_cast<const f4 *>(src), nvec, per, sink);
    return hipGetLastError();
}

hipError_t launch_copy(void *dst, const void *src, int64_t bytes, hipStream_t st)
{
    const int64_t nvec = bytes / 16;
    int64_t g = (nvec + 255) / 256;
    const int grid = (int)(g < 8192 ? (g > 0 ? g : 1) : 8192);
    hipLaunchKernelGGL(k_copy, dim3(grid), dim3(256), 0, st, static_cast<f4 *>(dst),
                       static_cast<const f4 *>(src), nvec);
    return hipGetLastError();
}

}  // namespace tvl
