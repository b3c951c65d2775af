// tvl_multi.hip -- several-vector GEMV (beam search with up to 8
// hypotheses, Sec. 9.1): the weights are read once for all x vectors.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvl_device.h"

namespace tvl {
namespace {

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

}  // namespace

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

}  // namespace tvl
