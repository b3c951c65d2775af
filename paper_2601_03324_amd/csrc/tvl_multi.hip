// tvl_multi.hip -- several-vector GEMV (beam search with up to 16
// hypotheses, Sec. 9.1): the weights are read once for all x vectors, on the
// vector ALUs (up to 8 vectors) or on the matrix cores (up to 16).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

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

// ------------------------------------------------------------ matrix cores
// With several vectors the GEMV is a skinny dense contraction,
// Y^T[M x nb] = W[M x K] X^T[K x nb], and the VALU form above spends its
// issue slots on nb FMAs per weight.  The matrix cores take the products:
// v_mfma_f32_4x4x1f32 (16 blocks) computes 16 independent 4 x 4 outer
// products per instruction, in fp32 with fp32 accumulation.
//
// Operand layout of the 16-block 4x4x1 form (CDNA3/4 ISA): lane l = 4 b + q
// supplies A_b[q][0] and B_b[0][q] and holds D_b[v][q] in element v of its
// 4-float accumulator, for block b = l / 4.
//
// So the four lanes of a quad must hold four rows (and four vectors) at one
// column.  Loading that layout directly would have every quad touch four
// cache lines (the direct-load 16 x 16 x 4 form below has loads of that kind
// and measures what they cost); instead every load here is the fully
// coalesced one of the VALU kernels
// (lane l reads 16 bytes at column N l of ONE row: 1 KB per wavefront load),
// four rows (or four vectors) are loaded, and a 4 x 4 transpose across each
// quad (two DPP exchange steps) moves row q's 16 bytes at column N (4 b + s)
// into register s of lane 4 b + q.  MFMA (s, e) then multiplies, in block b,
// column N (4 b + s) + e of the rows by the same column of the vectors.  A
// chunk is 64 N columns; per chunk and group of 4 rows that is 4 N MFMAs per
// group of 4 vectors, and the 16 blocks are added across lanes at the end
// (a fixed tree).
//
// Accumulation: every kFlush chunks the block accumulators are added into a
// per-wavefront fp32 total in LDS and cleared (the totals stay out of the
// register file, which bounds the loads a wavefront keeps in flight), so each
// output sums at most 4 N kFlush products per block and window, then
// K / (64 N kFlush) window totals, then a 16-way tree:
// |error| <= (4 N kFlush + K / (64 N kFlush) + 6) * 2^-24 * sum_j |W_ij x_j|
// to first order (2.9e-6 at K = 11008, fp32).
constexpr int kFlush = 2;

__device__ __forceinline__ f4 mfma4x4(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_4x4x1f32(a, b, c, 0, 0, 0);
}

// value of v in lane (lane ^ 1) / (lane ^ 2) of the same quad (DPP quad_perm)
__device__ __forceinline__ float quad_xor1(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1,
                                                              0xF, 0xF, false));
}
__device__ __forceinline__ float quad_xor2(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E,
                                                              0xF, 0xF, false));
}

// 4 x 4 transpose across a quad, element by element: on return register s of
// lane q holds what register q of lane s held (q = lane % 4).  Each step
// swaps one bit of the register index with the same bit of the lane index:
// the lane whose bit is set sends its lower register, the other its upper.
__device__ __forceinline__ void quad_transpose(f4 (&v)[4], int lane)
{
    const bool q0 = (lane & 1) != 0, q1 = (lane & 2) != 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        // plain values (selecting between array elements would make the
        // compiler address the array, i.e. put it in scratch memory)
        float m0 = v[0][e], m1 = v[1][e], m2 = v[2][e], m3 = v[3][e];
        // pairs (0, 1), (2, 3): lane bit 0
        const float r01 = quad_xor1(q0 ? m0 : m1);
        const float r23 = quad_xor1(q0 ? m2 : m3);
        m0 = q0 ? r01 : m0;
        m1 = q0 ? m1 : r01;
        m2 = q0 ? r23 : m2;
        m3 = q0 ? m3 : r23;
        // pairs (0, 2), (1, 3): lane bit 1
        const float r02 = quad_xor2(q1 ? m0 : m2);
        const float r13 = quad_xor2(q1 ? m1 : m3);
        v[0][e] = q1 ? r02 : m0;
        v[2][e] = q1 ? m2 : r02;
        v[1][e] = q1 ? r13 : m1;
        v[3][e] = q1 ? m3 : r13;
    }
}

// TT groups of 4 rows, P groups of 4 vectors.  A wavefront issues a whole
// chunk (4 TT weight loads of 1 KB and 4 P NX x loads) before it transposes
// and multiplies it.
template <typename T, int TT, int P>
struct MfmaRows {
    using V = typename Vec<T>::type;
    static constexpr int N = Vec<T>::N;  // columns per 16-byte weight load
    static constexpr int CH = kWave * N; // columns per chunk
    static constexpr int NX = N / 4;     // x float4 per lane per vector per chunk
    const T *w0;     // the wavefront's first row, at this lane's column N l
    const float *x0; // vector 0, at column N l
    int64_t ldw, ldx;
    int rmax, nb, kn, nfull, lane; // rmax: last row offset in range (rows past M re-read it)

    __device__ __forceinline__ MfmaRows(const T *W, int64_t ldw_, int wrow0, int M,
                                        const float *x, int64_t ldx_, int nb_, int K, int lane_)
        : w0(W + (int64_t)wrow0 * ldw_ + N * lane_), x0(x + N * lane_), ldw(ldw_), ldx(ldx_),
          rmax(M - 1 - wrow0), nb(nb_), kn(K), nfull(K / CH), lane(lane_)
    {
    }

    // rows 4t .. 4t+3 (row r in register r) and vectors 4p .. 4p+3 (vector r
    // in register r) of chunk c, columns past K masked to zero when RAGGED.
    // An x float4 is read only when it starts before K, so it lies in a
    // 16-byte block holding a valid element.
    template <bool RAGGED>
    __device__ __forceinline__ void load(int c, V (&w)[TT][4], f4 (&xv)[P][NX][4]) const
    {
        const int valid = kn - (c * CH + N * lane);
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const T *src = w0 + (int64_t)min(4 * t + r, rmax) * ldw + c * CH;
                if constexpr (RAGGED)
                    w[t][r] = valid > 0 ? mask_from<V, N>(load_w<T>(src), valid) : V{};
                else
                    w[t][r] = load_w<T>(src);
            }
        const f4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool on = 4 * p + r < nb; // wave-uniform
                const float *src = x0 + (int64_t)(on ? 4 * p + r : 0) * ldx + c * CH;
#pragma unroll
                for (int h = 0; h < NX; ++h) {
                    if constexpr (RAGGED)
                        xv[p][h][r] = (on && valid > 4 * h)
                                          ? mask_from<f4, 4>(load_x4(src + 4 * h), valid - 4 * h)
                                          : z;
                    else
                        xv[p][h][r] = on ? load_x4(src + 4 * h) : z;
                }
            }
    }

    __device__ __forceinline__ void compute(V (&w)[TT][4], f4 (&xv)[P][NX][4],
                                            f4 (&acc)[TT][P]) const
    {
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
            for (int h = 0; h < NX; ++h)
                quad_transpose(xv[p][h], lane);
#pragma unroll
        for (int t = 0; t < TT; ++t) {
            // transpose the raw 16-byte weight pieces (fp16: two halves per
            // dword move together; converted to fp32 per piece below)
            f4 raw[4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
                raw[r] = __builtin_bit_cast(f4, w[t][r]);
            quad_transpose(raw, lane);
            f4 wf[NX][4];
#pragma unroll
            for (int sidx = 0; sidx < 4; ++sidx) {
                if constexpr (N == 4) {
                    wf[0][sidx] = raw[sidx];
                } else {
                    const f8 c8 = __builtin_convertvector(__builtin_bit_cast(V, raw[sidx]), f8);
                    wf[0][sidx] = f4{c8[0], c8[1], c8[2], c8[3]}; // exact
                    wf[1][sidx] = f4{c8[4], c8[5], c8[6], c8[7]};
                }
            }
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
                for (int sidx = 0; sidx < 4; ++sidx)
#pragma unroll
                    for (int h = 0; h < NX; ++h)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            acc[t][p] = mfma4x4(wf[h][sidx][e], xv[p][h][sidx][e], acc[t][p]);
        }
    }

    template <bool RAGGED>
    __device__ __forceinline__ void chunk(int c, f4 (&acc)[TT][P]) const
    {
        V w[TT][4];
        f4 xv[P][NX][4];
        load<RAGGED>(c, w, xv);
        __builtin_amdgcn_sched_barrier(0); // the chunk's loads first
        compute(w, xv, acc);
        __builtin_amdgcn_sched_barrier(0); // the next chunk's loads stay below
    }

    // slot[(t * P + p) * 64]: this lane's LDS total of group (t, p)
    __device__ __forceinline__ static void flush(f4 (&acc)[TT][P], f4 *slot)
    {
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int p = 0; p < P; ++p) {
                slot[(t * P + p) * kWave] += acc[t][p];
                acc[t][p] = f4{0.f, 0.f, 0.f, 0.f};
            }
    }

    // on return tot[t][p] holds the group's block sums
    __device__ __forceinline__ void run(f4 (&tot)[TT][P], f4 *slot) const
    {
        f4 acc[TT][P];
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int p = 0; p < P; ++p) {
                acc[t][p] = f4{0.f, 0.f, 0.f, 0.f};
                slot[(t * P + p) * kWave] = acc[t][p];
            }
        int c = 0;
        for (; c + kFlush <= nfull; c += kFlush) {
#pragma unroll
            for (int h = 0; h < kFlush; ++h)
                chunk<false>(c + h, acc);
            flush(acc, slot);
        }
        for (; c < nfull; ++c)
            chunk<false>(c, acc);
        if (c * CH < kn) // every lane reaches the DPP steps and the MFMAs
            chunk<true>(c, acc);
        // LDS totals + the last window, still in registers
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int p = 0; p < P; ++p)
                tot[t][p] = slot[(t * P + p) * kWave] + acc[t][p];
    }
};

// One row tile of a several-vector item on the matrix cores: WV wavefronts
// x TT groups of 4 rows, all nb <= 4 P vectors.  `slots`: this wavefront's
// TT * P * 64 float4 of LDS.
template <typename T, int TT, int P, int WV, int U>
__device__ __forceinline__ void tile_mfma_p(const DevItem &it, int row0, f4 *slots)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (4 * TT);
    if (wrow0 >= it.M) return; // no barrier follows
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f4 tot[TT][P];
    const MfmaRows<T, TT, P> mr(static_cast<const T *>(it.W), it.ldw, wrow0, it.M, it.x, it.ldx,
                                   nb, it.K, lane);
    mr.run(tot, slots + lane);
    // add the 16 blocks: lane l = 4 b + j holds D_b[v][j] in element v; two
    // exchange steps leave row v = (l >> 4) & 3 in each lane, two more sum
    // the remaining 4 blocks, and lanes with b % 4 == 0 store
    const int i = (lane >> 4) & 3, j = lane & 3;
#pragma unroll
    for (int t = 0; t < TT; ++t) {
        const int row = wrow0 + 4 * t + i;
#pragma unroll
        for (int p = 0; p < P; ++p) {
            float v[4] = {tot[t][p].x, tot[t][p].y, tot[t][p].z, tot[t][p].w};
            halve<2, 32>(v, lane);
            halve<1, 16>(v, lane);
            v[0] += __shfl_xor(v[0], 8);
            v[0] += __shfl_xor(v[0], 4);
            if ((lane & 12) == 0 && row < it.M && 4 * p + j < nb)
                it.y[(int64_t)(4 * p + j) * it.ldy + row] = v[0];
        }
    }
}

// Weight dtypes a matrix-core launch holds: fp32 only, fp16 only, or both
// (a mixed launch pays the registers of both paths).
constexpr int kWF32 = 0, kWF16 = 1, kWMixed = 2;

template <int WM, int TT, int P, int WV, int U>
__device__ __forceinline__ void tile_mfma(const DevItem &it, int row0, f4 *slots)
{
    if constexpr (WM == kWF32)
        tile_mfma_p<float, TT, P, WV, U>(it, row0, slots);
    else if constexpr (WM == kWF16)
        tile_mfma_p<_Float16, TT, P, WV, U>(it, row0, slots);
    else if (it.dtype == 1)
        tile_mfma_p<_Float16, TT, P, WV, U>(it, row0, slots);
    else
        tile_mfma_p<float, TT, P, WV, U>(it, row0, slots);
}

// P groups of 4 vectors: chosen per launch from the largest nrhs (registers
// grow with P, so a launch holds only the groups it needs)
template <int WM, int TT, int P, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_sweep_mfma(const DevItem *__restrict__ items,
                                                           const DevTile *__restrict__ tiles,
                                                           int ntiles)
{
    __shared__ f4 lds[WV * TT * P * kWave];
    f4 *slots = lds + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave) * (TT * P * kWave);
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_mfma<WM, TT, P, WV, U>(it, tl.row0, slots);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int WM, int TT, int P, int WV, int U>
__global__ __launch_bounds__(WV *kWave) void k_item_mfma(const DevItem it)
{
    __shared__ f4 lds[WV * TT * P * kWave];
    f4 *slots = lds + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave) * (TT * P * kWave);
    tile_mfma<WM, TT, P, WV, U>(it, (int)blockIdx.x * (4 * TT * WV), slots);
}

// (rows per wavefront = 4 TT in {8, 16}, waves per block, U = 1: one chunk
// of 64 N columns in flight) of the matrix-core form; any number of vectors
// up to 16.
#define TVL_MFMA_SHAPES(X) X(8, 4, 1) X(16, 1, 1) X(16, 2, 1)

template <int R, int WV, int U>
struct InstMfma {
    template <int WM, int P>
    static hipError_t sweep_p(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                              hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_mfma<WM, R / 4, P, WV, U>), dim3(grid), dim3(WV * kWave), 0,
                           st, items, tiles, ntiles);
        return hipGetLastError();
    }
    template <int WM>
    static hipError_t sweep_w(int B, const DevItem *items, const DevTile *tiles, int ntiles,
                              int grid, hipStream_t st)
    {
        return B <= 4   ? sweep_p<WM, 1>(items, tiles, ntiles, grid, st)
               : B <= 8 ? sweep_p<WM, 2>(items, tiles, ntiles, grid, st)
                        : sweep_p<WM, 4>(items, tiles, ntiles, grid, st);
    }
    // B: the launch's vector bound (2, 4, 8 or 16) -> P = ceil(B / 4);
    // wm: the weight dtypes the launch holds
    static hipError_t sweep(int B, int wm, const DevItem *items, const DevTile *tiles, int ntiles,
                            int grid, hipStream_t st)
    {
        return wm == kWF32   ? sweep_w<kWF32>(B, items, tiles, ntiles, grid, st)
               : wm == kWF16 ? sweep_w<kWF16>(B, items, tiles, ntiles, grid, st)
                             : sweep_w<kWMixed>(B, items, tiles, ntiles, grid, st);
    }
    template <int WM, int P>
    static hipError_t item_p(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        hipLaunchKernelGGL((k_item_mfma<WM, R / 4, P, WV, U>), grid, block, 0, st, it);
        return hipGetLastError();
    }
    template <int WM>
    static hipError_t item_w(int B, const DevItem &it, hipStream_t st)
    {
        return B <= 4 ? item_p<WM, 1>(it, st) : B <= 8 ? item_p<WM, 2>(it, st) : item_p<WM, 4>(it, st);
    }
    static hipError_t item(int B, const DevItem &it, hipStream_t st)
    {
        return it.dtype == 1 ? item_w<kWF16>(B, it, st) : item_w<kWF32>(B, it, st);
    }
};

// ------------------------------------------------ matrix cores, 16 x 16 x 4
// v_mfma_f32_16x16x4f32: D[16 x 16] += A[16 x 4] B[4 x 16], fp32 inputs and
// accumulation.  Lane l = 16 g + i supplies A[i][g] and B[g][i] and holds
// D[4 g + v][i] in element v of its accumulator (checked on gfx950).
//
// A is 16 rows of W and B holds up to 16 x vectors (vector j in column j),
// so each lane loads 16 bytes of row i: 16-byte block g of a 64-byte row
// segment.  One wavefront load then covers 16 rows x 64 bytes (N columns
// per lane: 4 fp32 or 8 fp16), and its e-th MFMA multiplies column
// 4 N q + N g + e of the 16 rows by the same column of the 16 vectors.
// The loads feed the matrix cores as they arrive: no lane exchange, and
// only the loaded registers in flight (62-144 VGPRs against 146-256 for the
// 4 x 4 x 1 form).  The price: such a load touches 16 half lines rather than
// 8 whole ones (the other half comes with the next load of the same batch).
// HBM bytes stay within 4 % of the whole-line form, but the L1 receives 1.7x
// the requests and the address unit stalls on it (rocprofv3 on MI355X), so
// this form tops out near 3.8 TB/s whatever the vector count.  The LDS-staged
// forms below avoid the half lines and are faster; this form serves their
// rows too long for a buffer descriptor and explicit tunings.
//
// The x loads (vector i, columns as for the weights) hit the cache: every
// wavefront of a matrix reads the same vectors; RG groups of 16 rows share
// each x load.  Vectors past nb re-read vector nb - 1, rows past M the last
// row; those results are dropped.
//
// Accumulation: the MFMAs of one batch (Q loads per row group) chain into
// one accumulator, which is then added into a first-level total and cleared;
// every kMfmaLevel batches the first-level total is added into a second.
// Each output therefore sums at most Q N MFMA steps of 4 products, then
// kMfmaLevel batch sums, then K / (kMfmaLevel 4 N Q) totals:
// |error| <= (Q N + 4 + kMfmaLevel + K / (kMfmaLevel 4 N Q) + 1) 2^-24
// sum_j |W_ij x_j| to first order (3.5e-6 at K = 11008, fp32, Q = 8).
constexpr int kMfmaLevel = 16;

__device__ __forceinline__ f4 mfma16(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <typename T, int RG, int Q>
struct Mfma16Rows {
    using V = typename Vec<T>::type;
    static constexpr int N = Vec<T>::N; // columns per lane per load
    static constexpr int CL = 4 * N;    // columns per wavefront load
    static constexpr int CB = Q * CL;   // columns per batch
    const T *w[RG];  // row 16 rg + i of the wavefront, at column N g
    const float *xv; // vector i (clamped), at column N g
    int kn, g;

    __device__ __forceinline__ Mfma16Rows(const T *W, int64_t ldw, int wrow0, int M,
                                          const float *x, int64_t ldx, int nb, int K, int lane)
        : kn(K), g(lane >> 4)
    {
        const int i = lane & 15;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            w[rg] = W + (int64_t)min(wrow0 + 16 * rg + i, M - 1) * ldw + N * g;
        xv = x + (int64_t)min(i, nb - 1) * ldx + N * g;
    }

    // one batch: columns [c0, c0 + CB); when RAGGED, columns past K are
    // masked to zero (a 16-byte piece is loaded only when it starts before
    // K, so it lies in the row's padded extent and in an x block holding a
    // valid element)
    template <bool RAGGED>
    __device__ __forceinline__ void batch(int c0, f4 (&acc)[RG]) const
    {
        V wv[Q][RG];
        f4 xa[Q], xb[Q];
        const f4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int c = c0 + CL * q;
            const int valid = kn - (c + N * g);
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                if constexpr (RAGGED)
                    wv[q][rg] = valid > 0 ? mask_from<V, N>(load_w<T>(w[rg] + c), valid) : V{};
                else
                    wv[q][rg] = load_w<T>(w[rg] + c);
            }
            if constexpr (RAGGED) {
                xa[q] = valid > 0 ? mask_from<f4, 4>(load_x4(xv + c), valid) : z;
                xb[q] = (N == 8 && valid > 4) ? mask_from<f4, 4>(load_x4(xv + c + 4), valid - 4)
                                              : z;
            } else {
                xa[q] = load_x4(xv + c);
                xb[q] = (N == 8) ? load_x4(xv + c + 4) : z;
            }
        }
        __builtin_amdgcn_sched_barrier(0); // the batch's loads first
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                if constexpr (N == 4) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[rg] = mfma16(wv[q][rg][e], xa[q][e], acc[rg]);
                } else {
                    const f8 wf = __builtin_convertvector(wv[q][rg], f8); // exact
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[rg] = mfma16(wf[e], xa[q][e], acc[rg]);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[rg] = mfma16(wf[4 + e], xb[q][e], acc[rg]);
                }
            }
        __builtin_amdgcn_sched_barrier(0); // the next batch's loads stay below
    }

    // on return out[rg] holds D of row group rg
    __device__ __forceinline__ void run(f4 (&out)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        f4 acc[RG], t1[RG], t2[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] = t1[rg] = t2[rg] = z;
        int c0 = 0, n1 = 0;
        for (; c0 + CB <= kn; c0 += CB) {
            batch<false>(c0, acc);
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                t1[rg] += acc[rg];
                acc[rg] = z;
            }
            if (++n1 == kMfmaLevel) {
#pragma unroll
                for (int rg = 0; rg < RG; ++rg) {
                    t2[rg] += t1[rg];
                    t1[rg] = z;
                }
                n1 = 0;
            }
        }
        if (c0 < kn) // every lane reaches the MFMAs
            batch<true>(c0, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            out[rg] = t2[rg] + (t1[rg] + acc[rg]);
    }
};

// One row tile of a several-vector item: WV wavefronts x RG groups of 16
// rows, all nb <= 16 vectors.
template <typename T, int RG, int Q, int WV>
__device__ __forceinline__ void tile_mfma16(const DevItem &it, int row0)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (16 * RG);
    if (wrow0 >= it.M) return;
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f4 out[RG];
    const Mfma16Rows<T, RG, Q> mr(static_cast<const T *>(it.W), it.ldw, wrow0, it.M, it.x,
                                  it.ldx, nb, it.K, lane);
    mr.run(out);
    // D[4 g + v][i]: row wrow0 + 16 rg + 4 g + v, vector i
    const int i = lane & 15, g = lane >> 4;
    if (i < nb) {
        float *yv = it.y + (int64_t)i * it.ldy;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wrow0 + 16 * rg + 4 * g + v;
                if (row < it.M) yv[row] = out[rg][v];
            }
    }
}

template <int WM, int RG, int Q, int WV>
__device__ __forceinline__ void tile_mfma16_w(const DevItem &it, int row0)
{
    if constexpr (WM == kWF32)
        tile_mfma16<float, RG, Q, WV>(it, row0);
    else if constexpr (WM == kWF16)
        tile_mfma16<_Float16, RG, Q, WV>(it, row0);
    else if (it.dtype == 1)
        tile_mfma16<_Float16, RG, Q, WV>(it, row0);
    else
        tile_mfma16<float, RG, Q, WV>(it, row0);
}

template <int WM, int RG, int Q, int WV>
__global__ __launch_bounds__(WV *kWave) void k_sweep_mfma16(const DevItem *__restrict__ items,
                                                             const DevTile *__restrict__ tiles,
                                                             int ntiles)
{
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_mfma16_w<WM, RG, Q, WV>(it, tl.row0);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int WM, int RG, int Q, int WV>
__global__ __launch_bounds__(WV *kWave) void k_item_mfma16(const DevItem it)
{
    tile_mfma16_w<WM, RG, Q, WV>(it, (int)blockIdx.x * (16 * RG * WV));
}

// (rows per wavefront = 16 RG, waves per block, Q = loads per row group in
// flight) of the 16 x 16 x 4 form; any number of vectors up to 16.  Q >= 4
// keeps these apart from the 4 x 4 x 1 shapes (U = 1).
#define TVL_MFMA16_SHAPES(X) X(16, 4, 8) X(32, 1, 4) X(32, 2, 4) X(64, 1, 4)

template <int R, int WV, int Q>
struct InstMfma16 {
    static constexpr int RG = R / 16;
    template <int WM>
    static hipError_t sweep_w(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                              hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_mfma16<WM, RG, Q, WV>), dim3(grid), dim3(WV * kWave), 0, st,
                           items, tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t sweep(int wm, const DevItem *items, const DevTile *tiles, int ntiles,
                            int grid, hipStream_t st)
    {
        return wm == kWF32   ? sweep_w<kWF32>(items, tiles, ntiles, grid, st)
               : wm == kWF16 ? sweep_w<kWF16>(items, tiles, ntiles, grid, st)
                             : sweep_w<kWMixed>(items, tiles, ntiles, grid, st);
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (it.dtype == 1)
            hipLaunchKernelGGL((k_item_mfma16<kWF16, RG, Q, WV>), grid, block, 0, st, it);
        else
            hipLaunchKernelGGL((k_item_mfma16<kWF32, RG, Q, WV>), grid, block, 0, st, it);
        return hipGetLastError();
    }
};

// -------------------------------- matrix cores, 16 x 16 x 4, LDS-staged rows
// The same contraction as above with whole-line weight loads: every
// wavefront load covers whole 128-byte lines of the rows.  fp32: lanes 0-31
// bring 512 contiguous bytes of row 2t and lanes 32-63 those of row 2t + 1
// (8 lines); fp16: each 16-lane quarter brings 256 bytes of one of the rows
// 4t .. 4t + 3 (8 lines), converted exactly to fp32 in registers.  The rows
// go to a wavefront-private LDS tile of fp32 values and come back in the
// A-operand layout (lane 16 g + i: row i, 16-byte block 4 q + g).  Rows sit
// 528 bytes apart (512 + 16 of padding), so row i starts 4 i banks further
// on: the 16 lanes reading one 16-byte block of 16 rows hit 16 different
// bank groups, and every LDS access of a chunk is one base register plus an
// immediate offset.  One wavefront's LDS reads follow its writes in order:
// no barrier.  The x vectors keep their direct B-layout loads.
// Accumulation as in the form above, with 32 MFMA steps per chunk.
//
// Which columns an LDS block holds (the x loads follow the same map):
//   fp32: block k holds columns 4k .. 4k + 3 of the chunk;
//   fp16: the lane that loads columns 8j .. 8j + 7 writes their first half
//         to block j and their second half to block 16 + j, so the 16 lanes
//         of a row write 16 consecutive blocks.  Block k < 16 then holds
//         columns 8k .. 8k + 3, block 16 + k columns 8k + 4 .. 8k + 7.
constexpr int kLdsCols = 128;                   // columns per chunk (one LDS row)
constexpr int kLdsRow = kLdsCols / 4 + 1;       // f4 per LDS row, padding included

// Row groups (2 fp32 or 4 fp16 rows, 1 KiB of a chunk) are read through
// buffer descriptors: the descriptor of group t starts at the group's first
// row and holds only its rows below M, so the hardware's range check returns
// zeros for rows past M and every load needs just one 32-bit lane offset in
// a VGPR, the chunk's column in the scalar offset.  A group must then fit in
// the descriptor's 31-bit size: 8 ldw bytes, rows of up to kLdsMaxLdw
// elements (longer rows go to the direct-load form).
constexpr int64_t kLdsMaxLdw = (int64_t(1) << 28) - 64;

template <typename T, int RG>
struct MfmaLdsRows {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int LR = kLdsCols * ES / 16; // lanes per row of a load (16 bytes each)
    static constexpr int RL = kWave / LR;         // rows per load
    static constexpr int NT = 16 / RL * RG;       // loads per chunk
    static_assert(RL * LR == kWave && 16 % RL == 0, "a load covers whole rows of a chunk");
    const T *W;      // the wavefront's first row (wavefront-uniform)
    int64_t ldw;
    const float *xv; // vector i (clamped)
    int vrows, kn, lane;
    int voff; // this lane's byte offset in a row group

    __device__ __forceinline__ MfmaLdsRows(const T *W_, int64_t ldw_, int wrow0, int M,
                                           const float *x, int64_t ldx, int nb, int K, int lane_)
        : W(W_ + (int64_t)wrow0 * ldw_), ldw(ldw_), vrows(M - wrow0), kn(K), lane(lane_),
          voff((int)((lane_ / LR) * ldw_ * ES + 16 * (lane_ % LR)))
    {
        xv = x + (int64_t)min(lane & 15, nb - 1) * ldx;
    }

    // chunk column of x block 4 q + g (the map above)
    static __device__ __forceinline__ int xcol(int q, int g)
    {
        if constexpr (ES == 4)
            return 16 * q + 4 * g;
        else
            return 32 * (q & 3) + 8 * g + 4 * (q >> 2);
    }

    // rows RL t .. RL t + RL - 1 of the wavefront, those below M
    __device__ __forceinline__ __amdgpu_buffer_rsrc_t group(int t) const
    {
        const int n = min(max(vrows - RL * t, 0), RL);
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<T *>(W + RL * t * ldw), (short)0,
                                                 (int)(n * ldw * ES), 0x00020000);
    }

    // one 16-byte load: columns c0 + (16 / ES) (lane % LR) .. of its row,
    // non-temporal (cache policy 2) like load_w
    __device__ __forceinline__ u4 load(int t, int c0) const
    {
        return __builtin_bit_cast(
            u4, __builtin_amdgcn_raw_buffer_load_b128(group(t), voff, ES * c0, 2));
    }

    // tile: this wavefront's 16 LDS rows of kLdsRow float4
    template <bool RAGGED>
    __device__ __forceinline__ void chunk(int c0, f4 *tile, f4 (&acc)[RG]) const
    {
        const int g = lane >> 4, i = lane & 15, b = lane % LR;
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        const u4 zu = {0u, 0u, 0u, 0u};
        u4 w[NT];
        f4 xb[8];
        const int wcol = c0 + (16 / ES) * b;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if constexpr (RAGGED)
                w[t] = wcol < kn ? load(t, c0) : zu;
            else
                w[t] = load(t, c0);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int c = c0 + xcol(q, g);
            if constexpr (RAGGED) {
                const int valid = kn - c;
                xb[q] = valid > 0 ? mask_from<f4, 4>(load_x4(xv + c), valid) : z;
            } else {
                xb[q] = load_x4(xv + c);
            }
        }
        __builtin_amdgcn_sched_barrier(0); // the chunk's loads first
        // one 16-row group at a time through the same 16 LDS rows (a
        // wavefront's LDS accesses run in order: group rg + 1 overwrites
        // rows that group rg has finished reading)
        f4 *wt = tile + (lane / LR) * kLdsRow + b; // row lane / LR, block b
        const f4 *rt = tile + i * kLdsRow + g;      // row i, block g (+ 4 q blocks)
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
#pragma unroll
            for (int t = 0; t < 16 / RL; ++t) {
                const u4 raw = w[16 / RL * rg + t];
                if constexpr (ES == 4) {
                    f4 v = __builtin_bit_cast(f4, raw);
                    if constexpr (RAGGED) v = mask_from<f4, 4>(v, kn - wcol);
                    wt[RL * t * kLdsRow] = v;
                } else {
                    const f8 wf = __builtin_convertvector(__builtin_bit_cast(h8, raw), f8);
                    f4 lo = {wf[0], wf[1], wf[2], wf[3]};
                    f4 hi = {wf[4], wf[5], wf[6], wf[7]};
                    if constexpr (RAGGED) {
                        lo = mask_from<f4, 4>(lo, kn - wcol);
                        hi = mask_from<f4, 4>(hi, kn - wcol - 4);
                    }
                    wt[RL * t * kLdsRow] = lo;
                    wt[RL * t * kLdsRow + 16] = hi;
                }
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const f4 a = rt[4 * q];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[rg] = mfma16(a[e], xb[q][e], acc[rg]);
            }
        }
        __builtin_amdgcn_sched_barrier(0); // the next chunk's loads stay below
    }

    __device__ __forceinline__ void run(f4 *tile, f4 (&out)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        f4 acc[RG], t1[RG], t2[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] = t1[rg] = t2[rg] = z;
        int c0 = 0, n1 = 0;
        for (; c0 + kLdsCols <= kn; c0 += kLdsCols) {
            chunk<false>(c0, tile, acc);
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                t1[rg] += acc[rg];
                acc[rg] = z;
            }
            if (++n1 == kMfmaLevel) {
#pragma unroll
                for (int rg = 0; rg < RG; ++rg) {
                    t2[rg] += t1[rg];
                    t1[rg] = z;
                }
                n1 = 0;
            }
        }
        if (c0 < kn) // every lane reaches the MFMAs
            chunk<true>(c0, tile, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            out[rg] = t2[rg] + (t1[rg] + acc[rg]);
    }
};

template <typename T, int RG, int WV>
__device__ __forceinline__ void tile_mfma_lds(const DevItem &it, int row0, f4 *tile)
{
    if (it.ldw > kLdsMaxLdw) { // wavefront-uniform
        tile_mfma16<T, RG, 4, WV>(it, row0);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (16 * RG);
    if (wrow0 >= it.M) return; // no barrier follows
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f4 out[RG];
    const MfmaLdsRows<T, RG> mr(static_cast<const T *>(it.W), it.ldw, wrow0, it.M, it.x, it.ldx,
                                nb, it.K, lane);
    mr.run(tile, out);
    const int i = lane & 15, g = lane >> 4;
    if (i < nb) {
        float *yv = it.y + (int64_t)i * it.ldy;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wrow0 + 16 * rg + 4 * g + v;
                if (row < it.M) yv[row] = out[rg][v];
            }
    }
}

template <int WM, int RG, int WV>
__device__ __forceinline__ void tile_mfma_lds_w(const DevItem &it, int row0, f4 *tile)
{
    if constexpr (WM == kWF32)
        tile_mfma_lds<float, RG, WV>(it, row0, tile);
    else if constexpr (WM == kWF16)
        tile_mfma_lds<_Float16, RG, WV>(it, row0, tile);
    else if (it.dtype == 1)
        tile_mfma_lds<_Float16, RG, WV>(it, row0, tile);
    else
        tile_mfma_lds<float, RG, WV>(it, row0, tile);
}

template <int WM, int RG, int WV>
__global__ __launch_bounds__(WV *kWave) void k_sweep_mfma_lds(const DevItem *__restrict__ items,
                                                               const DevTile *__restrict__ tiles,
                                                               int ntiles)
{
    constexpr int kTile = 16 * kLdsRow; // f4 per wavefront
    __shared__ f4 lds[WV * kTile];
    f4 *tile = lds + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave) * kTile;
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_mfma_lds_w<WM, RG, WV>(it, tl.row0, tile);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int WM, int RG, int WV>
__global__ __launch_bounds__(WV *kWave) void k_item_mfma_lds(const DevItem it)
{
    constexpr int kTile = 16 * kLdsRow;
    __shared__ f4 lds[WV * kTile];
    f4 *tile = lds + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave) * kTile;
    tile_mfma_lds_w<WM, RG, WV>(it, (int)blockIdx.x * (16 * RG * WV), tile);
}

// ------------------- matrix cores, 16 x 16 x 4, weights streamed into LDS
// The same contraction with the weight loads writing LDS directly: a buffer
// load with the LDS bit puts lane l's 16 bytes at M0 + 16 l and holds no
// VGPR, so with S LDS stages a wavefront keeps S - 1 chunks in flight while
// it multiplies the current one.  One load covers 1 KiB: the chunk of RPL
// rows (CC columns, RB = CC * sizeof(T) bytes each), lane l landing in row
// l / LPR at 16-byte position l % LPR.  Rows are stored without padding, so
// the blocks of row r are XOR-swizzled (the lane at position p reads block
// p ^ f(r)) such that the 16 lanes that read one column block of 16 rows hit
// the 16 different 16-byte bank groups of a 256-byte LDS line: f(r) = r for
// rows of 256 bytes or more, f(r) = r / 2 for 128-byte rows (two rows per
// line).  fp16 weights stay fp16 in LDS: the A operand of a step is then 8
// bytes (4 columns), converted exactly after the LDS read.  x: direct
// B-layout loads S - 2 chunks ahead, in S - 1 register buffers; more rows
// per wavefront share each x load (x from the cache adds nb 4 CC bytes per
// chunk of 16 RG rows to the weights' 16 RG RB).
//
// Chunk step c issues, in this order, the x loads of chunk c + S - 2 (NQ)
// and the weight loads of chunk c + S - 1 (NL); near the end of the rows the
// same loads go to empty descriptors (no memory access; they fill a stage
// that is no longer read) and to the last chunk's x.  So (S - 1)(NQ + NL)
// loads always follow a chunk's weight loads when its products start, and
// one fixed vmcnt wait brings them in while S - 1 chunks stay in flight (the
// compiler's own waits for x, NQ loads stricter, leave the same chunks in
// flight; the compiler does not track these loads' LDS writes).  A ragged
// last chunk drains the loads and goes through registers (masked) into the
// same layout.  Accumulation as in the forms above (4 NQ MFMA steps per
// chunk).
#define TVL_LDS __attribute__((address_space(3)))

// 16 bytes per lane from a buffer into LDS at lds + 16 lane; weights
// non-temporal (cache policy 2, streamed once), x (NT = false) with the
// default policy (every block of a matrix reads it)
template <bool NT = true>
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t r, TVL_LDS void *lds, int voff,
                                          int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, voff, soff, 0, NT ? 2 : 0);
}

typedef _Float16 h4 __attribute__((ext_vector_type(4)));

// fp16 weights on the fp16 matrix cores (HX): each chunk's x values are
// scaled per vector by a power of two 2^k (k = 14 - e for the chunk's
// largest |x| in [2^(e-1), 2^e), clamped to +-126), which puts the largest
// in [2^13, 2^14), far below the fp16 maximum, and split into a high and a
// low fp16 part, both rounded to nearest: x 2^k = hi + lo + r with
// |r| <= 2^-11 |x 2^k - hi| <= 2^-22 |x 2^k| while lo is normal, and
// |r| <= 2^-25 (half the smallest fp16 subnormal) below.  Products of fp16 values are
// exact in fp32, so one v_mfma_f32_16x16x32_f16 per part does the work of
// eight fp32 16 x 16 x 4 steps; the chunk's sum is then scaled back by 2^-k
// (exact).  A operand: lane 16 g + i holds row i, columns 8 g .. 8 g + 7 of
// the 32-column step (one 16-byte LDS read); B: vector i, the same columns.
//
// The absolute 2^-25 would lose the small entries of a chunk whose range is
// wider than the two parts hold (an entry 2^40 beside ones rounds the ones
// to zero), and S = sum_j |W_ij x_j| need not see the large entry (its
// weight may be zero), so such a chunk runs on the fp32 matrix cores
// instead: any nonzero |x 2^k| below kSplitMin in any vector of the
// wavefront sends the whole chunk there.  On the split path every entry then
// has |r| <= max(2^-22, 2^-25 / kSplitMin) |x 2^k| = 2^-18 |x 2^k|, so the
// split adds at most 2^-18 S to the fp32 forms' error bound, for any finite
// x.  For x ~ N(0, 1), ~0.3 % of 128-column chunks of 16 vectors take the
// fp32 path (each costs four times the matrix-core steps of a split chunk).
constexpr float kSplitMin = 0x1p-7f;
// (The range test reads each x value's bits with __float_as_uint on the
// element's value: this compiler lowers __builtin_bit_cast of a vector
// element such as xb[q][e] to the bits of element 0, which would test only
// every fourth column.)

__device__ __forceinline__ f4 mfma16h(h8 a, h8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

template <typename T, int RG, int CC, int S, bool HX = false>
struct MfmaDmaRows {
    static_assert(!HX || sizeof(T) == 2, "split x with fp16 weights only");
    static constexpr int ES = (int)sizeof(T);
    static constexpr int RB = CC * ES;         // bytes of a row's chunk (one LDS row)
    static constexpr int RPL = 1024 / RB;      // rows per load
    static constexpr int LPR = kWave / RPL;    // lanes (16-byte positions) per row
    static constexpr int TPG = 16 / RPL;       // loads per 16-row group
    static constexpr int NL = TPG * RG;        // weight loads per chunk
    static constexpr int NQ = CC / 16;         // x loads and MFMA column steps per chunk
    static constexpr int STAGE = 16 * RG * RB; // bytes per stage
    static constexpr int kStages = S;
    static constexpr int NX = S - 1; // x buffers
    static constexpr int WAIT = (S - 1) * (NL + NQ);
    static constexpr int SH = RB < 256 ? 1 : 0; // rows per 256-byte line, log2
    // RPL rows in a buffer descriptor's 31-bit size
    static constexpr int64_t MAXLDW = (int64_t(1) << 31) / (ES * RPL) - 64;
    static_assert(RB >= 128 && LPR * RPL == kWave && S >= 3 && WAIT < 64, "chunk shape");

    // the swizzle of row r (0..15 in its group)
    static __device__ __forceinline__ int swz(int r) { return (r >> SH) & (LPR - 1); }

    const T *W; // the wavefront's first row (wavefront-uniform)
    int64_t ldw;
    const float *xv; // vector i (clamped), at column 4 g (8 g with HX)
    int vrows, kn, lane;
    TVL_LDS char *lds; // this wavefront's stages
    int voff[TPG];     // per load of a row group: the lane's byte offset in it
    int raddr[NQ];     // per MFMA column step: the lane's A operand in a stage

    // chunk column of the lane's x load k, relative to xv
    static __device__ __forceinline__ int xoff(int k)
    {
        return HX ? 32 * (k >> 1) + 4 * (k & 1) : 16 * k;
    }

    __device__ __forceinline__ MfmaDmaRows(const T *W_, int64_t ldw_, int wrow0, int M,
                                           const float *x, int64_t ldx, int nb, int K, int lane_,
                                           TVL_LDS char *lds_)
        : W(W_ + (int64_t)wrow0 * ldw_), ldw(ldw_), vrows(M - wrow0), kn(K), lane(lane_),
          lds(lds_)
    {
        xv = x + (int64_t)min(lane & 15, nb - 1) * ldx + (HX ? 8 : 4) * (lane >> 4);
        const int h = lane / LPR, p = lane % LPR, g = lane >> 4, i = lane & 15;
#pragma unroll
        for (int t = 0; t < TPG; ++t)
            voff[t] = (int)(h * ldw_ * ES) + 16 * (p ^ swz(RPL * t + h));
        // columns 16 q + 4 g .. + 3 of row i: 16-byte block 4 q + g (fp32),
        // the (g & 1) half of block 2 q + g / 2 (fp16); HX: columns
        // 32 q + 8 g .. + 7, block 4 q + g
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            raddr[q] = ES == 4 || HX
                           ? i * RB + 16 * ((4 * q + g) ^ swz(i))
                           : i * RB + 16 * ((2 * q + (g >> 1)) ^ swz(i)) + 8 * (g & 1);
    }

    // rows RPL j .. RPL j + RPL - 1 of the wavefront, those below M; none if
    // !live
    __device__ __forceinline__ __amdgpu_buffer_rsrc_t group(int j, bool live) const
    {
        const int n = live ? min(max(vrows - RPL * j, 0), RPL) : 0;
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<T *>(W + RPL * j * ldw), (short)0,
                                                 (int)(n * ldw * ES), 0x00020000);
    }

    // the chunk at column c0 into stage ST (non-temporal, cache policy 2)
    template <int ST>
    __device__ __forceinline__ void issue(int c0, bool live) const
    {
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int t = 0; t < TPG; ++t)
                lds_dma16(group(TPG * rg + t, live),
                          (TVL_LDS void *)(lds + ST * STAGE + rg * 16 * RB + t * 1024), voff[t],
                          ES * c0);
    }

    __device__ __forceinline__ void load_x(int c0, f4 (&xb)[NQ]) const
    {
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            xb[q] = load_x4(xv + c0 + xoff(q));
    }

    template <int ST>
    __device__ __forceinline__ void multiply(const f4 (&xb)[NQ], f4 (&acc)[RG]) const
    {
        if constexpr (HX) {
            multiply_hx<ST>(xb, acc);
            return;
        }
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const TVL_LDS char *ap = lds + ST * STAGE + rg * 16 * RB + raddr[q];
                f4 a;
                if constexpr (ES == 4)
                    a = *(const TVL_LDS f4 *)ap;
                else // exact conversion
                    a = __builtin_convertvector(*(const TVL_LDS h4 *)ap, f4);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[rg] = mfma16(a[e], xb[q][e], acc[rg]);
            }
    }

    // HX: the chunk's products on the fp16 matrix cores (scaled, split x),
    // or on the fp32 ones when the chunk's range is too wide (kSplitMin)
    template <int ST>
    __device__ __forceinline__ void multiply_hx(const f4 (&xb)[NQ], f4 (&acc)[RG]) const
    {
        // the vector's largest |x| over its 4 lanes (g = 0..3 hold the
        // chunk's columns) sets the scale
        float m = 0.f;
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                m = fmaxf(m, fabsf(xb[q][e]));
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        int e2 = 0;
        if (m > 0.f && m <= 3.4028235e38f) e2 = __builtin_amdgcn_frexp_expf(m);
        const int k = min(max(14 - e2, -126), 126);
        const float sc = __builtin_ldexpf(1.f, k), inv = __builtin_ldexpf(1.f, -k);
        // the split path first (speculatively: a chunk too wide for it, rare,
        // is redone below and this result dropped), so the range check does
        // not stand between the scale and the matrix-core steps.
        // hi = f16(x 2^k), lo = f16(x 2^k - hi): each one fused multiply-add
        // with an fp16 result (v_fma_mix); x 2^k is exact (a power of two)
        h8 hi[NQ / 2], lo[NQ / 2];
#pragma unroll
        for (int q = 0; q < NQ / 2; ++q)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float xv = xb[2 * q + e / 4][e % 4];
                const _Float16 vh = (_Float16)__builtin_fmaf(xv, sc, 0.f);
                hi[q][e] = vh;
                lo[q][e] = (_Float16)__builtin_fmaf(xv, sc, -(float)vh);
            }
        f4 cs[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            f4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < NQ / 2; ++q) {
                const h8 a = *(const TVL_LDS h8 *)(lds + ST * STAGE + rg * 16 * RB + raddr[q]);
                c = mfma16h(a, hi[q], c);
                c = mfma16h(a, lo[q], c);
            }
            cs[rg] = c;
        }
        // a nonzero |x| below kSplitMin 2^-k (a power of two, >= 2^-131)?
        // Only if the lane's smallest |x| is below it: then (rare for dense
        // x) look again without the zeros, as (bits << 1) - 2, where the sign
        // bit drops out, magnitudes keep their order and zero wraps to the top
        // (four independent running minima keep the chain short)
        float mzq[4] = {3.4028235e38f, 3.4028235e38f, 3.4028235e38f, 3.4028235e38f};
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                mzq[q & 3] = fminf(mzq[q & 3], fabsf(xb[q][e]));
        const float mz = fminf(fminf(mzq[0], mzq[1]), fminf(mzq[2], mzq[3]));
        const float thr = __builtin_ldexpf(kSplitMin, -k);
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(mz < thr) != 0, 0)) { // wave-uniform
            uint32_t mn = 0xFFFFFFFFu;
#pragma unroll
            for (int q = 0; q < NQ; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    mn = min(mn, (__float_as_uint(xb[q][e]) << 1) - 2u);
            const bool wide = mn < (__builtin_bit_cast(uint32_t, thr) << 1) - 2u;
            if (__builtin_amdgcn_ballot_w64(wide) != 0) { // wave-uniform
                // fp32 matrix cores: step e multiplies column 8 g + e of the
                // lane's 8 weights (converted exactly) by the same column of x
#pragma unroll
                for (int rg = 0; rg < RG; ++rg) {
                    f4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int q = 0; q < NQ / 2; ++q) {
                        const h8 a =
                            *(const TVL_LDS h8 *)(lds + ST * STAGE + rg * 16 * RB + raddr[q]);
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            c = mfma16((float)a[e], xb[2 * q + e / 4][e % 4], c);
                    }
                    acc[rg] += c;
                }
                return;
            }
        }
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] += cs[rg] * inv;
    }

    // one chunk step: chunk c (stage ST = c % S, x buffer XB = c % NX);
    // true after the last full chunk
    template <int ST, int XB>
    __device__ __forceinline__ bool step(int &c, int nfull, f4 (&xs)[NX][NQ], f4 (&acc)[RG],
                                         f4 (&t1)[RG], f4 (&t2)[RG], int &n1) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        load_x(min(c + S - 2, nfull - 1) * CC, xs[(XB + S - 2) % NX]);
        issue<(ST + S - 1) % S>((c + S - 1) * CC, c + S - 1 < nfull);
        __builtin_amdgcn_sched_barrier(0);
        // vmcnt(WAIT): expcnt and lgkmcnt left alone
        __builtin_amdgcn_s_waitcnt((WAIT & 15) | ((WAIT >> 4) << 14) | 0x0F70);
        __builtin_amdgcn_sched_barrier(0);
        multiply<ST>(xs[XB], acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            t1[rg] += acc[rg];
            acc[rg] = z;
        }
        if (++n1 == kMfmaLevel) {
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                t2[rg] += t1[rg];
                t1[rg] = z;
            }
            n1 = 0;
        }
        __builtin_amdgcn_sched_barrier(0);
        return ++c == nfull;
    }

    // S NX steps: stages and x buffers back where they started
    template <int... J>
    __device__ __forceinline__ bool turn(std::integer_sequence<int, J...>, int &c, int nfull,
                                         f4 (&xs)[NX][NQ], f4 (&acc)[RG], f4 (&t1)[RG],
                                         f4 (&t2)[RG], int &n1) const
    {
        return (step<J % S, J % NX>(c, nfull, xs, acc, t1, t2, n1) || ...);
    }

    // prologue: after the weights of chunk 0, x of chunk j - 1 and the
    // weights of chunk j for j = 1 .. S - 2
    template <int... J>
    __device__ __forceinline__ void start(std::integer_sequence<int, J...>, int nfull,
                                          f4 (&xs)[NX][NQ]) const
    {
        ((load_x(min(J, nfull - 1) * CC, xs[J]), issue<J + 1>((J + 1) * CC, J + 1 < nfull)),
         ...);
    }

    // the ragged last chunk at c0 (after every load has landed), through
    // registers into stage 0
    __device__ __forceinline__ void tail(int c0, f4 (&acc)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        const int h = lane / LPR, p = lane % LPR, g = lane >> 4;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int t = 0; t < TPG; ++t) {
                const int wcol = c0 + 16 / ES * (p ^ swz(RPL * t + h));
                u4 w = {0u, 0u, 0u, 0u};
                if (wcol < kn) {
                    w = __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(
                                                   group(TPG * rg + t, true), voff[t], ES * c0, 2));
                    if constexpr (ES == 4)
                        w = __builtin_bit_cast(
                            u4, mask_from<f4, 4>(__builtin_bit_cast(f4, w), kn - wcol));
                    else
                        w = __builtin_bit_cast(
                            u4, mask_from<h8, 8>(__builtin_bit_cast(h8, w), kn - wcol));
                }
                *(TVL_LDS u4 *)(lds + rg * 16 * RB + t * 1024 + 16 * lane) = w;
            }
        f4 xb[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int valid = kn - (c0 + xoff(q) + (HX ? 8 : 4) * g);
            xb[q] = valid > 0 ? mask_from<f4, 4>(load_x4(xv + c0 + xoff(q)), valid) : z;
        }
        multiply<0>(xb, acc);
    }

    __device__ __forceinline__ void run(f4 (&out)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        f4 acc[RG], t1[RG], t2[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] = t1[rg] = t2[rg] = z;
        const int nfull = kn / CC;
        int c = 0, n1 = 0;
        if (nfull > 0) {
            f4 xs[NX][NQ];
            issue<0>(0, true);
            start(std::make_integer_sequence<int, S - 2>{}, nfull, xs);
            while (!turn(std::make_integer_sequence<int, S * NX>{}, c, nfull, xs, acc, t1, t2, n1)) {
            }
            __builtin_amdgcn_s_waitcnt(0x0F70); // the empty loads too, before LDS is reused
        }
        if (c * CC < kn)
            tail(c * CC, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            out[rg] = t2[rg] + (t1[rg] + acc[rg]);
    }
};

// lds: this wavefront's stages
template <typename T, int RG, int WV, int CC, int S, bool HX>
__device__ __forceinline__ void tile_mfma_dma(const DevItem &it, int row0, TVL_LDS char *lds)
{
    using Rows = MfmaDmaRows<T, RG, CC, S, HX>;
    if (it.ldw > Rows::MAXLDW) { // wavefront-uniform
        tile_mfma16<T, RG, 4, WV>(it, row0);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (16 * RG);
    if (wrow0 >= it.M) return; // no barrier follows
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f4 out[RG];
    const Rows mr(static_cast<const T *>(it.W), it.ldw, wrow0, it.M, it.x, it.ldx, nb, it.K,
                  lane, lds);
    mr.run(out);
    const int i = lane & 15, g = lane >> 4;
    if (i < nb) {
        float *yv = it.y + (int64_t)i * it.ldy;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wrow0 + 16 * rg + 4 * g + v;
                if (row < it.M) yv[row] = out[rg][v];
            }
    }
}

// x shared by the wavefronts of a block (fp32 weights, three stages).  The
// WV wavefronts of a block work on one row tile, so they need the same x
// chunks: each loads 1/WV of every x chunk into a shared LDS ring (buffer
// loads with the LDS bit, vector v in an LDS row of CC * 4 bytes, swizzled
// like the weight rows), and the B operand comes from there.  L1/L2 then
// deliver nb 4 CC x bytes per chunk of the block's 16 RG WV rows instead of
// per wavefront.  One s_barrier per chunk step: after a wavefront's own loads
// of chunk c have landed (vmcnt) every wavefront's have, and every
// wavefront has finished chunk c - 1, whose stages (x shared, weights
// private) the step's new loads overwrite.  Every wavefront of the block
// takes part in every barrier: wavefronts with no rows left stream empty
// descriptors and store nothing, and all choices of path depend only on the
// item.
template <typename T, int RG, int CC, int WV, bool HX>
struct MfmaDmaXsRows : MfmaDmaRows<T, RG, CC, 3, HX> {
    using Base = MfmaDmaRows<T, RG, CC, 3, HX>;
    using Base::NL;
    using Base::NQ;
    using Base::STAGE;
    static constexpr int XRB = CC * 4;             // bytes of a vector's chunk (an x LDS row)
    static constexpr int XVPL = 1024 / XRB;        // vectors per x load
    static constexpr int XLPR = kWave / XVPL;      // lanes per vector of an x load
    static constexpr int XNL = 16 / XVPL;          // x loads per chunk, whole block
    static constexpr int XW = (XNL + WV - 1) / WV; // x loads per chunk, per wavefront (at most)
    static constexpr int XSTAGE = 16 * XRB;        // bytes of an x stage (16 vectors)
    static constexpr int WAIT = NL + XW;           // loads of one chunk step (at most)
    static constexpr int64_t MAXLDX = (int64_t(1) << 31) / (4 * XVPL) - 64;
    static_assert(XRB >= 256 && ((XNL % WV == 0) || XW == 1) && WAIT < 64,
                  "x rows of >= 256 bytes; x loads: all or one per wavefront");

    // x rows are >= 256 bytes: the swizzle of vector v is v itself
    static __device__ __forceinline__ int xswz(int v) { return v & (XLPR - 1); }

    const float *X; // vector 0 of the item
    int64_t ldx;
    int nb, wave;
    TVL_LDS char *xlds; // the block's x stages
    int xvoff[XW];      // per x load of this wavefront: the lane's byte offset
    int xraddr[NQ];     // per x operand load: the lane's 16 bytes in an x stage

    __device__ __forceinline__ MfmaDmaXsRows(const T *W_, int64_t ldw_, int wrow0, int M,
                                             const float *x, int64_t ldx_, int nb_, int K,
                                             int lane_, int wave_, TVL_LDS char *lds_,
                                             TVL_LDS char *xlds_)
        : Base(W_, ldw_, wrow0, M, x, ldx_, nb_, K, lane_, lds_), X(x), ldx(ldx_), nb(nb_),
          wave(wave_), xlds(xlds_)
    {
        const int h = lane_ / XLPR, p = lane_ % XLPR, g = lane_ >> 4, j = lane_ & 15;
#pragma unroll
        for (int u = 0; u < XW; ++u) {
            const int v = XVPL * (wave_ + WV * u) + h; // vector, < 16 when loaded
            xvoff[u] = (int)(h * ldx_ * 4) + 16 * (p ^ xswz(v));
        }
        // the B operand's columns (Base::xoff(k) + 4 or 8 g): 16-byte block
        // 4 k + g, or with HX 8 (k / 2) + 2 g + k % 2, of vector j's row
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            const int blk = HX ? 8 * (k >> 1) + 2 * g + (k & 1) : 4 * k + g;
            xraddr[k] = j * XRB + 16 * (blk ^ xswz(j));
        }
    }

    // vectors XVPL j .. XVPL j + XVPL - 1 below nb; none if !live
    __device__ __forceinline__ __amdgpu_buffer_rsrc_t xgroup(int j, bool live) const
    {
        const int n = live ? min(max(nb - XVPL * j, 0), XVPL) : 0;
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(X + XVPL * j * ldx), (short)0,
                                                 (int)(n * ldx * 4), 0x00020000);
    }

    // x loads this wavefront issues per chunk: XW, or (more wavefronts than x
    // loads) 1 for the first XNL wavefronts and 0 for the others
    __device__ __forceinline__ bool loads_x() const { return XNL % WV == 0 || wave < XNL; }

    // this wavefront's share of the weights (all its rows) and of x for the
    // chunk at c0, into stage ST
    template <int ST>
    __device__ __forceinline__ void issue_all(int c0, bool live) const
    {
        Base::template issue<ST>(c0, live);
        if (!loads_x()) return; // wavefront-uniform
#pragma unroll
        for (int u = 0; u < XW; ++u) {
            const int j = wave + WV * u;
            lds_dma16<false>(xgroup(j, live), (TVL_LDS void *)(xlds + ST * XSTAGE + j * 1024),
                             xvoff[u], 4 * c0);
        }
    }

    template <int ST>
    __device__ __forceinline__ bool step(int &c, int nfull, f4 (&acc)[RG], f4 (&t1)[RG],
                                         f4 (&t2)[RG], int &n1) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_sched_barrier(0);
        // vmcnt(loads of one step): this wavefront's loads of chunk c have landed
        if (loads_x())
            __builtin_amdgcn_s_waitcnt((WAIT & 15) | ((WAIT >> 4) << 14) | 0x0F70);
        else
            __builtin_amdgcn_s_waitcnt((NL & 15) | ((NL >> 4) << 14) | 0x0F70);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        issue_all<(ST + 2) % 3>((c + 2) * CC, c + 2 < nfull);
        __builtin_amdgcn_sched_barrier(0);
        f4 xb[NQ];
#pragma unroll
        for (int k = 0; k < NQ; ++k)
            xb[k] = *(const TVL_LDS f4 *)(xlds + ST * XSTAGE + xraddr[k]);
        Base::template multiply<ST>(xb, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            t1[rg] += acc[rg];
            acc[rg] = z;
        }
        if (++n1 == kMfmaLevel) {
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                t2[rg] += t1[rg];
                t1[rg] = z;
            }
            n1 = 0;
        }
        __builtin_amdgcn_sched_barrier(0);
        return ++c == nfull;
    }

    __device__ __forceinline__ void run(f4 (&out)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        f4 acc[RG], t1[RG], t2[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] = t1[rg] = t2[rg] = z;
        const int nfull = this->kn / CC;
        int c = 0, n1 = 0;
        // the previous tile's readers of the shared stages are done
        __builtin_amdgcn_s_barrier();
        if (nfull > 0) {
            issue_all<0>(0, true);
            issue_all<1>(CC, nfull > 1);
            for (;;) {
                if (step<0>(c, nfull, acc, t1, t2, n1)) break;
                if (step<1>(c, nfull, acc, t1, t2, n1)) break;
                if (step<2>(c, nfull, acc, t1, t2, n1)) break;
            }
            __builtin_amdgcn_s_waitcnt(0x0F70); // the empty loads too
        }
        if (c * CC < this->kn) // private: weights stage 0, x in registers
            Base::tail(c * CC, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            out[rg] = t2[rg] + (t1[rg] + acc[rg]);
    }
};

// DPP move within rows of 16 lanes (CTRL: quad permutation 0x00-0xFF,
// 0x140 row mirror, 0x141 half-row mirror)
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}

// the largest of v >= 0 (not NaN) over each group of N consecutive lanes (N =
// 4, 8, 16, 32), in every lane of the group, as the largest bit pattern (the
// order of non-negative floats): lane pairs and quads by quad permutations,
// then half rows and rows by mirrors (each lane meets a lane of the other
// half), then across two rows by one lane exchange
template <int N>
__device__ __forceinline__ float group_max(float v)
{
    static_assert(N == 4 || N == 8 || N == 16 || N == 32, "group of 4 .. 32 lanes");
    uint32_t u = __builtin_bit_cast(uint32_t, v);
    u = max(u, dpp_u32<0xB1>(u)); // quad permutation 1 0 3 2
    u = max(u, dpp_u32<0x4E>(u)); // quad permutation 2 3 0 1
    if constexpr (N >= 8) u = max(u, dpp_u32<0x141>(u));
    if constexpr (N >= 16) u = max(u, dpp_u32<0x140>(u));
    if constexpr (N == 32) u = max(u, (uint32_t)__shfl_xor((int)u, 16));
    return __builtin_bit_cast(float, u);
}

// fp16 weights with x split once per block (the split-x form with x shared
// by the block).  The WV wavefronts of a block need the same split x, and the
// analysis and split of a chunk cost more vector operations than its
// matrix-core steps: so each wavefront splits only vectors VPW w .. VPW w +
// VPW - 1 (LPV lanes per vector, CPL columns per lane), one chunk ahead, from
// x it loads into registers, and writes the two fp16 parts straight into the
// B-operand layout in LDS: MFMA lane L = 16 g + j at 32-column step s finds
// columns 32 s + 8 g .. + 7 of vector j in the 256-byte row s * 4 + g of a
// part, at 16-byte slot j ^ h(s, g), h = (4 s + g) * 4 / NS.  Without the XOR
// the 16 lanes writing one vector's columns would all hit one slot position
// (16-way bank conflicts); with it writers and readers each touch 16
// distinct slots per 256 bytes (checked on the CPU for every shape).  With
// the parts go each vector's 2^-k and a flag per wavefront for a chunk too
// wide for the split (kSplitMin).  After the next step's barrier every wavefront reads
// its B operands there.  Each value is scaled and split exactly as in the
// per-wavefront form (the same per-vector maximum), and the matrix-core
// steps are the same, so the results are the same bit for bit; a chunk any
// wavefront flagged goes to the fp32 matrix cores with x read from global
// memory (rare for dense x).  Per chunk step (c): wait for the weights of c
// and this wavefront's x of c + 1 (the weights of c + 1 stay in flight), one
// s_barrier, issue x of c + 2 (registers) and the weights of c + 2, issue the
// matrix-core steps of chunk c (weight stage c % 3, split stage c % 2), split
// x of c + 1 into split stage (c + 1) % 2 while they run, then add chunk c's
// products.  The barrier of step c + 1 separates the writes of a split stage
// from the reads of the step before and after.  The maximum over a vector's
// lanes uses DPP moves (no LDS round trips on the split's critical path).
template <int RG, int CC, int WV>
struct MfmaXsHxRows : MfmaDmaRows<_Float16, RG, CC, 3, true> {
    using Base = MfmaDmaRows<_Float16, RG, CC, 3, true>;
    using Base::NL;
    using Base::STAGE;
    static constexpr int NS = CC / 32;        // 32-column matrix-core steps per chunk
    static constexpr int VPW = 16 / WV;       // vectors split by each wavefront
    static constexpr int LPV = kWave / VPW;   // lanes per vector
    static constexpr int CPL = CC / LPV;      // columns per lane
    static constexpr int XL = CPL / 4;        // 16-byte x loads per lane per chunk
    static constexpr int HPART = NS * 1024;   // bytes of one fp16 part of a chunk
    static constexpr int HSCALE = 2 * HPART;  // 16 floats: 2^-k of each vector
    static constexpr int HFLAG = HSCALE + 64; // WV ints: a wavefront found a wide chunk
    static constexpr int HSTAGE = (HFLAG + 4 * WV + 15) / 16 * 16;
    static constexpr int64_t MAXLDX = int64_t(1) << 62; // x is read through plain pointers
    static_assert(CPL == 4 || CPL == 8 || CPL == 16, "columns per lane");
    static_assert(2 * NL + XL < 64, "vmcnt range");

    const float *X; // vector 0 of the item
    int64_t ldx;
    int nb, wave;
    TVL_LDS char *hl; // the block's two split stages
    const float *xs;             // this lane's vector (clamped to nb - 1) at its first column
    static constexpr int PC = CPL < 8 ? CPL : 8; // columns per LDS write
    int woff[CPL / PC];          // byte offset in a part of each write of the lane
    int roff[NS];                // byte offset in a part of the B operand of each step

    // the 16-byte slot of (step s, 8-column group g, vector v) in a part
    static __device__ __forceinline__ int slot(int s, int g, int v)
    {
        return s * 1024 + g * 256 + 16 * (v ^ ((4 * s + g) * (4 / NS)));
    }

    __device__ __forceinline__ MfmaXsHxRows(const _Float16 *W_, int64_t ldw_, int wrow0, int M,
                                            const float *x, int64_t ldx_, int nb_, int K,
                                            int lane_, int wave_, TVL_LDS char *lds_,
                                            TVL_LDS char *hl_)
        : Base(W_, ldw_, wrow0, M, x, ldx_, nb_, K, lane_, lds_), X(x), ldx(ldx_), nb(nb_),
          wave(wave_), hl(hl_)
    {
        // vectors past nb repeat vector nb - 1, as in the per-wavefront
        // form: same scale and range decisions, columns never stored
        const int v = VPW * wave_ + lane_ / LPV, col = (lane_ % LPV) * CPL;
        xs = x + (int64_t)min(v, nb_ - 1) * ldx_ + col;
#pragma unroll
        for (int p = 0; p < CPL / PC; ++p) { // the next 8 columns: group g + 1
            const int c8 = col + p * PC;
            woff[p] = slot(c8 / 32, (c8 % 32) / 8, v) + 2 * (c8 % 8);
        }
#pragma unroll
        for (int q = 0; q < NS; ++q)
            roff[q] = slot(q, lane_ >> 4, lane_ & 15);
    }

    // this lane's x of chunk c
    __device__ __forceinline__ void load_xs(int c, f4 (&xr)[XL]) const
    {
#pragma unroll
        for (int u = 0; u < XL; ++u)
            xr[u] = load_x4(xs + c * CC + 4 * u);
    }

    // scale and split this lane's x into split stage HS (see MfmaDmaRows'
    // multiply_hx for the arithmetic and the range test)
    template <int HS>
    __device__ __forceinline__ void split(const f4 (&xr)[XL]) const
    {
        float m = 0.f, mz = 3.4028235e38f;
#pragma unroll
        for (int u = 0; u < XL; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                m = fmaxf(m, fabsf(xr[u][e]));
                mz = fminf(mz, fabsf(xr[u][e]));
            }
        m = group_max<LPV>(m); // the vector's lanes are consecutive; m >= 0, never NaN
        int e2 = 0;
        if (m > 0.f && m <= 3.4028235e38f) e2 = __builtin_amdgcn_frexp_expf(m);
        const int k = min(max(14 - e2, -126), 126);
        const float sc = __builtin_ldexpf(1.f, k);
        const float thr = __builtin_ldexpf(kSplitMin, -k);
        bool wide = false;
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(mz < thr) != 0, 0)) { // wave-uniform
            uint32_t mn = 0xFFFFFFFFu;
#pragma unroll
            for (int u = 0; u < XL; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    mn = min(mn, (__float_as_uint(xr[u][e]) << 1) - 2u);
            wide = mn < (__builtin_bit_cast(uint32_t, thr) << 1) - 2u;
        }
        const int any = __builtin_amdgcn_ballot_w64(wide) != 0; // all lanes take part
        TVL_LDS char *hb = hl + HS * HSTAGE;
        const int lane = this->lane;
        if (lane == 0) *(TVL_LDS int *)(hb + HFLAG + 4 * wave) = any;
        if (lane % LPV == 0)
            ((TVL_LDS float *)(hb + HSCALE))[VPW * wave + lane / LPV] = __builtin_ldexpf(1.f, -k);
        // hi = f16(x 2^k), lo = f16(x 2^k - hi), CPL values, in pieces of up
        // to 8 columns (one B-operand slot each)
#pragma unroll
        for (int p = 0; p < CPL / PC; ++p) {
            _Float16 hv[PC], lv[PC];
#pragma unroll
            for (int e = 0; e < PC; ++e) {
                const float xv = xr[(p * PC + e) / 4][(p * PC + e) % 4];
                const _Float16 vh = (_Float16)__builtin_fmaf(xv, sc, 0.f);
                hv[e] = vh;
                lv[e] = (_Float16)__builtin_fmaf(xv, sc, -(float)vh);
            }
            const int off = woff[p];
            if constexpr (PC == 8) {
                *(TVL_LDS h8 *)(hb + off) = h8{hv[0], hv[1], hv[2], hv[3], hv[4], hv[5], hv[6], hv[7]};
                *(TVL_LDS h8 *)(hb + HPART + off) =
                    h8{lv[0], lv[1], lv[2], lv[3], lv[4], lv[5], lv[6], lv[7]};
            } else {
                *(TVL_LDS h4 *)(hb + off) = h4{hv[0], hv[1], hv[2], hv[3]};
                *(TVL_LDS h4 *)(hb + HPART + off) = h4{lv[0], lv[1], lv[2], lv[3]};
            }
        }
    }

    // some wavefront found chunk c too wide for the split (split stage HS)
    template <int HS>
    __device__ __forceinline__ bool wide_chunk() const
    {
        const TVL_LDS char *hb = hl + HS * HSTAGE;
        int wide = 0;
#pragma unroll
        for (int w = 0; w < WV; ++w)
            wide |= *(const TVL_LDS int *)(hb + HFLAG + 4 * w);
        return __builtin_amdgcn_readfirstlane(wide) != 0;
    }

    // chunk c on the fp32 matrix cores (weight stage ST): x of vector
    // lane & 15, columns 32 q + 8 g + e, read from global memory
    template <int ST>
    __device__ __forceinline__ void products_fp32(int c, f4 (&cf)[RG]) const
    {
        const int lane = this->lane, j = lane & 15, g = lane >> 4;
        const float *xq = X + (int64_t)min(j, nb - 1) * ldx + c * CC + 8 * g;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            f4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                const f4 x0 = load_x4(xq + 32 * q), x1 = load_x4(xq + 32 * q + 4);
                const h8 a = *(const TVL_LDS h8 *)(this->lds + ST * STAGE + rg * 16 * Base::RB +
                                                  this->raddr[q]);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    t = mfma16((float)a[e], e < 4 ? x0[e] : x1[e - 4], t);
            }
            cf[rg] = t;
        }
    }

    // chunk c on the fp16 matrix cores (weight stage ST, split stage HS):
    // cf times the returned 2^-k is the chunk's contribution
    template <int ST, int HS>
    __device__ __forceinline__ float products_split(f4 (&cf)[RG]) const
    {
        const TVL_LDS char *hb = hl + HS * HSTAGE;
        const int lane = this->lane;
        const float inv = ((const TVL_LDS float *)(hb + HSCALE))[lane & 15];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            f4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                const h8 a = *(const TVL_LDS h8 *)(this->lds + ST * STAGE + rg * 16 * Base::RB +
                                                  this->raddr[q]);
                const h8 hi = *(const TVL_LDS h8 *)(hb + roff[q]);
                const h8 lo = *(const TVL_LDS h8 *)(hb + HPART + roff[q]);
                t = mfma16h(a, hi, t);
                t = mfma16h(a, lo, t);
            }
            cf[rg] = t;
        }
        return inv;
    }

    template <int ST, int HS>
    __device__ __forceinline__ bool step(int &c, int nfull, f4 (&xr)[2][XL], f4 (&acc)[RG],
                                         f4 (&t1)[RG], f4 (&t2)[RG], int &n1) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_sched_barrier(0);
        // vmcnt(NL): the weights of c and this wavefront's x of c + 1 have
        // landed; the weights of c + 1 may still be in flight
        __builtin_amdgcn_s_waitcnt((NL & 15) | ((NL >> 4) << 14) | 0x0F70);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        load_xs(min(c + 2, nfull - 1), xr[HS]); // x of c, split last step: free
        Base::template issue<(ST + 2) % 3>((c + 2) * CC, c + 2 < nfull);
        __builtin_amdgcn_sched_barrier(0);
        // the matrix-core steps of chunk c first, speculatively on the split
        // parts (a chunk too wide for them, rare, is redone on the fp32
        // matrix cores and these products dropped), so that neither the flag
        // test nor the split of x of c + 1 (past the end: never read) stands
        // before them; the split runs while they do (in both branches, so that
        // the products stay in the accumulators until added)
        f4 cf[RG];
        const float inv = products_split<ST, HS>(cf);
        if (__builtin_expect(wide_chunk<HS>(), 0)) {
            products_fp32<ST>(c, cf);
            split<1 - HS>(xr[1 - HS]);
#pragma unroll
            for (int rg = 0; rg < RG; ++rg)
                acc[rg] += cf[rg];
        } else {
            __builtin_amdgcn_sched_barrier(0);
            split<1 - HS>(xr[1 - HS]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int rg = 0; rg < RG; ++rg)
                acc[rg] += cf[rg] * inv;
        }
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
            t1[rg] += acc[rg];
            acc[rg] = z;
        }
        if (++n1 == kMfmaLevel) {
#pragma unroll
            for (int rg = 0; rg < RG; ++rg) {
                t2[rg] += t1[rg];
                t1[rg] = z;
            }
            n1 = 0;
        }
        __builtin_amdgcn_sched_barrier(0);
        return ++c == nfull;
    }

    __device__ __forceinline__ void run(f4 (&out)[RG]) const
    {
        const f4 z = {0.f, 0.f, 0.f, 0.f};
        f4 acc[RG], t1[RG], t2[RG];
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            acc[rg] = t1[rg] = t2[rg] = z;
        const int nfull = this->kn / CC;
        int c = 0, n1 = 0;
        // the previous tile's readers of the shared split stages are done
        __builtin_amdgcn_s_barrier();
        if (nfull > 0) {
            f4 xr[2][XL];
            load_xs(0, xr[0]);
            Base::template issue<0>(0, true);
            load_xs(min(1, nfull - 1), xr[1]);
            Base::template issue<1>(CC, nfull > 1);
            __builtin_amdgcn_sched_barrier(0);
            // this wavefront's x of chunk 0 has landed (the weights of 0 and
            // 1 and the x of 1 may still be in flight)
            constexpr int W0 = 2 * NL + XL;
            __builtin_amdgcn_s_waitcnt((W0 & 15) | ((W0 >> 4) << 14) | 0x0F70);
            __builtin_amdgcn_sched_barrier(0);
            split<0>(xr[0]);
            for (;;) {
                if (step<0, 0>(c, nfull, xr, acc, t1, t2, n1)) break;
                if (step<1, 1>(c, nfull, xr, acc, t1, t2, n1)) break;
                if (step<2, 0>(c, nfull, xr, acc, t1, t2, n1)) break;
                if (step<0, 1>(c, nfull, xr, acc, t1, t2, n1)) break;
                if (step<1, 0>(c, nfull, xr, acc, t1, t2, n1)) break;
                if (step<2, 1>(c, nfull, xr, acc, t1, t2, n1)) break;
            }
            __builtin_amdgcn_s_waitcnt(0x0F70); // the empty loads too
        }
        if (c * CC < this->kn) // private: weights stage 0, x in registers
            Base::tail(c * CC, acc);
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
            out[rg] = t2[rg] + (t1[rg] + acc[rg]);
    }
};

// One row tile with x shared by the block; every wavefront runs it to the
// end (see above).  lds: the block's LDS (weight stages, then the shared x
// or split-x stages).
template <typename T, int RG, int CC, int WV, bool HX>
struct XsRowsOf {
    using type = MfmaDmaXsRows<T, RG, CC, WV, HX>;
    static constexpr int kShared = 3 * type::XSTAGE; // LDS bytes after the weight stages
};
template <int RG, int CC, int WV>
struct XsRowsOf<_Float16, RG, CC, WV, true> {
    using type = MfmaXsHxRows<RG, CC, WV>;
    static constexpr int kShared = 2 * type::HSTAGE;
};

template <typename T, int RG, int WV, int CC, bool HX>
__device__ __forceinline__ void tile_mfma_dma_xs(const DevItem &it, int row0, TVL_LDS char *lds)
{
    using Rows = typename XsRowsOf<T, RG, CC, WV, HX>::type;
    if (it.ldw > Rows::MAXLDW || it.ldx > Rows::MAXLDX) { // the item decides, no barrier
        tile_mfma16<T, RG, 4, WV>(it, row0);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wrow0 = row0 + wave * (16 * RG); // may be past M: empty loads, no stores
    const int nb = it.nrhs < 1 ? 1 : it.nrhs;
    f4 out[RG];
    const Rows mr(static_cast<const T *>(it.W), it.ldw, wrow0, it.M, it.x, it.ldx, nb, it.K,
                  lane, wave, lds + wave * (3 * Rows::STAGE), lds + WV * (3 * Rows::STAGE));
    mr.run(out);
    const int i = lane & 15, g = lane >> 4;
    if (i < nb) {
        float *yv = it.y + (int64_t)i * it.ldy;
#pragma unroll
        for (int rg = 0; rg < RG; ++rg)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wrow0 + 16 * rg + 4 * g + v;
                if (row < it.M) yv[row] = out[rg][v];
            }
    }
}

template <typename T, int RG, int WV, int CC, bool HX>
constexpr int dma_xs_lds()
{
    using Of = XsRowsOf<T, RG, CC, WV, HX>;
    return WV * 3 * Of::type::STAGE + Of::kShared;
}

// launches of one weight dtype (T); HX with fp16 only
template <typename T, int RG, int WV, int CC, bool HX>
__global__ __launch_bounds__(WV *kWave) void k_sweep_mfma_xs(const DevItem *__restrict__ items,
                                                              const DevTile *__restrict__ tiles,
                                                              int ntiles)
{
    __shared__ f4 lds[dma_xs_lds<T, RG, WV, CC, HX>() / 16];
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) { // block-uniform
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_mfma_dma_xs<T, RG, WV, CC, HX>(it, tl.row0, (TVL_LDS char *)lds);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <typename T, int RG, int WV, int CC, bool HX>
__global__ __launch_bounds__(WV *kWave) void k_item_mfma_xs(const DevItem it)
{
    __shared__ f4 lds[dma_xs_lds<T, RG, WV, CC, HX>() / 16];
    tile_mfma_dma_xs<T, RG, WV, CC, HX>(it, (int)blockIdx.x * (16 * RG * WV),
                                        (TVL_LDS char *)lds);
}

// LDS bytes per wavefront of a launch with weight dtypes WM.  A mixed launch
// gives every wavefront the fp32 size: the wavefronts of a block move on to
// their next tiles independently, so one may run an fp32 tile while another
// still runs an fp16 one.
template <int WM, int RG, int CC, int S>
constexpr int dma_wave_lds()
{
    if constexpr (WM == kWF16)
        return S * MfmaDmaRows<_Float16, RG, CC, S>::STAGE;
    else
        return S * MfmaDmaRows<float, RG, CC, S>::STAGE;
}

template <int WM, int RG, int CC, int S>
__device__ __forceinline__ TVL_LDS char *dma_wave_base(f4 *lds)
{
    return (TVL_LDS char *)lds +
           __builtin_amdgcn_readfirstlane(threadIdx.x / kWave) * dma_wave_lds<WM, RG, CC, S>();
}

// HX: fp16 items on the fp16 matrix cores (fp32 items are unaffected)
template <int WM, int RG, int WV, int CC, int S, bool HX>
__device__ __forceinline__ void tile_mfma_dma_w(const DevItem &it, int row0, TVL_LDS char *lds)
{
    if constexpr (WM == kWF32)
        tile_mfma_dma<float, RG, WV, CC, S, false>(it, row0, lds);
    else if constexpr (WM == kWF16)
        tile_mfma_dma<_Float16, RG, WV, CC, S, HX>(it, row0, lds);
    else if (it.dtype == 1)
        tile_mfma_dma<_Float16, RG, WV, CC, S, HX>(it, row0, lds);
    else
        tile_mfma_dma<float, RG, WV, CC, S, false>(it, row0, lds);
}

template <int WM, int RG, int WV, int CC, int S, bool HX>
__global__ __launch_bounds__(WV *kWave) void k_sweep_mfma_dma(const DevItem *__restrict__ items,
                                                               const DevTile *__restrict__ tiles,
                                                               int ntiles)
{
    __shared__ f4 lds[WV * dma_wave_lds<WM, RG, CC, S>() / 16];
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_mfma_dma_w<WM, RG, WV, CC, S, HX>(it, tl.row0, dma_wave_base<WM, RG, CC, S>(lds));
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int WM, int RG, int WV, int CC, int S, bool HX>
__global__ __launch_bounds__(WV *kWave) void k_item_mfma_dma(const DevItem it)
{
    __shared__ f4 lds[WV * dma_wave_lds<WM, RG, CC, S>() / 16];
    tile_mfma_dma_w<WM, RG, WV, CC, S, HX>(it, (int)blockIdx.x * (16 * RG * WV),
                                           dma_wave_base<WM, RG, CC, S>(lds));
}

// (rows per wavefront = 16 RG, waves per block, U = 2 marks this form).
// Two variants ran slower on MI355X with 8 vectors and were not kept: the
// next chunk's loads issued before the current chunk's products (~200 VGPRs
// at 16 rows: 4.9-5.0 against 5.2-5.3 TB/s), and x staged through LDS too
// (whole-line x loads: 5.05 against 5.24 TB/s).
#define TVL_MFMA_LDS_SHAPES(X) X(16, 1, 2) X(16, 4, 2) X(32, 1, 2) X(32, 2, 2) X(32, 4, 2) X(64, 1, 2)

// (rows per wavefront = 16 RG, waves per block, U, columns per chunk, stages,
// HX) of the form with weights streamed into LDS: U = 10 S + log2(CC / 16),
// + 100 for fp16 weights on the fp16 matrix cores (HX).  Chunks of at least
// 64 columns (a 128-byte fp16 row chunk).
#define TVL_MFMA_DMA_SHAPES(X)                                                                    \
    X(16, 1, 33, 128, 3, false) X(16, 2, 33, 128, 3, false) X(32, 1, 33, 128, 3, false)          \
        X(16, 1, 32, 64, 3, false) X(16, 4, 32, 64, 3, false) X(32, 1, 32, 64, 3, false)          \
            X(32, 2, 32, 64, 3, false) X(16, 4, 42, 64, 4, false) X(32, 1, 42, 64, 4, false)      \
                X(32, 1, 52, 64, 5, false) X(16, 1, 133, 128, 3, true)                            \
                    X(16, 2, 133, 128, 3, true) X(32, 1, 133, 128, 3, true)                       \
                        X(32, 2, 133, 128, 3, true) X(64, 1, 133, 128, 3, true)                   \
                            X(32, 1, 132, 64, 3, true) X(64, 1, 132, 64, 3, true)

template <int R, int WV, int U>
struct InstMfmaLds {
    static constexpr int RG = R / 16;
    template <int WM>
    static hipError_t sweep_w(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                              hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_mfma_lds<WM, RG, WV>), dim3(grid), dim3(WV * kWave), 0, st,
                           items, tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t sweep(int wm, const DevItem *items, const DevTile *tiles, int ntiles,
                            int grid, hipStream_t st)
    {
        return wm == kWF32   ? sweep_w<kWF32>(items, tiles, ntiles, grid, st)
               : wm == kWF16 ? sweep_w<kWF16>(items, tiles, ntiles, grid, st)
                             : sweep_w<kWMixed>(items, tiles, ntiles, grid, st);
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (it.dtype == 1)
            hipLaunchKernelGGL((k_item_mfma_lds<kWF16, RG, WV>), grid, block, 0, st, it);
        else
            hipLaunchKernelGGL((k_item_mfma_lds<kWF32, RG, WV>), grid, block, 0, st, it);
        return hipGetLastError();
    }
};

// (rows per wavefront = 16 RG, waves per block, U, columns per chunk, HX)
// of the streamed form with x shared by the block: U = 200 + log2(CC / 16),
// + 100 for fp16 weights on the fp16 matrix cores (HX).  Launches mixing
// weight dtypes, and for HX shapes launches holding fp32 weights, run the
// LDS-staged form with the same rows and waves.
#define TVL_MFMA_XS_SHAPES(X)                                                                     \
    X(16, 4, 202, 64, false) X(32, 2, 202, 64, false) X(32, 4, 202, 64, false)                    \
        X(16, 2, 203, 128, false) X(16, 4, 203, 128, false) X(16, 8, 202, 64, false)              \
            X(16, 4, 303, 128, true) X(32, 2, 303, 128, true) X(32, 4, 303, 128, true)            \
                X(16, 8, 303, 128, true) X(16, 4, 302, 64, true) X(32, 4, 302, 64, true)

template <int R, int WV, int CC, bool HX>
struct InstMfmaXs {
    static constexpr int RG = R / 16;
    static hipError_t sweep(int wm, const DevItem *items, const DevTile *tiles, int ntiles,
                            int grid, hipStream_t st)
    {
        const dim3 g(grid), b(WV * kWave);
        if (wm == kWF16) {
            hipLaunchKernelGGL((k_sweep_mfma_xs<_Float16, RG, WV, CC, HX>), g, b, 0, st, items,
                               tiles, ntiles);
            return hipGetLastError();
        }
        if constexpr (!HX) {
            if (wm == kWF32) {
                hipLaunchKernelGGL((k_sweep_mfma_xs<float, RG, WV, CC, false>), g, b, 0, st,
                                   items, tiles, ntiles);
                return hipGetLastError();
            }
        }
        return InstMfmaLds<R, WV, 2>::sweep(wm, items, tiles, ntiles, grid, st);
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (it.dtype == 1) {
            hipLaunchKernelGGL((k_item_mfma_xs<_Float16, RG, WV, CC, HX>), grid, block, 0, st, it);
            return hipGetLastError();
        }
        if constexpr (!HX) {
            hipLaunchKernelGGL((k_item_mfma_xs<float, RG, WV, CC, false>), grid, block, 0, st, it);
            return hipGetLastError();
        }
        return InstMfmaLds<R, WV, 2>::item(it, st);
    }
};

template <int R, int WV, int CC, int S, bool HX>
struct InstMfmaDma {
    static constexpr int RG = R / 16;
    template <int WM>
    static hipError_t sweep_w(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                              hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_mfma_dma<WM, RG, WV, CC, S, HX>), dim3(grid), dim3(WV * kWave),
                           0, st, items, tiles, ntiles);
        return hipGetLastError();
    }
    // HX shapes serve launches of fp16 weights only; others run the
    // LDS-staged form with the same rows and waves
    static hipError_t sweep(int wm, const DevItem *items, const DevTile *tiles, int ntiles,
                            int grid, hipStream_t st)
    {
        if constexpr (HX) {
            if (wm != kWF16) return InstMfmaLds<R, WV, 2>::sweep(wm, items, tiles, ntiles, grid, st);
            return sweep_w<kWF16>(items, tiles, ntiles, grid, st);
        } else {
            return wm == kWF32   ? sweep_w<kWF32>(items, tiles, ntiles, grid, st)
                   : wm == kWF16 ? sweep_w<kWF16>(items, tiles, ntiles, grid, st)
                                 : sweep_w<kWMixed>(items, tiles, ntiles, grid, st);
        }
    }
    static hipError_t item(const DevItem &it, hipStream_t st)
    {
        const dim3 grid((it.M + R * WV - 1) / (R * WV)), block(WV * kWave);
        if (it.dtype == 1) {
            hipLaunchKernelGGL((k_item_mfma_dma<kWF16, RG, WV, CC, S, HX>), grid, block, 0, st, it);
        } else {
            if constexpr (HX)
                return InstMfmaLds<R, WV, 2>::item(it, st);
            else
                hipLaunchKernelGGL((k_item_mfma_dma<kWF32, RG, WV, CC, S, HX>), grid, block, 0, st,
                                   it);
        }
        return hipGetLastError();
    }
};

// (R, waves per block, U, B) with B x vectors per launch (B >= nrhs).
#define TVL_MULTI_SHAPES(X)                                                                       \
    X(2, 4, 2, 2) X(2, 4, 4, 2) X(4, 4, 2, 2) X(2, 4, 1, 4) X(2, 4, 2, 4) X(4, 4, 1, 4)          \
        X(4, 4, 2, 4) X(2, 4, 1, 8) X(2, 4, 2, 8) X(4, 4, 1, 8) X(8, 4, 1, 4) X(8, 2, 1, 4)      \
            X(8, 2, 1, 2)

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
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return s.xmode == kXDirect && B <= 16;
    TVL_MULTI_SHAPES(X)
    TVL_MFMA_SHAPES(Y)
    TVL_MFMA16_SHAPES(Y)
    TVL_MFMA_LDS_SHAPES(Y)
#define D(R_, W_, U_, CC_, S_, HX_) Y(R_, W_, U_)
    TVL_MFMA_DMA_SHAPES(D)
#undef D
#define D(R_, W_, U_, CC_, HX_) Y(R_, W_, U_)
    TVL_MFMA_XS_SHAPES(D)
#undef D
#undef X
#undef Y
    return false;
}

hipError_t launch_sweep_multi(const Shape &s, int B, int wmode, const DevItem *items,
                              const DevTile *tiles, int ntiles, int grid, hipStream_t st)
{
#define X(R_, W_, U_, B_)                                                                         \
    if (s.R == R_ && s.W == W_ && s.U == U_ && B == B_)                                          \
        return InstMulti<R_, W_, U_, B_>::sweep(items, tiles, ntiles, grid, st);
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfma<R_, W_, U_>::sweep(B, wmode, items, tiles, ntiles, grid, st);
#define Z(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfma16<R_, W_, U_>::sweep(wmode, items, tiles, ntiles, grid, st);
#define V(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfmaLds<R_, W_, U_>::sweep(wmode, items, tiles, ntiles, grid, st);
    TVL_MULTI_SHAPES(X)
    TVL_MFMA_SHAPES(Y)
    TVL_MFMA16_SHAPES(Z)
    TVL_MFMA_LDS_SHAPES(V)
#define D(R_, W_, U_, CC_, S_, HX_)                                                               \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfmaDma<R_, W_, CC_, S_, HX_>::sweep(wmode, items, tiles, ntiles, grid, st);
    TVL_MFMA_DMA_SHAPES(D)
#undef D
#define D(R_, W_, U_, CC_, HX_)                                                                   \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfmaXs<R_, W_, CC_, HX_>::sweep(wmode, items, tiles, ntiles, grid, st);
    TVL_MFMA_XS_SHAPES(D)
#undef D
#undef X
#undef Y
#undef Z
#undef V
    return hipErrorInvalidValue;
}

hipError_t launch_item_multi(const Shape &s, int B, const DevItem &item, hipStream_t st)
{
#define X(R_, W_, U_, B_)                                                                         \
    if (s.R == R_ && s.W == W_ && s.U == U_ && B == B_)                                          \
        return InstMulti<R_, W_, U_, B_>::item(item, st);
#define Y(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstMfma<R_, W_, U_>::item(B, item, st);
#define Z(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstMfma16<R_, W_, U_>::item(item, st);
#define V(R_, W_, U_)                                                                             \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstMfmaLds<R_, W_, U_>::item(item, st);
    TVL_MULTI_SHAPES(X)
    TVL_MFMA_SHAPES(Y)
    TVL_MFMA16_SHAPES(Z)
    TVL_MFMA_LDS_SHAPES(V)
#define D(R_, W_, U_, CC_, S_, HX_)                                                               \
    if (s.R == R_ && s.W == W_ && s.U == U_)                                                     \
        return InstMfmaDma<R_, W_, CC_, S_, HX_>::item(item, st);
    TVL_MFMA_DMA_SHAPES(D)
#undef D
#define D(R_, W_, U_, CC_, HX_)                                                                   \
    if (s.R == R_ && s.W == W_ && s.U == U_) return InstMfmaXs<R_, W_, CC_, HX_>::item(item, st);
    TVL_MFMA_XS_SHAPES(D)
#undef D
#undef X
#undef Y
#undef Z
#undef V
    return hipErrorInvalidValue;
}

}  // namespace tvl
