// tvl_gemv.hip -- plain fp32 / fp16 GEMV kernels for gfx950: the single
// GEMV (row split in both x modes, K split) and the grouped sweep that runs
// every GEMV of a decode token in one launch (Sec. 1: each token streams
// every weight matrix once).  LDS-x mode stages x once per workgroup in
// slices of up to 8192 elements; direct-x mode reads it next to the weights.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>

#include "tvl_device.h"

// Scratch of the allocation-free K split (tvl_gemv_noalloc): the fp32
// partials of every slice, then one int arrival counter per row tile, for
// callers that cannot allocate device memory.  Each GPU the library runs on
// holds its own copy until the process ends.  In host code this name stands
// for a host-side shadow, not a device address: kernels are given the address
// that hipGetSymbolAddress returns for the current device (noalloc_scratch).
static __device__ __align__(256) unsigned char
    scratch[(tvl::kNoallocPartials + tvl::kNoallocCounters) * 4];

namespace tvl {
namespace {

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
// workgroup that brings the counter to S takes an agent-scope acquire fence,
// adds the S partials in the order 0..S-1 (device-coherent loads) and resets
// the counter for the next launch.
//
// The publishing side has no release fence: on a multi-XCD part an
// agent-scope release compiles to a write-back of the whole L2, once per
// workgroup (measured 20-100x slower than the row split).  It is not needed
// for exactly the data published here: the partials are agent-scope atomic
// stores, written through to the coherence point (sc1), and the wait for
// their acknowledgement before the barrier and the counter update is what
// the release would add for them.  The acquire fence (an L2 invalidation in
// the last workgroup only, once per row tile) orders the partial loads after
// the counter.  A CPU test compiles this kernel and checks that code.
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
        // acquire (agent scope) for the partials the other slices published:
        // one per row tile, in the last workgroup only
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
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

// ------------------------------------------------------ shape dispatch
// (R, waves per block, U) triples the library instantiates, per x mode.
#define TVL_LDS_SHAPES(X)                                                                         \
    X(1, 4, 4) X(1, 4, 8) X(2, 4, 2) X(2, 4, 3) X(2, 4, 4) X(2, 4, 8) X(4, 4, 1) X(4, 4, 2)       \
    X(4, 4, 3) X(4, 4, 4) X(8, 4, 1) X(8, 4, 2) X(2, 8, 4) X(2, 8, 8) X(4, 8, 2) X(1, 2, 8)       \
    X(2, 2, 8) X(4, 2, 4) X(8, 2, 2)
#define TVL_DIRECT_SHAPES(X)                                                                      \
    X(1, 1, 4) X(1, 1, 8) X(2, 1, 2) X(2, 1, 3) X(2, 1, 4) X(2, 1, 8) X(4, 1, 1) X(4, 1, 2)       \
    X(4, 1, 3) X(4, 1, 4) X(8, 1, 1) X(8, 1, 2) X(1, 4, 4) X(1, 4, 8) X(2, 4, 2) X(2, 4, 3)       \
    X(2, 4, 4) X(2, 4, 8) X(4, 4, 1) X(4, 4, 2) X(4, 4, 3) X(4, 4, 4) X(8, 4, 1) X(8, 4, 2)       \
    X(1, 8, 8) X(2, 8, 3) X(2, 8, 4) X(4, 8, 2)

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

namespace {
std::mutex g_scratch_mu;
std::map<int, unsigned char *> g_scratch; // device -> its copy of `scratch`
}  // namespace

hipError_t noalloc_scratch(int dev, hipStream_t st, float **partials, int **counters)
{
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch.find(dev);
    if (it == g_scratch.end()) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(st, &cap);
        if (e != hipSuccess) return e;
        if (cap != hipStreamCaptureStatusNone) return hipErrorStreamCaptureUnsupported;
        unsigned char *p = nullptr;
        e = hipGetSymbolAddress(reinterpret_cast<void **>(&p), HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        // Every K-split launch leaves its counters at zero; they must start
        // there.  The synchronisation makes the cleared counters visible to
        // launches on any stream of this device.
        e = launch_zero_i32(reinterpret_cast<int *>(p + kNoallocPartials * 4), kNoallocCounters,
                            st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return e;
        it = g_scratch.emplace(dev, p).first;
    }
    *partials = reinterpret_cast<float *>(it->second);
    *counters = reinterpret_cast<int *>(it->second + kNoallocPartials * 4);
    return hipSuccess;
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

}  // namespace tvl
