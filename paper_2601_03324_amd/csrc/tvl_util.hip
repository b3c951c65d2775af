// tvl_util.hip -- the TVL pack kernel (dense rows -> 128-byte-aligned rows,
// Sec. 3.2), the counter-zeroing kernel of the K split, and two measurement
// diagnostics: a read-only stream with the GEMV's load kind (the practical
// read ceiling) and a copy of known size (calibrates the traffic counters).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvl_device.h"

namespace tvl {
namespace {

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
// flight per lane (the last batch of a span with its loads past the span
// switched off, so a short span keeps its loads in flight too).  The
// workgroup's first thread writes its own partial sum to sink[b]: every
// thread's loads are still issued (they feed the same code), and a
// workgroup ends without a reduction or barrier, which for short launches
// of many small workgroups is part of what is measured.
__global__ __launch_bounds__(256) void k_read_stream(const f4 *__restrict__ src, int64_t nvec,
                                                     int64_t per, float *__restrict__ sink)
{
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
    if (i < end) {
        f4 a[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            a[u] = i + u * 256 < end ? __builtin_nontemporal_load(g + i + u * 256)
                                     : f4{0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            acc += a[u];
    }
    if (threadIdx.x == 0) sink[blockIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
}

__global__ __launch_bounds__(256) void k_copy(f4 *__restrict__ dst, const f4 *__restrict__ src,
                                              int64_t nvec)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec;
         i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = __builtin_nontemporal_load(src + i);
}



}  // namespace

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
    // spans of whole 128-byte lines, so each wavefront load covers 8 lines
    // (trailing workgroups may get empty spans)
    const int64_t per = ((nvec + grid - 1) / grid + 7) / 8 * 8;
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
