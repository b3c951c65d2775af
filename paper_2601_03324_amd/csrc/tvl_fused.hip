// tvl_fused.hip -- sweep and single-item kernels whose items may carry a
// fused RMSNorm of x (Sec. 2.1 pre-normalisation, Sec. 11.2 listing) and/or
// be SwiGLU pairs y = silu(w1 x) * (w3 x) (the gated FFN input of Sec. 2.1).
// The per-tile code is tile_any in tvl_device.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvl_device.h"

namespace tvl {
namespace {

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

// (R, waves per block, U) triples with fused RMSNorm / SwiGLU support.
#define TVL_FUSED_SHAPES(X)                                                                       \
    X(2, 4, 2) X(2, 4, 3) X(2, 4, 4) X(2, 1, 4) X(4, 1, 2) X(4, 1, 4) X(4, 4, 2) X(2, 1, 8)          \
        X(8, 4, 1) X(8, 2, 1) X(4, 4, 3)

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

}  // namespace

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

}  // namespace tvl
