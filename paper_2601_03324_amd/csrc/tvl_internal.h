// tvl_internal.h -- declarations shared by the C-ABI layer (tvl_abi.cpp) and
// the gfx950 kernels (tvl_*.hip, tvl_device.h).  Not installed, not part of
// the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace tvl {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kLineBytes = 128;    // TVL row alignment: one gfx950 L2 cache line
constexpr int kChunkElems = 512;   // LDS slice granularity: 64 lanes x 8 fp16 = 2 x (64 x 4 fp32)
constexpr int kSliceCap = 8192;    // x elements staged per pass: 32 KB of LDS

// Item operations (mirrors tvl_item.op).
constexpr int kOpGemv = 0;
constexpr int kOpSwiglu = 1;

// One GEMV as the kernels read it (96 bytes).  M and K fit in int32 (the
// ABI rejects larger), ldw stays 64-bit.  W3 is the second matrix of a
// SwiGLU item; g (or NULL) the RMSNorm weight applied to x first; nrhs x
// vectors at a stride of ldx floats give nrhs outputs at a stride of ldy.
// lanes: for block-quantised weights, the lanes of a wavefront that share
// one row (8, 16, 32 or 64; see quant_lanes); unused otherwise.
struct DevItem {
    const void *W;
    int64_t ldw;
    const float *x;
    float *y;
    int32_t M;
    int32_t K;
    int32_t dtype;
    int32_t op;
    const void *W3;
    const float *g;
    float eps;
    int32_t nrhs;
    int64_t ldx;
    int64_t ldy;
    int32_t lanes;
    int32_t reserved;
};
static_assert(sizeof(DevItem) == 96, "DevItem layout");

// Lanes per row for a block-quantised row of K columns at `bits` per code.
// A lane loads 16 bytes (128 / bits columns) at a time, so a row is
// nv = ceil(K * bits / 128) loads.  Short rows would leave most of a
// 64-lane wavefront idle (a 4-bit row of 768 columns is 24 loads), so a
// wavefront splits into 64 / G groups of G lanes, one row per group: G is
// the group size in {64, 32, 16, 8} that pads nv the least.  Ties go to the
// larger G (more tiles, shorter chains of loads per lane), except with
// `few_lanes`: then to the smaller G.  A lane's 32 4-bit codes need 128
// contiguous bytes of x, so one x load instruction touches G cache lines
// (the code load it serves touches 8): for 4-bit rows in launches long
// enough to hide the longer per-lane chains, G = 8 keeps x from costing the
// load pipeline more than the codes do (the 4-bit Llama-2 7B token: 5.74 ->
// 6.33 TB/s; the 110M one, 62 MB, loses a third with it).
inline int quant_lanes(int64_t K, int bits, bool few_lanes = false)
{
    const int64_t nv = (K * bits + 127) / 128;
    int best = 64;
    int64_t best_pad = (nv + 63) / 64 * 64;
    for (int g = 32; g >= 8; g /= 2) {
        const int64_t pad = (nv + g - 1) / g * g;
        if (pad < best_pad || (few_lanes && pad == best_pad)) {
            best = g;
            best_pad = pad;
        }
    }
    return best;
}

// One row tile of a sweep: item index and first row.
struct DevTile {
    int32_t item;
    int32_t row0;
};
static_assert(sizeof(DevTile) == 8, "DevTile layout");

// How a wavefront gets x: staged once per workgroup in LDS, or read
// directly from global memory (L1/L2-cached) next to the weights.
constexpr int kXLds = 0;
constexpr int kXDirect = 1;

// Launch shape: rows per wave, waves per block, loads in flight per row,
// x mode.
struct Shape {
    int R;
    int W;
    int U;
    int xmode;
};

bool shape_supported(const Shape &s);

// Elements of x staged per LDS pass for a row of K columns.
inline int slice_cap(int64_t K)
{
    const int64_t r = (K + kChunkElems - 1) / kChunkElems * kChunkElems;
    return (int)(r < kSliceCap ? r : kSliceCap);
}

hipError_t launch_gemv_rows(const Shape &s, int dtype, const void *W, int64_t ldw,
                            const float *x, float *y, int M, int K, hipStream_t st);

hipError_t launch_gemv_ksplit(const Shape &s, int dtype, const void *W, int64_t ldw,
                              const float *x, float *y, int M, int K, int S,
                              float *partials, int *counters, hipStream_t st);

hipError_t launch_sweep(const Shape &s, const DevItem *items, const DevTile *tiles,
                        int ntiles, int grid, int ks_cap, hipStream_t st);

// Scratch of the allocation-free K split (tvl_gemv_noalloc): one file-scope
// device array per GPU holding kNoallocPartials fp32 partials followed by
// kNoallocCounters int arrival counters (4.25 MiB).
constexpr int64_t kNoallocPartials = int64_t(1) << 20;
constexpr int64_t kNoallocCounters = int64_t(1) << 16;
// Device address of the current device's scratch (device `dev` must be
// current).  The first call per device looks the array up with
// hipGetSymbolAddress, clears its counters on `st` and synchronises `st`;
// it returns hipErrorStreamCaptureUnsupported, doing nothing, if `st` is
// being captured.  Later calls make no HIP call.
hipError_t noalloc_scratch(int dev, hipStream_t st, float **partials, int **counters);

// Sweep with fused RMSNorm / SwiGLU items (direct-x mode, R even).
bool fused_shape_supported(const Shape &s);
hipError_t launch_sweep_fused(const Shape &s, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, hipStream_t st);
// One item (any op) as one launch: grid = its row tiles, item by value.
hipError_t launch_item(const Shape &s, const DevItem &item, hipStream_t st);

// Plans or items with block-quantised weights (any plain item).  Direct-x,
// or (xmode kXLds) the quantised items' x staged once per row tile in LDS,
// xbytes = quant_x_lds_bytes(largest quantised K) of dynamic LDS per
// workgroup; plain items read x directly either way.
bool quant_shape_supported(const Shape &s);
hipError_t launch_sweep_quant(const Shape &s, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, int xbytes, hipStream_t st);
hipError_t launch_item_quant(const Shape &s, const DevItem &item, int xbytes, hipStream_t st);

// LDS bytes for x of K columns in the quantised kernels' layout: whole
// 1 KiB blocks of 256 columns (the staging loads' unit; the ragged last load
// of a row reads at most to the end of its 32-column run).
inline int64_t quant_x_lds_bytes(int64_t K) { return (K + 255) / 256 * 1024; }

// Several x vectors per item (B = 2, 4, 8 or 16 >= every item's nrhs;
// direct-x).  Shapes with R >= 8 run on the matrix cores (any B); wmode tells
// them which weight dtypes the launch holds: 0 fp32 only, 1 fp16 only, 2 both.
bool multi_shape_supported(const Shape &s, int B);
hipError_t launch_sweep_multi(const Shape &s, int B, int wmode, const DevItem *items,
                              const DevTile *tiles, int ntiles, int grid, hipStream_t st);
hipError_t launch_item_multi(const Shape &s, int B, const DevItem &item, hipStream_t st);

hipError_t launch_pack(int dtype, void *dst, int64_t ldw, const void *src, int64_t M,
                       int64_t K, hipStream_t st);

hipError_t launch_zero_i32(int *p, int64_t n, hipStream_t st);

hipError_t launch_read_stream(const void *src, int64_t bytes, float *sink, int grid,
                              hipStream_t st);

hipError_t launch_copy(void *dst, const void *src, int64_t bytes, hipStream_t st);

}  // namespace tvl
