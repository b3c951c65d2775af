// tvl_quant.hip -- GEMV over block-quantised weights (8- and 4-bit codes,
// one fp32 scale per 64 columns; the format is defined in tvl.h), the
// on-the-fly unpacking the paper proposes for low-bit weights (Sec. 8.2).
// A plan holding quantised items may also hold plain fp32 / fp16 items.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvl_device.h"

namespace tvl {
namespace {

// Block-quantised weights (8- or 4-bit two's-complement codes in M rows of
// ldw bytes; fp32 scale per 64 columns in a row-major plane after the code
// rows).  A 16-byte load brings N = 16 (8-bit) or 32 (4-bit) codes of one
// row, all in one 64-column scale group, so each load is dotted with x first
// and scaled once.
//
// Decoding costs VALU work per code (a 4-bit row streams two codes per byte),
// so every code converts with ONE conversion instruction and one FMA, exactly:
//   8-bit: a sign-extending SDWA conversion of a byte (v_cvt_f32_i32 with a
//          byte select); the bytes are the codes;
//   4-bit: v_cvt_off_f32_i4 turns the signed nibble in bits 3:0 of its
//          operand into q / 16; an SDWA byte select reaches the low nibble
//          of each byte of a dword v, and of v >> 4 (its high nibbles).  The
//          factor 1/16 is folded into the scale (a power of two, exact).
//
// Short rows: a wavefront splits into 64 / G groups of G lanes, one row per
// group (G from quant_lanes), so a 384-byte row still fills its lanes.
//
// x, direct or through LDS.  All 64 / G groups of a wavefront read the same
// x, and each lane reads 128 bytes of it per 16-byte code load (4-bit), so x
// load instructions are as many as code loads.  With x staged in LDS (XL)
// they leave the vector-memory path to the codes: each workgroup copies the
// row tile's x into LDS once, by buffer loads that write LDS themselves
// (1 KiB per wavefront load, no VGPRs, one wait), between two barriers, and
// the lanes read it from there.  Within each 1 KiB block the 16-byte pieces
// of each 128-byte row r are XOR-swizzled (piece t stored at t ^ r), so the
// lanes of a group, whose x runs start 128 (4-bit) or 64 (8-bit) bytes
// apart, read 8 distinct 16-byte bank groups per step.
#define TVL_LDS __attribute__((address_space(3)))
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

// q / 16 for the signed nibble in bits 3:0 of byte B of v
#define TVL_NIB16(B)                                                                              \
    __device__ __forceinline__ float nib16_##B(unsigned v)                                        \
    {                                                                                             \
        float r;                                                                                  \
        asm("v_cvt_off_f32_i4_sdwa %0, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #B \
            : "=v"(r) : "v"(v));                                                                  \
        return r;                                                                                 \
    }
TVL_NIB16(0)
TVL_NIB16(1)
TVL_NIB16(2)
TVL_NIB16(3)
#undef TVL_NIB16

// 4-bit: sum_j q_j x_j / 16 over the 32 columns of one 16-byte vector.  Dword
// d holds columns 8d .. 8d+7, column 8d + 2b in the low nibble of byte b and
// 8d + 2b + 1 in its high nibble.  Per 8 codes: one shift, 8 conversions and
// 8 FMAs.
__device__ __forceinline__ float qdot4(const u4 w, const f4 (&xv)[8])
{
    float ta = 0.f, tb = 0.f; // even columns; odd columns
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const unsigned lo = w[d], hi = w[d] >> 4;
        const f4 x0 = xv[2 * d], x1 = xv[2 * d + 1];
        ta = fmaf(nib16_0(lo), x0.x, ta);
        tb = fmaf(nib16_0(hi), x0.y, tb);
        ta = fmaf(nib16_1(lo), x0.z, ta);
        tb = fmaf(nib16_1(hi), x0.w, tb);
        ta = fmaf(nib16_2(lo), x1.x, ta);
        tb = fmaf(nib16_2(hi), x1.y, tb);
        ta = fmaf(nib16_3(lo), x1.z, ta);
        tb = fmaf(nib16_3(hi), x1.w, tb);
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

// the f4 of x at column col (a multiple of 4) in the swizzled LDS layout:
// f4 j lives at 16-byte slot (j with its low 3 bits XORed by bits 5:3)
__device__ __forceinline__ f4 lds_x4(const TVL_LDS float *xl, int col)
{
    const int j = col >> 2;
    const int slot = (j & ~7) | ((j ^ (j >> 3)) & 7);
    return *(const TVL_LDS f4 *)(xl + 4 * slot);
}

template <int BITS, int G, int R, int U, bool XL = false>
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
    const TVL_LDS float *xl; // XL: the tile's x in LDS

    // lrow[r]: the lane's r-th row relative to the wave's first row (in range:
    // rows past M are clamped by the caller); srow0: the lane's first row in
    // the scale plane (rows past M read padding or, past the plane, zeros).
    // Scale of row i, group g: float (i/4)*4*ng + 4*g + i%4.
    __device__ __forceinline__ QuantRows(const unsigned char *codes0, int64_t code_bytes,
                                         const float *plane, int64_t plane_bytes, int64_t ldw,
                                         int ng, const int (&lrow)[R], int srow0, const float *x,
                                         int K, int seg_, const TVL_LDS float *xl_ = nullptr)
        : wr(make_rsrc(codes0, code_bytes)), sr(make_rsrc(plane, plane_bytes)),
          xr(make_rsrc(x, ((int64_t)K * 4 + 15) & ~(int64_t)15)),
          vs(16 * ((srow0 / 4) * ng + seg_ * N / 64) + 4 * (srow0 % 4)), sblk(16 * ng),
          vx(seg_ * N * 4), kn(K), nv((K + N - 1) / N), nfull(K / CH), seg(seg_), xl(xl_)
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
        if constexpr (XL)
            return lds_x4(xl, c * CH + seg * N + 4 * k);
        else
            return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(xr, vx + 16 * k, c * XB, 0));
    }
    // The same load with the whole offset in the range-checked VGPR part:
    // past the end of x (rounded to 16 bytes) it returns zeros, no branch
    // (XL: past K the staged segment holds what the last 16-byte load of x
    // brought, and the caller masks it).
    __device__ __forceinline__ f4 xload_checked(int c, int k) const
    {
        if constexpr (XL)
            return lds_x4(xl, c * CH + seg * N + 4 * k);
        else
            return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(xr, vx + 16 * k + c * XB, 0, 0));
    }

    __device__ __forceinline__ void accumulate(float &acc, const u4 w, float sc, const f4 (&xv)[NX]) const
    {
        if constexpr (BITS == 4)
            acc = fmaf(sc * 16.f, qdot4(w, xv), acc);
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

    // Full chunks from c in batches of U (all code loads of a batch issued
    // first; x with them, or with x in LDS and U > 1 read just before each
    // chunk's decode, so that it holds no VGPRs while the codes are in flight).
    __device__ __forceinline__ void run_batched(float (&acc)[R], int c = 0) const
    {
        constexpr bool LAZY_X = XL && U > 1;
        for (; c + U <= nfull; c += U) {
            u4 w[U][R];
            float sc[U][R];
            f4 xv[U][NX];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                load_codes(c + u, w[u], sc[u]);
                if constexpr (!LAZY_X) load_x(c + u, xv[u]);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (LAZY_X) load_x(c + u, xv[u]);
                compute(acc, w[u], sc[u], xv[u]);
            }
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
        run_tail(acc);
    }

    // U = 1, chunk 0's codes already loaded (w0, sc0; when nfull > 0)
    __device__ __forceinline__ void run_preloaded(float (&acc)[R], const u4 (&w0)[R],
                                                  const float (&sc0)[R]) const
    {
        static_assert(U == 1, "one chunk per batch");
        if (nfull > 0) { // wavefront-uniform
            f4 xv[NX];
            load_x(0, xv);
            compute(acc, w0, sc0, xv);
            run_batched(acc, 1);
        }
        run_tail(acc);
    }

    __device__ __forceinline__ void run_tail(float (&acc)[R]) const
    {
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
// XL: copy x[0, K) into the workgroup's LDS (the layout of lds_x4), then a
// barrier before this tile's readers (the caller has taken one after the
// previous tile's); every wavefront of the workgroup takes both.  Wavefront
// w loads 1 KiB blocks w, w + WV, ...: lane l = 8 r + t of a block's load
// fills slot l with f4 8 r + (t ^ r) of the block.  The descriptor covers K
// rounded up to 16 bytes, as for direct x: the last piece may hold up to 3
// values past K (the ragged last chunk masks them), and pieces past it read
// as zeros without touching memory.
template <int WV>
__device__ __forceinline__ void stage_x_quant(const DevItem &it, TVL_LDS float *xl)
{
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(it.x, ((int64_t)it.K * 4 + 15) & ~(int64_t)15);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int r = lane >> 3, t = lane & 7;
    const int voff = 16 * (8 * r + (t ^ r));
    const int nblk = (it.K + 255) / 256;
    // (the block offset goes in the per-lane offset, which the descriptor's
    // range check covers; the scalar offset is not checked)
    for (int b = wave; b < nblk; b += WV) // wavefront-uniform
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (TVL_LDS void *)(xl + 256 * b), 16,
                                                 voff + 1024 * b, 0, 0, 0);
    __builtin_amdgcn_s_waitcnt(0x0F70); // vmcnt(0): the LDS writes of these loads
    __syncthreads();
}

template <int BITS, int G, int R, int WV, int U, bool XL>
__device__ __forceinline__ void tile_quant_g(const DevItem &it, int row0, TVL_LDS float *xl)
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
    if constexpr (XL) {
        __syncthreads(); // the previous tile's readers of x are done
        if (wrow0 >= it.M) { // wavefront-uniform: no rows, but its share of x
            stage_x_quant<WV>(it, xl);
            return;
        }
    } else if (wrow0 >= it.M) {
        return;
    }
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
    const QuantRows<BITS, G, R, U, XL> qr(codes + (int64_t)wrow0 * it.ldw,
                                          (int64_t)rows_left * it.ldw, plane, (int64_t)4 * Mp * ng,
                                          it.ldw, ng, lrow, wrow0 + sub * R, it.x, it.K, seg, xl);
    if constexpr (XL && U == 1) {
        // the first chunk's codes in flight while x is staged (the wait for
        // the x loads, issued after them, covers both).  Loaded whether or
        // not the row has a full chunk (then unused): a 16-byte load per row
        // at the lane's offset, inside the range-checked descriptor.
        u4 w0[R];
        float sc0[R];
        qr.load_codes(0, w0, sc0);
        __builtin_amdgcn_sched_barrier(0);
        stage_x_quant<WV>(it, xl);
        __builtin_amdgcn_sched_barrier(0);
        qr.run_preloaded(acc, w0, sc0);
    } else if constexpr (XL) {
        stage_x_quant<WV>(it, xl);
        qr.run(acc);
    } else {
        qr.run(acc);
    }
    const float v = reduce_group<R, G>(acc, lane);
    constexpr int S = G / R; // lanes holding each row's total
    if (seg % S == 0) {
        const int row = wrow0 + sub * R + seg / S;
        if (row < it.M) it.y[row] = v;
    }
}

template <int BITS, int R, int WV, int U, bool XL>
__device__ __forceinline__ void tile_quant(const DevItem &it, int row0, TVL_LDS float *xl)
{
    switch (it.lanes) {
    case 8: tile_quant_g<BITS, 8, R, WV, U, XL>(it, row0, xl); break;
    case 16: tile_quant_g<BITS, 16, R, WV, U, XL>(it, row0, xl); break;
    case 32: tile_quant_g<BITS, 32, R, WV, U, XL>(it, row0, xl); break;
    default: tile_quant_g<BITS, 64, R, WV, U, XL>(it, row0, xl); break;
    }
}

// Any plain item (fp32, fp16, 8-bit or 4-bit weights); XL: the quantised
// ones with x in LDS (the others read x directly).  The choice depends only
// on the item: every wavefront of a workgroup takes the same path.
template <int R, int WV, int U, bool XL>
__device__ __forceinline__ void tile_plain_any(const DevItem &it, int row0, TVL_LDS float *xl)
{
    switch (it.dtype) {
    case 3: tile_quant<4, R, WV, U, XL>(it, row0, xl); break;
    case 2: tile_quant<8, R, WV, U, XL>(it, row0, xl); break;
    case 1: tile_fused<_Float16, R, WV, U, false, false>(it, row0); break;
    default: tile_fused<float, R, WV, U, false, false>(it, row0); break;
    }
}

// XL: dynamic LDS of quant_x_lds_bytes(largest quantised K) per workgroup
template <int R, int WV, int U, bool XL>
__global__ __launch_bounds__(WV *kWave) void k_sweep_quant(const DevItem *__restrict__ items,
                                                            const DevTile *__restrict__ tiles,
                                                            int ntiles)
{
    extern __shared__ f4 qx_lds[];
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) { // workgroup-uniform
        const DevTile tl = tiles[t];
        const DevItem it = items[tl.item];
        tile_plain_any<R, WV, U, XL>(it, tl.row0, (TVL_LDS float *)qx_lds);
        __builtin_amdgcn_s_waitcnt(0x0F70); // as in k_sweep
    }
}

template <int R, int WV, int U, bool XL>
__global__ __launch_bounds__(WV *kWave) void k_item_quant(const DevItem it)
{
    extern __shared__ f4 qx_lds[];
    tile_plain_any<R, WV, U, XL>(it, (int)blockIdx.x * (R * WV * (kWave / it.lanes)),
                                 (TVL_LDS float *)qx_lds);
}

// (R, waves per block, U) for plans holding block-quantised weights:
// direct-x, and with x staged in LDS.
#define TVL_QUANT_SHAPES(X)                                                                       \
    X(2, 4, 2) X(4, 4, 1) X(4, 4, 2) X(4, 1, 2) X(8, 4, 1) X(8, 2, 1)
#define TVL_QUANT_LDS_SHAPES(X) X(4, 4, 1) X(8, 4, 1) X(8, 2, 1) X(4, 4, 2)

template <int R, int WV, int U, bool XL>
struct InstQuant {
    static hipError_t sweep(const DevItem *items, const DevTile *tiles, int ntiles, int grid,
                            int xbytes, hipStream_t st)
    {
        hipLaunchKernelGGL((k_sweep_quant<R, WV, U, XL>), dim3(grid), dim3(WV * kWave),
                           XL ? xbytes : 0, st, items, tiles, ntiles);
        return hipGetLastError();
    }
    static hipError_t item(const DevItem &it, int xbytes, hipStream_t st)
    {
        const int rows = R * WV * (kWave / it.lanes);
        const dim3 grid((it.M + rows - 1) / rows), block(WV * kWave);
        hipLaunchKernelGGL((k_item_quant<R, WV, U, XL>), grid, block, XL ? xbytes : 0, st, it);
        return hipGetLastError();
    }
};

}  // namespace

bool quant_shape_supported(const Shape &s)
{
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXDirect && s.R == R_ && s.W == W_ && s.U == U_) return true;
    TVL_QUANT_SHAPES(X)
#undef X
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXLds && s.R == R_ && s.W == W_ && s.U == U_) return true;
    TVL_QUANT_LDS_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_sweep_quant(const Shape &s, const DevItem *items, const DevTile *tiles,
                              int ntiles, int grid, int xbytes, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXDirect && s.R == R_ && s.W == W_ && s.U == U_)                              \
        return InstQuant<R_, W_, U_, false>::sweep(items, tiles, ntiles, grid, 0, st);
    TVL_QUANT_SHAPES(X)
#undef X
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXLds && s.R == R_ && s.W == W_ && s.U == U_)                                 \
        return InstQuant<R_, W_, U_, true>::sweep(items, tiles, ntiles, grid, xbytes, st);
    TVL_QUANT_LDS_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_item_quant(const Shape &s, const DevItem &item, int xbytes, hipStream_t st)
{
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXDirect && s.R == R_ && s.W == W_ && s.U == U_)                              \
        return InstQuant<R_, W_, U_, false>::item(item, 0, st);
    TVL_QUANT_SHAPES(X)
#undef X
#define X(R_, W_, U_)                                                                             \
    if (s.xmode == kXLds && s.R == R_ && s.W == W_ && s.U == U_)                                 \
        return InstQuant<R_, W_, U_, true>::item(item, xbytes, st);
    TVL_QUANT_LDS_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

}  // namespace tvl
