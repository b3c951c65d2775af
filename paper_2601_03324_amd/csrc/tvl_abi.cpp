// tvl_abi.cpp -- the C ABI declared in include/tvl.h: argument validation,
// variant choice by shape, sweep plans, K-split workspaces, error reporting.
//
// Every entry point validates all of its arguments before it makes any HIP
// call, so the validation paths run (and are tested) on a host without a GPU.
#include "tvl.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "tvl_internal.h"

using tvl::DevItem;
using tvl::DevTile;
using tvl::Shape;

struct tvl_plan {
    int device = -1;
    bool fused = false;
    int multiB = 0; // > 0: several-vector plan holding B x vectors
    int wmode = 0;  // weight dtypes: 0 fp32 only, 1 fp16 only, 2 both
    bool quant = false; // some item has block-quantised weights
    int qxbytes = 0;    // quantised plan with x in LDS: dynamic LDS per workgroup
    Shape shape{4, 4, 2, tvl::kXLds};
    int ks_cap = 0;
    int ntiles = 0;
    int grid = 0;
    bool captured = false; // a cached plan launched into a graph capture
    DevItem *d_items = nullptr;
    DevTile *d_tiles = nullptr;
    std::vector<tvl_item> items;
};

namespace {

thread_local char g_err[512] = "";

tvl_status fail(tvl_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

tvl_status fail_hip(hipError_t e, const char *what)
{
    return fail(TVL_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

constexpr int64_t kMaxDim = 2147483647LL; // M and tile counts fit in int32
constexpr int64_t kMaxK = 1LL << 30;       // K plus one LDS slice still fits in int32
constexpr int64_t kMaxQuantK = 1LL << 24;  // quantised K and ldw (bytes)
constexpr int64_t kMaxLdsBytes = 160 * 1024; // LDS per workgroup (gfx950)

// Bytes per ldw unit: quantised rows are measured in bytes.
int elem_size(int32_t dt) { return dt == TVL_F16 ? 2 : (dt == TVL_F32 ? 4 : 1); }

bool dtype_ok(int32_t dt) { return dt >= TVL_F32 && dt <= TVL_Q4; }
bool is_quant(int32_t dt) { return dt == TVL_Q8 || dt == TVL_Q4; }

// Bytes of one quantised code row (128-byte aligned); the fp32 scales, one
// per 64 columns, sit in a plane of their own after the M code rows.
int64_t q_row_bytes(int64_t K, int32_t dt)
{
    const int bits = dt == TVL_Q4 ? 4 : 8;
    return ((K * bits + 7) / 8 + 127) / 128 * 128;
}
// Scale plane: M rounded up to 4 rows of ceil(K/64) fp32 scales, in blocks of
// 4 rows (the scale of row i, group g at (i/4)*4*ng + 4*g + i%4).
int64_t q_scale_bytes(int64_t M, int64_t K) { return 4 * ((M + 3) / 4 * 4) * ((K + 63) / 64); }

struct Range {
    uintptr_t b, e; // [b, e)
};

// Validate one GEMV's arguments (no HIP calls).
tvl_status check_one(const void *W, int64_t ldw, int32_t dt, const float *x, const float *y,
                     int64_t M, int64_t K, const char *who)
{
    if (!W || !x || !y) return fail(TVL_ERR_NULL, "%s: W, x and y must be non-NULL", who);
    if (!dtype_ok(dt)) return fail(TVL_ERR_DTYPE, "%s: unknown weight dtype %d", who, (int)dt);
    if (M < 1 || K < 1 || M > kMaxDim || K > kMaxK)
        return fail(TVL_ERR_SHAPE, "%s: need 1 <= M <= 2^31-1 and 1 <= K <= 2^30 (M=%lld K=%lld)",
                    who, (long long)M, (long long)K);
    if (!is_quant(dt) && ldw < K)
        return fail(TVL_ERR_SHAPE, "%s: ldw (%lld) < K (%lld)", who, (long long)ldw,
                    (long long)K);
    if (is_quant(dt) && ldw < q_row_bytes(K, dt))
        return fail(TVL_ERR_SHAPE, "%s: a quantised row of K=%lld needs ldw >= %lld bytes", who,
                    (long long)K, (long long)q_row_bytes(K, dt));
    // quantised kernels address a row tile and the scale plane with 32-bit
    // buffer offsets
    if (is_quant(dt) && (K > kMaxQuantK || ldw > kMaxQuantK))
        return fail(TVL_ERR_SHAPE, "%s: quantised weights need K and ldw <= 2^24 (K=%lld ldw=%lld)",
                    who, (long long)K, (long long)ldw);
    if (is_quant(dt) && q_scale_bytes(M, K) > 0x7fffffffLL)
        return fail(TVL_ERR_SHAPE, "%s: quantised scale plane of %lld bytes exceeds 2^31 - 1", who,
                    (long long)q_scale_bytes(M, K));
    const int s = elem_size(dt);
    // the weight span (with a quantised matrix's scale plane, < 2^31 bytes,
    // checked below) must be addressable: M * ldw * s < 2^61
    if (ldw > (int64_t(1) << 61) / M / s)
        return fail(TVL_ERR_SHAPE, "%s: M * ldw overflows", who);
    if (reinterpret_cast<uintptr_t>(W) % tvl::kLineBytes != 0)
        return fail(TVL_ERR_ALIGN, "%s: W must be 128-byte aligned", who);
    if ((ldw * s) % tvl::kLineBytes != 0)
        return fail(TVL_ERR_ALIGN, "%s: ldw * %d bytes (=%lld) must be a multiple of 128", who, s,
                    (long long)(ldw * s));
    if (reinterpret_cast<uintptr_t>(x) % 16 != 0)
        return fail(TVL_ERR_ALIGN, "%s: x must be 16-byte aligned", who);
    if (reinterpret_cast<uintptr_t>(y) % 4 != 0)
        return fail(TVL_ERR_ALIGN, "%s: y must be 4-byte aligned", who);
    return TVL_OK;
}

// A TVL matrix spans M whole rows of ldw elements: the kernels' 16-byte loads
// may touch the padding of the last row (its values are never used).  A
// quantised matrix also spans its scale plane.
Range w_range(const void *W, int64_t ldw, int32_t dt, int64_t M, int64_t K)
{
    const uintptr_t b = reinterpret_cast<uintptr_t>(W);
    const int64_t n = M * ldw * elem_size(dt) + (is_quant(dt) ? q_scale_bytes(M, K) : 0);
    return {b, b + (uintptr_t)n};
}
Range f_range(const float *p, int64_t n)
{
    const uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return {b, b + (uintptr_t)(n * 4)};
}
bool overlap(const Range &a, const Range &b) { return a.b < b.e && b.b < a.e; }

// Outputs must not overlap each other or any input of the batch.
int64_t nvec(const tvl_item &t) { return t.nrhs > 1 ? t.nrhs : 1; }
// x and y spans: one vector, or nrhs rows at strides ldx / ldy
Range x_range(const tvl_item &t)
{
    return f_range(t.x, nvec(t) > 1 ? (nvec(t) - 1) * t.ldx + t.K : t.K);
}
Range y_range(const tvl_item &t)
{
    return f_range(t.y, nvec(t) > 1 ? (nvec(t) - 1) * t.ldy + t.M : t.M);
}

tvl_status check_alias(const tvl_item *items, int32_t n)
{
    std::vector<Range> wr(n);
    for (int32_t i = 0; i < n; ++i)
        wr[i] = y_range(items[i]);
    std::vector<int32_t> ord(n);
    for (int32_t i = 0; i < n; ++i)
        ord[i] = i;
    std::sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) { return wr[a].b < wr[b].b; });
    for (int32_t i = 1; i < n; ++i)
        if (overlap(wr[ord[i - 1]], wr[ord[i]]))
            return fail(TVL_ERR_ALIAS, "items %d and %d: outputs overlap", (int)ord[i - 1],
                        (int)ord[i]);
    std::vector<Range> sorted(n);
    for (int32_t i = 0; i < n; ++i)
        sorted[i] = wr[ord[i]];
    auto hits = [&](const Range &r) -> int32_t {
        // last output starting before r ends; outputs are disjoint and sorted
        auto it = std::lower_bound(sorted.begin(), sorted.end(), r.e,
                                   [](const Range &a, uintptr_t v) { return a.b < v; });
        if (it == sorted.begin()) return -1;
        --it;
        return overlap(*it, r) ? ord[it - sorted.begin()] : -1;
    };
    for (int32_t i = 0; i < n; ++i) {
        const tvl_item &t = items[i];
        int32_t h = hits(w_range(t.W, t.ldw, t.dtype, t.M, t.K));
        if (h >= 0)
            return fail(TVL_ERR_ALIAS, "output of item %d overlaps W of item %d", (int)h, (int)i);
        h = hits(x_range(t));
        if (h >= 0)
            return fail(TVL_ERR_ALIAS, "output of item %d overlaps x of item %d", (int)h, (int)i);
        if (t.op == TVL_OP_SWIGLU) {
            h = hits(w_range(t.W3, t.ldw, t.dtype, t.M, t.K));
            if (h >= 0)
                return fail(TVL_ERR_ALIAS, "output of item %d overlaps W3 of item %d", (int)h,
                            (int)i);
        }
        if (t.g) {
            h = hits(f_range(t.g, t.K));
            if (h >= 0)
                return fail(TVL_ERR_ALIAS, "output of item %d overlaps g of item %d", (int)h,
                            (int)i);
        }
    }
    return TVL_OK;
}

bool is_fused(const tvl_item &t) { return t.op != TVL_OP_GEMV || t.g != nullptr; }
bool is_multi(const tvl_item &t) { return t.nrhs > 1; }

// The item's GEMV arguments plus its RMSNorm / SwiGLU fields.
tvl_status check_fused(const tvl_item &t, const char *who)
{
    tvl_status st = check_one(t.W, t.ldw, t.dtype, t.x, t.y, t.M, t.K, who);
    if (st != TVL_OK) return st;
    if (t.nrhs < 0 || t.nrhs > 16) return fail(TVL_ERR_ARG, "%s: nrhs must be 0..16", who);
    if (t.nrhs > 1) {
        if (t.op != TVL_OP_GEMV || t.g)
            return fail(TVL_ERR_ARG, "%s: several x vectors only for plain GEMV items", who);
        if (t.ldx < t.K || t.ldy < t.M)
            return fail(TVL_ERR_SHAPE, "%s: need ldx >= K and ldy >= M", who);
        if (t.ldx % 4 != 0)
            return fail(TVL_ERR_ALIGN, "%s: ldx must be a multiple of 4 (16-byte rows)", who);
        if (t.ldx > (int64_t(1) << 40) || t.ldy > (int64_t(1) << 40))
            return fail(TVL_ERR_SHAPE, "%s: ldx or ldy too large", who);
    }
    if (t.op != TVL_OP_GEMV && t.op != TVL_OP_SWIGLU)
        return fail(TVL_ERR_ARG, "%s: unknown op %d", who, (int)t.op);
    if (is_quant(t.dtype) && (t.op != TVL_OP_GEMV || t.g || t.nrhs > 1))
        return fail(TVL_ERR_ARG, "%s: quantised weights only for plain one-vector GEMV items",
                    who);
    if (t.op == TVL_OP_SWIGLU) {
        if (!t.W3) return fail(TVL_ERR_NULL, "%s: a SwiGLU item needs W3", who);
        if (reinterpret_cast<uintptr_t>(t.W3) % tvl::kLineBytes != 0)
            return fail(TVL_ERR_ALIGN, "%s: W3 must be 128-byte aligned", who);
    } else if (t.W3) {
        return fail(TVL_ERR_ARG, "%s: W3 is only for SwiGLU items", who);
    }
    if (t.g) {
        if (reinterpret_cast<uintptr_t>(t.g) % 16 != 0)
            return fail(TVL_ERR_ALIGN, "%s: g must be 16-byte aligned", who);
        if (!std::isfinite(t.eps) || t.eps < 0.f)
            return fail(TVL_ERR_ARG, "%s: eps must be finite and >= 0", who);
    }
    return TVL_OK;
}

tvl_status check_items(const tvl_item *items, int32_t n)
{
    if (n < 0) return fail(TVL_ERR_SHAPE, "sweep: n < 0");
    if (n > 0 && !items) return fail(TVL_ERR_NULL, "sweep: items is NULL");
    for (int32_t i = 0; i < n; ++i) {
        const tvl_item &t = items[i];
        char who[48];
        snprintf(who, sizeof who, "sweep item %d", (int)i);
        const tvl_status st = check_fused(t, who);
        if (st != TVL_OK) return st;
    }
    bool any_fused = false, any_multi = false, any_quant = false;
    for (int32_t i = 0; i < n; ++i) {
        any_fused = any_fused || is_fused(items[i]);
        any_multi = any_multi || is_multi(items[i]);
        any_quant = any_quant || is_quant(items[i].dtype);
    }
    if ((any_fused ? 1 : 0) + (any_multi ? 1 : 0) + (any_quant ? 1 : 0) > 1)
        return fail(TVL_ERR_ARG, "sweep: several-vector, RMSNorm/SwiGLU and quantised items "
                                 "need separate launches");
    return check_alias(items, n);
}


// x vectors a several-vector kernel must hold: the next power of two >= n
// (the matrix-core form holds any number up to 16)
int multi_B(int n) { return n <= 2 ? 2 : n <= 4 ? 4 : n <= 8 ? 8 : 16; }

// Default several-vector shape (direct-x), by B, measured on MI355X on the
// 110M decode token and a 70B-shaped fp16 layer.  Up to 4 vectors the VALU
// form wins: more rows per wavefront amortise each x read over more weights
// (3-4 vectors: 8 rows, 6.36-6.39 TB/s against 6.09-6.10 with 4 rows on the
// 110M token; fp16, 2 wavefronts per block: 6.02-6.10 against 5.62-5.75;
// 2 fp16 vectors: 6.36 against 6.09-6.17, while 2 fp32 vectors keep 4 rows,
// 7.00-7.01 against 6.90-6.91), and one load in flight keeps the R x B
// accumulators in registers.  From 5 vectors on,
// the FMAs would take ~half the VALU issue slots and the matrix cores win.
// fp32 weights: the 16 x 16 x 4 form with the weights streamed into LDS and
// x shared by the block's four wavefronts (16 rows each, 64-column chunks;
// 8 vectors: 6.05-6.10 TB/s against 5.55-5.92 streamed with x per wavefront,
// 5.43-5.49 for the LDS-staged form, 4.73 for the 4 x 4 x 1 form and 4.07 on
// the VALU; 16 vectors: 5.48-5.51 against 4.96-5.08 streamed, 4.88-4.90
// LDS-staged and 3.68 for the direct-load form).  Launches with only fp16 weights (one
// 70B-shaped layer), 5-16 vectors: the streamed form on the fp16 matrix
// cores with x split in two fp16 parts once per block and shared by the
// block's four wavefronts (16 rows each, 128-column chunks; 8 vectors: 6.15
// TB/s against 5.67-5.98 for 2 or 8 wavefronts or 32 rows, 5.73 with x per
// wavefront (32 rows), 4.64 on the fp32 matrix cores and 4.48 for 4 x 4 x 1;
// 16: 6.01 against 5.68-5.82 for 2 or 8 wavefronts or 32 rows, 4.84 with x
// per wavefront and 3.60 for the LDS-staged form, where each converted fp16
// chunk costs as many fp32 matrix-core steps as an fp32 chunk of twice the
// bytes).  Launches mixing
// fp32 and fp16 weights: the streamed form with x per wavefront (32 rows)
// with 5-8 vectors, the LDS-staged form with 16 rows beyond.
Shape default_multi_shape(int B, bool all_f32, bool all_f16)
{
    if (B > 4 && all_f32) return Shape{16, 4, 202, tvl::kXDirect};
    if (B > 4 && all_f16) return Shape{16, 4, 303, tvl::kXDirect};
    if (B > 8) return Shape{16, 1, 2, tvl::kXDirect};
    if (B > 4) return Shape{32, 1, 32, tvl::kXDirect};
    if (B == 4) return all_f16 ? Shape{8, 2, 1, tvl::kXDirect} : Shape{8, 4, 1, tvl::kXDirect};
    return all_f16 ? Shape{8, 2, 1, tvl::kXDirect} : Shape{4, 4, 2, tvl::kXDirect};
}

int quant_bits(int32_t dt) { return dt == TVL_Q4 ? 4 : 8; }

// Lanes per row of an item (block-quantised weights may share a wavefront
// between several short rows; every other item uses all 64 lanes).
int item_lanes(const tvl_item &t, bool few_lanes = false)
{
    return is_quant(t.dtype) ? tvl::quant_lanes(t.K, quant_bits(t.dtype), few_lanes) : 64;
}

tvl::DevItem dev_item(const tvl_item &t, bool few_lanes = false)
{
    return tvl::DevItem{t.W,    t.ldw, t.x,   t.y,        (int32_t)t.M, (int32_t)t.K,
                        t.dtype, t.op, t.W3, t.g,        t.eps,        (int32_t)nvec(t),
                        t.ldx,  t.ldy, item_lanes(t, few_lanes && t.dtype == TVL_Q4), 0};
}

tvl_status check_tuning(const tvl_tuning *t, bool allow_ksplit)
{
    if (!t) return TVL_OK;
    if (t->rows_per_wave < 0 || t->waves_per_block < 0 || t->unroll < 0 || t->ksplit < 0 ||
        t->grid < 0 || (t->flags & ~(TVL_FLAG_X_LDS | TVL_FLAG_X_DIRECT)) != 0)
        return fail(TVL_ERR_ARG, "tuning: negative field or unknown flag");
    if ((t->flags & TVL_FLAG_X_LDS) && (t->flags & TVL_FLAG_X_DIRECT))
        return fail(TVL_ERR_ARG, "tuning: TVL_FLAG_X_LDS and TVL_FLAG_X_DIRECT exclude each other");
    if (!allow_ksplit && t->ksplit > 1)
        return fail(TVL_ERR_ARG, "tuning: ksplit applies to tvl_gemv only");
    if (t->ksplit > 1024) return fail(TVL_ERR_ARG, "tuning: ksplit > 1024");
    return TVL_OK;
}

// ---------------------------------------------------------------- devices
struct DevInfo {
    int cus = 256;
    int xcds = 8; // gfx950: 32 compute units per XCD
};

std::mutex g_mu;
std::map<int, DevInfo> g_dev;

tvl_status current_device(int *dev, DevInfo *info)
{
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_dev.find(*dev);
    if (it == g_dev.end()) {
        DevInfo d;
        int cus = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, *dev);
        if (e != hipSuccess) return fail_hip(e, "hipDeviceGetAttribute");
        if (cus > 0) d.cus = cus;
        d.xcds = d.cus >= 64 ? d.cus / 32 : 1;
        it = g_dev.emplace(*dev, d).first;
    }
    *info = it->second;
    return TVL_OK;
}

// Default launch shape for a set of GEMVs, from the bytes they stream
// (measured on MI355X over every instantiated shape, both x modes):
//   mostly fp16 weights                  -> direct-x, R=4, W=1, U=4
//   fp32, rows of <= 3 KB (K <= 768)     -> direct-x, R=2, W=4, U=3 (one batch
//                                           covers the row)
//   fp32, rows of <= 8 KB (K <= 2048)    -> direct-x, R=2, W=4, U=4; in a
//                                           sweep R=2, W=8, U=3 (the 110M
//                                           token: 7.03 against 6.91 TB/s)
//   fp32, longer rows                    -> direct-x, R=1, W=4, U=8
// Direct-x reads x next to the weights, so no wavefront waits on a staging
// round trip; with fp16 weights each 16-byte load needs 32 bytes of x, so
// more rows per wavefront (R=4) share each x read.  `sweep`: a plan's one
// launch over many GEMVs (a single GEMV of short rows is faster with 4
// wavefronts per workgroup: more workgroups share the few rows).
Shape default_shape(double bytes_f16, double bytes_f32, double f32_row_bytes_weighted,
                    bool sweep)
{
    if (bytes_f16 > bytes_f32) return Shape{4, 1, 4, tvl::kXDirect};
    if (f32_row_bytes_weighted <= 3072.0) return Shape{2, 4, 3, tvl::kXDirect};
    if (f32_row_bytes_weighted <= 8192.0)
        return sweep ? Shape{2, 8, 3, tvl::kXDirect} : Shape{2, 4, 4, tvl::kXDirect};
    return Shape{1, 4, 8, tvl::kXDirect};
}

// Default shape for items with a fused RMSNorm or SwiGLU (direct-x only,
// an even R so a SwiGLU pair fits in one wavefront).  Measured on MI355X
// over every fused shape: the 110M decode token (fp32) runs best at
// (4, 4, 3) (6.88-6.91 TB/s against 6.53-6.61 at (2, 4, 3)), the 70B-shaped
// layers (fp16) at (8, 2, 1) (6.92 against 6.72 at (4, 4, 2)).  A fused item
// reads g next to x, so more rows per wavefront share both (x and g bytes
// per weight byte: 2 / (R · weight size) per 16-byte load).
Shape default_fused_shape(double bytes_f16, double bytes_f32)
{
    return bytes_f16 > bytes_f32 ? Shape{8, 2, 1, tvl::kXDirect} : Shape{4, 4, 3, tvl::kXDirect};
}

// Default shape for plans or items with block-quantised weights (from
// sweeps of the 110M and 7B tokens, 8- and 4-bit, on MI355X): 8 rows per
// lane group, except for 8-bit launches of under 1 GB of codes, which get 4
// (twice the wavefronts for a launch too short to reach full bandwidth;
// 110M token: 5.64 against 5.34-5.38 TB/s; 7B: 6.34 against 6.51, 4-bit 7B:
// 4.16 against 5.73, 4-bit 110M: 3.14 against 3.82).  Launches of >= 1 GB
// of codes read x from LDS, staged once per row tile, when it fits three
// workgroups per CU (K <= 13,312): 4-bit ones (8-lane groups, whose x loads
// were as many as their code loads) at 8 rows, one chunk in flight (7B
// 4-bit token: 6.61 against 6.35 TB/s); 8-bit ones at 4 rows with two
// chunks in flight, which x in LDS leaves room for in registers (7B 8-bit
// token: 7.12-7.13 against 7.00-7.01 TB/s at (8, 4, 1) with direct x, 6.96
// at (8, 4, 1) with x in LDS, 6.54 at (4, 4, 2) with direct x).  The 110M
// tokens are 1-2 % slower with x in LDS and keep direct x.  qbytes: code
// bytes of the launch's quantised items; q4: any of them 4-bit; kq: their
// largest K.
Shape default_quant_shape(double qbytes, bool q4, int64_t kq)
{
    if (!q4 && qbytes < 1e9) return Shape{4, 4, 1, tvl::kXDirect};
    if (qbytes >= 1e9 && tvl::quant_x_lds_bytes(kq) <= 52 * 1024)
        return q4 ? Shape{8, 4, 1, tvl::kXLds} : Shape{4, 4, 2, tvl::kXLds};
    return Shape{8, 4, 1, tvl::kXDirect};
}

Shape default_shape_items(const tvl_item *items, int32_t n)
{
    double b16 = 0, b32 = 0, row32 = 0;
    for (int32_t i = 0; i < n; ++i) {
        const double b = (double)items[i].M * (double)items[i].K * elem_size(items[i].dtype);
        if (items[i].dtype == TVL_F16) {
            b16 += b;
        } else {
            b32 += b;
            row32 += b * (double)items[i].K * 4.0;
        }
    }
    bool fused = false;
    int nmax = 1;
    for (int32_t i = 0; i < n; ++i) {
        fused = fused || is_fused(items[i]);
        nmax = std::max<int>(nmax, (int)nvec(items[i]));
    }
    bool quant = false, q4 = false;
    double qbytes = 0;
    int64_t kq = 1;
    for (int32_t i = 0; i < n; ++i)
        if (is_quant(items[i].dtype)) {
            quant = true;
            q4 = q4 || items[i].dtype == TVL_Q4;
            qbytes += (double)items[i].M * (double)items[i].K * quant_bits(items[i].dtype) / 8;
            kq = std::max<int64_t>(kq, items[i].K);
        }
    if (quant) return default_quant_shape(qbytes, q4, kq);
    if (nmax > 1) return default_multi_shape(multi_B(nmax), b16 == 0, b32 == 0);
    if (fused) return default_fused_shape(b16, b32);
    return default_shape(b16, b32, b32 > 0 ? row32 / b32 : 0.0, true);
}

int64_t item_bytes_factor(const tvl_item &t) { return t.op == TVL_OP_SWIGLU ? 2 : 1; }

// Shape from a tuning override, else the default.
// `plain`: check against the plain GEMV kernels (callers that launch the
// fused or several-vector kernels check their own lists).
tvl_status pick_shape(const tvl_tuning *t, Shape def, Shape *out, bool plain = true)
{
    Shape s = def;
    if (t) {
        if (t->rows_per_wave) s.R = t->rows_per_wave;
        if (t->waves_per_block) s.W = t->waves_per_block;
        if (t->unroll) s.U = t->unroll;
        if (t->flags & TVL_FLAG_X_LDS) s.xmode = tvl::kXLds;
        if (t->flags & TVL_FLAG_X_DIRECT) s.xmode = tvl::kXDirect;
        if (!t->rows_per_wave && !t->waves_per_block && !t->unroll && s.xmode != def.xmode) {
            // x mode forced, shape left to the library: the mode's all-rounder
            s.R = 2;
            s.W = 4;
            s.U = 4;
        }
        if (t->rows_per_wave && !t->unroll) {
            // keep about 16 KB of weights in flight per wavefront by default
            // (R >= 32: the 16 x 16 x 4 several-vector form, 4 loads per group)
            s.U = s.R >= 32 ? 4 : s.R >= 4 ? 2 : s.R == 2 ? 4 : 8;
        }
    }
    if (plain && !tvl::shape_supported(s))
        return fail(TVL_ERR_ARG, "tuning: (rows_per_wave %d, waves_per_block %d, unroll %d) is "
                                 "not an instantiated %s shape",
                    s.R, s.W, s.U, s.xmode == tvl::kXLds ? "LDS-x" : "direct-x");
    *out = s;
    return TVL_OK;
}

// Shape of a launch with quantised items: as pick_shape, but a tuning that
// forces only the x mode keeps the default rows and waves (they exist in both
// modes).  With x in LDS, xbytes is the dynamic LDS its largest quantised K
// needs, which must fit a workgroup's LDS.
tvl_status pick_quant_shape(const tvl_tuning *t, Shape def, int64_t kq, Shape *out, int *xbytes,
                            const char *who)
{
    tvl_status st = pick_shape(t, def, out, false);
    if (st != TVL_OK) return st;
    if (t && !t->rows_per_wave && !t->waves_per_block && !t->unroll) {
        out->R = def.R;
        out->W = def.W;
        out->U = def.U;
    }
    if (!tvl::quant_shape_supported(*out))
        return fail(TVL_ERR_ARG, "%s: no quantised-weight kernel for (%d, %d, %d) %s", who, out->R,
                    out->W, out->U, out->xmode == tvl::kXLds ? "LDS-x" : "direct-x");
    *xbytes = 0;
    if (out->xmode == tvl::kXLds) {
        const int64_t b = tvl::quant_x_lds_bytes(kq);
        if (b > kMaxLdsBytes)
            return fail(TVL_ERR_SHAPE, "%s: quantised weights with x in LDS: x of K=%lld needs "
                                       "%lld bytes, more than a workgroup's %lld (use direct x)",
                        who, (long long)kq, (long long)b, (long long)kMaxLdsBytes);
        *xbytes = (int)b;
    }
    return TVL_OK;
}

// ---------------------------------------------------------- K-split workspace
struct Workspace {
    float *partials = nullptr;
    int64_t partial_cap = 0; // floats
    int *counters = nullptr;
    int64_t counter_cap = 0; // ints
};
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
// Workspaces replaced by larger ones.  They are not freed until
// tvl_release_workspaces: a graph captured earlier may still use them, and
// launches already enqueued on the stream may too.
std::vector<std::pair<int, Workspace>> g_ws_retired;

// The caller holds g_mu, and keeps holding it until it has launched the
// kernel that uses the workspace: another thread growing the same stream's
// workspace, or tvl_release_workspaces, would otherwise free the buffers
// between this lookup and that launch.
tvl_status get_workspace_locked(int dev, hipStream_t st, int64_t nfloat, int64_t ncnt,
                                Workspace *out)
{
    Workspace &w = g_ws[{dev, st}];
    if (w.partial_cap < nfloat || w.counter_cap < ncnt) {
        hipError_t e;
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(st, &cap) == hipSuccess && cap != hipStreamCaptureStatusNone)
            return fail(TVL_ERR_NOMEM, "K-split workspace: stream %p is being captured and its "
                                       "workspace (%lld floats) is not allocated yet; run the "
                                       "same K-split call once on this stream before capture",
                        (void *)st, (long long)nfloat);
        const int64_t pf = std::max<int64_t>({nfloat, w.partial_cap, 1 << 16});
        const int64_t pc = std::max<int64_t>({ncnt, w.counter_cap, 1 << 12});
        Workspace nw;
        e = hipMalloc(&nw.partials, pf * sizeof(float));
        if (e != hipSuccess) return fail(TVL_ERR_NOMEM, "K-split workspace: %s", hipGetErrorString(e));
        e = hipMalloc(&nw.counters, pc * sizeof(int));
        if (e != hipSuccess) {
            (void)hipFree(nw.partials);
            return fail(TVL_ERR_NOMEM, "K-split workspace: %s", hipGetErrorString(e));
        }
        e = tvl::launch_zero_i32(nw.counters, pc, st);
        if (e != hipSuccess) {
            (void)hipFree(nw.partials);
            (void)hipFree(nw.counters);
            return fail_hip(e, "counter reset launch");
        }
        nw.partial_cap = pf;
        nw.counter_cap = pc;
        // the old buffers stay allocated (earlier launches and captured
        // graphs may use them) until tvl_release_workspaces
        if (w.partials || w.counters) g_ws_retired.emplace_back(dev, w);
        w = nw;
    }
    *out = w;
    return TVL_OK;
}

// XCD-aware tile order.  The dispatcher deals a launch's workgroups to the
// XCDs in turn (workgroup b to XCD b mod nx), and with one tile per
// workgroup tile b runs there too.  Each XCD's L2 fetches an item's x vectors
// once for the tiles it runs, so an item whose tiles are dealt over all XCDs
// has its x fetched nx times: at 16 x vectors that is several percent of a
// launch's bytes.  `tiles` is ordered longest tile first, each item's tiles
// contiguous, and key[t] is the bytes per row of tile t.  Each class of
// equally long tiles is cut into nx contiguous runs of equal length (the
// remainders going to XCDs in rotation), run c to XCD c, so an item spans one
// or two XCDs unless it is longer than a run; the XCD lists are then dealt
// back into the table (entry nx j + c: XCD c's j-th tile).  Every XCD gets as
// many tiles of every class as the others, plus at most one, so their bytes
// stay balanced, and each list keeps the longest tiles first.
std::vector<DevTile> xcd_order(const std::vector<DevTile> &tiles, const std::vector<int64_t> &key,
                               int nx)
{
    std::vector<std::vector<DevTile>> lists(nx);
    size_t a = 0;
    int rot = 0;
    while (a < tiles.size()) {
        size_t b = a;
        while (b < tiles.size() && key[b] == key[a])
            ++b;
        const size_t n = b - a, base = n / nx;
        const int rem = (int)(n % nx);
        size_t pos = a;
        for (int c = 0; c < nx; ++c) {
            const size_t len = base + (((c - rot) % nx + nx) % nx < rem ? 1 : 0);
            lists[c].insert(lists[c].end(), tiles.begin() + pos, tiles.begin() + pos + len);
            pos += len;
        }
        rot = (rot + rem) % nx;
        a = b;
    }
    std::vector<DevTile> out;
    out.reserve(tiles.size());
    for (size_t j = 0; out.size() < tiles.size(); ++j)
        for (int c = 0; c < nx; ++c)
            if (j < lists[c].size()) out.push_back(lists[c][j]);
    return out;
}

// -------------------------------------------------------------- plans
tvl_status plan_build(const tvl_item *items, int32_t n, const tvl_tuning *tuning, tvl_plan **out)
{
    bool special = false;
    for (int32_t i = 0; i < n; ++i)
        special = special || is_fused(items[i]) || is_multi(items[i]) || is_quant(items[i].dtype);
    // every argument check before the first HIP call
    bool fused = false, quant = false, f32 = false, f16 = false;
    int nmax = 1;
    int64_t kq = 1; // largest quantised K
    for (int32_t i = 0; i < n; ++i) {
        fused = fused || is_fused(items[i]);
        quant = quant || is_quant(items[i].dtype);
        nmax = std::max<int>(nmax, (int)nvec(items[i]));
        (items[i].dtype == TVL_F16 ? f16 : f32) = true;
        if (is_quant(items[i].dtype)) kq = std::max<int64_t>(kq, items[i].K);
    }
    Shape shape;
    int qxbytes = 0;
    tvl_status st = quant ? pick_quant_shape(tuning, default_shape_items(items, n), kq, &shape,
                                             &qxbytes, "plan")
                          : pick_shape(tuning, default_shape_items(items, n), &shape, !special);
    if (st != TVL_OK) return st;
    const int multiB = nmax > 1 ? multi_B(nmax) : 0;
    if (nmax > 1) {
        if (fused)
            return fail(TVL_ERR_ARG, "plan: several-vector items cannot share a plan with "
                                     "RMSNorm or SwiGLU items");
        if (!tvl::multi_shape_supported(shape, multiB))
            return fail(TVL_ERR_ARG, "plan: no several-vector kernel for (%d, %d, %d) with %d "
                                     "vectors",
                        shape.R, shape.W, shape.U, multiB);
    }
    if (fused && !tvl::fused_shape_supported(shape))
        return fail(TVL_ERR_ARG, "plan: items with RMSNorm or SwiGLU need a direct-x shape with "
                                 "fused support; (%d, %d, %d) %s has none",
                    shape.R, shape.W, shape.U, shape.xmode == tvl::kXLds ? "LDS-x" : "direct-x");
    int dev = 0;
    DevInfo info;
    st = current_device(&dev, &info);
    if (st != TVL_OK) return st;

    tvl_plan *p = new (std::nothrow) tvl_plan;
    if (!p) return fail(TVL_ERR_NOMEM, "plan: host allocation");
    p->device = dev;
    p->shape = shape;
    p->items.assign(items, items + n);
    p->fused = fused;
    p->quant = quant;
    p->qxbytes = qxbytes;
    p->multiB = multiB;
    p->wmode = f32 && f16 ? 2 : f16 ? 1 : 0;
    // output rows per tile: a SwiGLU tile streams R rows of W and of W3 per
    // wavefront, i.e. R/2 output rows; a quantised item whose rows share a
    // wavefront in groups of G lanes covers 64 / G times R rows per wavefront
    // 4-bit rows in launches of >= 1 GB of codes take the fewest lanes per
    // row that pad no more (see tvl::quant_lanes)
    double qbytes = 0;
    for (int32_t i = 0; i < n; ++i)
        if (is_quant(items[i].dtype))
            qbytes += (double)items[i].M * (double)items[i].K * quant_bits(items[i].dtype) / 8;
    const bool few_lanes = qbytes >= 1e9;
    auto lanes_of = [&](const tvl_item &t) {
        return item_lanes(t, few_lanes && t.dtype == TVL_Q4);
    };
    auto rows_of = [&](const tvl_item &t) {
        return (t.op == TVL_OP_SWIGLU ? shape.R / 2 : shape.R) * shape.W * (64 / lanes_of(t));
    };
    // bytes per tile, largest first, so the longest tiles start first
    std::vector<int32_t> ord(n);
    for (int32_t i = 0; i < n; ++i)
        ord[i] = i;
    std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) {
        return items[a].K * elem_size(items[a].dtype) * item_bytes_factor(items[a]) >
               items[b].K * elem_size(items[b].dtype) * item_bytes_factor(items[b]);
    });
    std::vector<DevItem> hitems(n);
    std::vector<DevTile> htiles;
    int64_t ntiles = 0;
    int64_t kmax = 1;
    for (int32_t i = 0; i < n; ++i) {
        const tvl_item &t = items[i];
        hitems[i] = dev_item(t, few_lanes);
        ntiles += (t.M + rows_of(t) - 1) / rows_of(t);
        kmax = std::max<int64_t>(kmax, t.K);
    }
    if (ntiles > kMaxDim) {
        delete p;
        return fail(TVL_ERR_SHAPE, "plan: %lld tiles exceed 2^31-1", (long long)ntiles);
    }
    htiles.reserve((size_t)ntiles);
    std::vector<int64_t> tkey;
    tkey.reserve((size_t)ntiles);
    for (int32_t k = 0; k < n; ++k) {
        const int32_t i = ord[k];
        for (int64_t r = 0; r < items[i].M; r += rows_of(items[i])) {
            htiles.push_back(DevTile{i, (int32_t)r});
            tkey.push_back(items[i].K * elem_size(items[i].dtype) * item_bytes_factor(items[i]));
        }
    }
    // Several x vectors per item, or quantised rows (32 x floats per 16 code
    // bytes): each XCD fetches the x of the items it runs, so keep every item
    // on as few XCDs as possible (measured on MI355X: +5 % for 8 and 16
    // vectors, +7 % for 4, +1-2 % for the 8- and 4-bit 110M tokens; the plain
    // fp32 sweep, whose x is 0.5 % of its bytes, keeps one global order)
    if ((multiB || quant) && info.xcds > 1) htiles = xcd_order(htiles, tkey, info.xcds);
    p->ntiles = (int)ntiles;
    p->ks_cap = tvl::slice_cap(kmax);
    p->grid = (tuning && tuning->grid) ? std::min<int>(tuning->grid, std::max(p->ntiles, 1))
                                       : p->ntiles;
    if (n > 0) {
        hipError_t e = hipMalloc(&p->d_items, sizeof(DevItem) * n);
        if (e == hipSuccess) e = hipMalloc(&p->d_tiles, sizeof(DevTile) * htiles.size());
        if (e == hipSuccess)
            e = hipMemcpy(p->d_items, hitems.data(), sizeof(DevItem) * n, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = hipMemcpy(p->d_tiles, htiles.data(), sizeof(DevTile) * htiles.size(),
                          hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(p->d_items);
            (void)hipFree(p->d_tiles);
            delete p;
            return fail(e == hipErrorOutOfMemory ? TVL_ERR_NOMEM : TVL_ERR_HIP,
                        "plan upload: %s", hipGetErrorString(e));
        }
    }
    *out = p;
    return TVL_OK;
}

tvl_status plan_launch(const tvl_plan *p, hipStream_t st)
{
    if (p->ntiles == 0) return TVL_OK;
    const hipError_t e =
        p->quant    ? tvl::launch_sweep_quant(p->shape, p->d_items, p->d_tiles, p->ntiles, p->grid,
                                              p->qxbytes, st)
        : p->multiB ? tvl::launch_sweep_multi(p->shape, p->multiB, p->wmode, p->d_items,
                                              p->d_tiles, p->ntiles, p->grid, st)
        : p->fused ? tvl::launch_sweep_fused(p->shape, p->d_items, p->d_tiles, p->ntiles, p->grid,
                                             st)
                   : tvl::launch_sweep(p->shape, p->d_items, p->d_tiles, p->ntiles, p->grid,
                                       p->ks_cap, st);
    if (e != hipSuccess) return fail_hip(e, "sweep launch");
    return TVL_OK;
}

void plan_free(tvl_plan *p)
{
    if (!p) return;
    int cur = -1;
    if (hipGetDevice(&cur) == hipSuccess && cur != p->device) (void)hipSetDevice(p->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(p->d_items);
    (void)hipFree(p->d_tiles);
    if (cur >= 0 && cur != p->device) (void)hipSetDevice(cur);
    delete p;
}

// batch-sweep cache: item list bytes + device -> plan
std::map<std::string, tvl_plan *> g_cache;
constexpr size_t kCacheMax = 64;
// evicted plans that were launched into a graph capture (freed only by
// tvl_release_workspaces)
std::vector<tvl_plan *> g_plans_retired;

// First tvl_gemv_noalloc call on a device: look up its static scratch and
// clear the counters (tvl::noalloc_scratch; later calls make no HIP call).
tvl_status noalloc_setup(int dev, hipStream_t stream, float **partials, int **counters)
{
    const hipError_t e = tvl::noalloc_scratch(dev, stream, partials, counters);
    if (e == hipErrorStreamCaptureUnsupported)
        return fail(TVL_ERR_ARG, "tvl_gemv_noalloc: the first call on device %d clears the "
                                 "static scratch and synchronises its stream, so it cannot be "
                                 "captured; make one call before capturing", dev);
    if (e != hipSuccess) return fail_hip(e, "tvl_gemv_noalloc scratch set-up");
    return TVL_OK;
}

// tvl_gemv_ex and tvl_gemv_noalloc: the same variant choice; `noalloc` puts
// the K split's partials and counters in the library's static per-device
// scratch instead of a per-stream workspace.
tvl_status gemv_impl(const void *W, int64_t ldw, int32_t dtype, const float *x, float *y,
                     int64_t M, int64_t K, const tvl_tuning *tuning, hipStream_t stream,
                     bool noalloc)
{
    const char *who = noalloc ? "tvl_gemv_noalloc" : "tvl_gemv";
    tvl_status st = check_one(W, ldw, dtype, x, y, M, K, who);
    if (st != TVL_OK) return st;
    tvl_item it{W, ldw, x, y, M, K, dtype, TVL_OP_GEMV, nullptr, nullptr, 0.f, 1, 0, 0};
    st = check_alias(&it, 1);
    if (st != TVL_OK) return st;
    st = check_tuning(tuning, true);
    if (st != TVL_OK) return st;

    // Variant by shape.  Row split when there are enough row tiles to give
    // every CU several workgroups; otherwise split K so that small-M GEMVs
    // still spread over the whole GPU.
    Shape shape;
    int S = 1;
    const bool user_shape =
        tuning && (tuning->rows_per_wave || tuning->waves_per_block || tuning->unroll);
    if (is_quant(dtype)) {
        if (tuning && tuning->ksplit > 1)
            return fail(TVL_ERR_ARG, "%s: quantised weights have no K split", who);
        Shape qs;
        int qxbytes = 0;
        st = pick_quant_shape(tuning,
                              default_quant_shape((double)M * (double)K * quant_bits(dtype) / 8,
                                                  dtype == TVL_Q4, K),
                              K, &qs, &qxbytes, who);
        if (st != TVL_OK) return st;
        int qdev = 0;
        DevInfo qinfo;
        st = current_device(&qdev, &qinfo);
        if (st != TVL_OK) return st;
        if (noalloc) { // no scratch here; the first call on a device still sets it up
            float *p = nullptr;
            int *c = nullptr;
            st = noalloc_setup(qdev, stream, &p, &c);
            if (st != TVL_OK) return st;
        }
        const hipError_t qe = tvl::launch_item_quant(qs, dev_item(it), qxbytes, stream);
        if (qe != hipSuccess) return fail_hip(qe, "quantised gemv launch");
        return TVL_OK;
    }
    const Shape def = default_shape(dtype == TVL_F16 ? 1.0 : 0.0, dtype == TVL_F16 ? 0.0 : 1.0,
                                    (double)K * 4.0, false);
    shape = def;
    if (user_shape || (tuning && tuning->flags)) {
        st = pick_shape(tuning, def, &shape);
        if (st != TVL_OK) return st;
    }

    int dev = 0;
    DevInfo info;
    st = current_device(&dev, &info);
    if (st != TVL_OK) return st;
    const bool auto_shape = !(user_shape || (tuning && tuning->flags));
    if (auto_shape) {
        // Few rows of more than 4 KB (measured on MI355X for M = 16 .. 1024):
        // one row per single-wavefront workgroup, 8 loads in flight, beats
        // both the large-M shapes and a K split: the split's publish-and-
        // combine step costs more than it saves unless rows are long and
        // very few.  Rows of <= 4 KB take one batch of loads anyway.
        const int64_t blocks = (M + def.R * def.W - 1) / (def.R * def.W);
        const int64_t row_bytes = K * elem_size(dtype);
        if (blocks < 2LL * info.cus && row_bytes > 4096) shape = Shape{1, 1, 8, tvl::kXDirect};
        if (!(tuning && tuning->ksplit) && M <= 128 && row_bytes >= 32768) {
            shape = Shape{1, 1, 4, tvl::kXDirect};
            S = (int)std::min<int64_t>(4, std::max<int64_t>(2, 256 / M));
        }
    }
    const int rows_per_tile = shape.R * shape.W;
    const int64_t tiles = (M + rows_per_tile - 1) / rows_per_tile;
    if (tuning && tuning->ksplit) S = tuning->ksplit;
    if (S > 1 && (int64_t)tiles * S > kMaxDim)
        return fail(TVL_ERR_ARG, "%s: grid too large", who);
    if (noalloc && S > 1 &&
        ((int64_t)S * M > tvl::kNoallocPartials || tiles > tvl::kNoallocCounters))
        return fail(TVL_ERR_SHAPE,
                    "tvl_gemv_noalloc: a K split of %lld rows into %d slices needs %lld partials "
                    "and %lld counters; the static scratch holds %lld and %lld",
                    (long long)M, S, (long long)S * M, (long long)tiles,
                    (long long)tvl::kNoallocPartials, (long long)tvl::kNoallocCounters);
    float *ns_partials = nullptr;
    int *ns_counters = nullptr;
    if (noalloc) { // every check done: the first call on a device sets the scratch up
        st = noalloc_setup(dev, stream, &ns_partials, &ns_counters);
        if (st != TVL_OK) return st;
    }
    hipError_t e;
    if (S <= 1) {
        e = tvl::launch_gemv_rows(shape, dtype, W, ldw, x, y, (int)M, (int)K, stream);
    } else {
        if (noalloc) {
            e = tvl::launch_gemv_ksplit(shape, dtype, W, ldw, x, y, (int)M, (int)K, S,
                                        ns_partials, ns_counters, stream);
        } else {
            Workspace ws;
            std::lock_guard<std::mutex> lk(g_mu); // until the launch (see get_workspace_locked)
            st = get_workspace_locked(dev, stream, (int64_t)S * M, tiles, &ws);
            if (st != TVL_OK) return st;
            e = tvl::launch_gemv_ksplit(shape, dtype, W, ldw, x, y, (int)M, (int)K, S,
                                        ws.partials, ws.counters, stream);
        }
    }
    if (e != hipSuccess) return fail_hip(e, noalloc ? "tvl_gemv_noalloc launch" : "gemv launch");
    return TVL_OK;
}


}  // namespace

// ================================================================== ABI
extern "C" {

int32_t tvl_version(void) { return TVL_VERSION; }

int64_t tvl_row_stride(int64_t K, int32_t dtype)
{
    if (K < 1 || !dtype_ok(dtype)) return -1;
    if (is_quant(dtype)) return K > kMaxK ? -1 : q_row_bytes(K, dtype);
    const int s = elem_size(dtype);
    if (K > (INT64_MAX - tvl::kLineBytes) / s) return -1;
    return (K * s + tvl::kLineBytes - 1) / tvl::kLineBytes * tvl::kLineBytes / s;
}

tvl_status tvl_pack_rows(void *dst, int64_t ldw, const void *src, int64_t M, int64_t K,
                         int32_t dtype, hipStream_t stream)
{
    g_err[0] = 0;
    if (!dst || !src) return fail(TVL_ERR_NULL, "tvl_pack_rows: dst and src must be non-NULL");
    if (!dtype_ok(dtype) || is_quant(dtype))
        return fail(TVL_ERR_DTYPE, "tvl_pack_rows: dtype %d (fp32 and fp16 only)", (int)dtype);
    if (M < 1 || K < 1 || M > kMaxDim || K > kMaxK || ldw < K)
        return fail(TVL_ERR_SHAPE, "tvl_pack_rows: need 1 <= M <= 2^31-1, 1 <= K <= 2^30, "
                                   "ldw >= K");
    const int s = elem_size(dtype);
    if (ldw > (int64_t(1) << 62) / s / M) return fail(TVL_ERR_SHAPE, "tvl_pack_rows: overflow");
    if (reinterpret_cast<uintptr_t>(dst) % tvl::kLineBytes != 0 || (ldw * s) % tvl::kLineBytes)
        return fail(TVL_ERR_ALIGN, "tvl_pack_rows: dst rows must start on 128-byte boundaries");
    if (reinterpret_cast<uintptr_t>(src) % s != 0)
        return fail(TVL_ERR_ALIGN, "tvl_pack_rows: src must be element aligned");
    const Range d = w_range(dst, ldw, dtype, M, K);
    const Range r = w_range(src, K, dtype, M, K);
    if (overlap(d, r)) return fail(TVL_ERR_ALIAS, "tvl_pack_rows: dst overlaps src");
    const hipError_t e = tvl::launch_pack(dtype, dst, ldw, src, M, K, stream);
    if (e != hipSuccess) return fail_hip(e, "pack launch");
    return TVL_OK;
}

tvl_status tvl_gemv_ex(const void *W, int64_t ldw, int32_t dtype, const float *x, float *y,
                       int64_t M, int64_t K, const tvl_tuning *tuning, hipStream_t stream)
{
    g_err[0] = 0;
    return gemv_impl(W, ldw, dtype, x, y, M, K, tuning, stream, false);
}

tvl_status tvl_gemv_noalloc(const void *W, int64_t ldw, int32_t dtype, const float *x, float *y,
                            int64_t M, int64_t K, const tvl_tuning *tuning, hipStream_t stream)
{
    g_err[0] = 0;
    return gemv_impl(W, ldw, dtype, x, y, M, K, tuning, stream, true);
}

tvl_status tvl_gemv(const void *W, int64_t ldw, int32_t dtype, const float *x, float *y,
                    int64_t M, int64_t K, hipStream_t stream)
{
    return tvl_gemv_ex(W, ldw, dtype, x, y, M, K, nullptr, stream);
}

tvl_status tvl_gemv_item(const tvl_item *item, const tvl_tuning *tuning, hipStream_t stream)
{
    g_err[0] = 0;
    if (!item) return fail(TVL_ERR_NULL, "tvl_gemv_item: item is NULL");
    tvl_status st = check_fused(*item, "tvl_gemv_item");
    if (st != TVL_OK) return st;
    if (!is_fused(*item) && !is_multi(*item))
        return tvl_gemv_ex(item->W, item->ldw, item->dtype, item->x, item->y, item->M, item->K,
                           tuning, stream);
    st = check_alias(item, 1);
    if (st != TVL_OK) return st;
    st = check_tuning(tuning, false);
    if (st != TVL_OK) return st;
    const bool f16 = item->dtype == TVL_F16;
    const int B = is_multi(*item) ? multi_B((int)item->nrhs) : 0;
    Shape shape;
    st = pick_shape(tuning,
                    B ? default_multi_shape(B, item->dtype == TVL_F32, item->dtype == TVL_F16)
                      : default_fused_shape(f16 ? 1.0 : 0.0, f16 ? 0.0 : 1.0),
                    &shape, false);
    if (st != TVL_OK) return st;
    if (B ? !tvl::multi_shape_supported(shape, B) : !tvl::fused_shape_supported(shape))
        return fail(TVL_ERR_ARG, "tvl_gemv_item: no %s kernel for (%d, %d, %d)",
                    B ? "several-vector" : "RMSNorm/SwiGLU", shape.R, shape.W, shape.U);
    if (tuning && tuning->grid)
        return fail(TVL_ERR_ARG, "tvl_gemv_item: grid applies to sweeps");
    int dev = 0;
    DevInfo info;
    st = current_device(&dev, &info);
    if (st != TVL_OK) return st;
    const DevItem d = dev_item(*item);
    const hipError_t e =
        B ? tvl::launch_item_multi(shape, B, d, stream) : tvl::launch_item(shape, d, stream);
    if (e != hipSuccess) return fail_hip(e, "item launch");
    return TVL_OK;
}

tvl_status tvl_sweep_plan_create(const tvl_item *items, int32_t n, const tvl_tuning *tuning,
                                 tvl_plan **plan)
{
    g_err[0] = 0;
    if (!plan) return fail(TVL_ERR_NULL, "tvl_sweep_plan_create: plan is NULL");
    *plan = nullptr;
    tvl_status st = check_items(items, n);
    if (st != TVL_OK) return st;
    st = check_tuning(tuning, false);
    if (st != TVL_OK) return st;
    return plan_build(items, n, tuning, plan);
}

tvl_status tvl_sweep_plan_run(const tvl_plan *plan, hipStream_t stream)
{
    g_err[0] = 0;
    if (!plan) return fail(TVL_ERR_NULL, "tvl_sweep_plan_run: plan is NULL");
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
    if (dev != plan->device)
        return fail(TVL_ERR_ARG, "tvl_sweep_plan_run: plan belongs to device %d, current is %d",
                    plan->device, dev);
    return plan_launch(plan, stream);
}

tvl_status tvl_sweep_plan_info(const tvl_plan *plan, int64_t *ntiles, int64_t *grid,
                               int32_t *rows_per_tile)
{
    if (!plan) return fail(TVL_ERR_NULL, "tvl_sweep_plan_info: plan is NULL");
    if (ntiles) *ntiles = plan->ntiles;
    if (grid) *grid = plan->grid;
    if (rows_per_tile) *rows_per_tile = plan->shape.R * plan->shape.W;
    return TVL_OK;
}

tvl_status tvl_sweep_plan_destroy(tvl_plan *plan)
{
    plan_free(plan);
    return TVL_OK;
}

tvl_status tvl_gemv_batch_sweep(const tvl_item *items, int32_t n, hipStream_t stream)
{
    g_err[0] = 0;
    tvl_status st = check_items(items, n);
    if (st != TVL_OK) return st;
    if (n == 0) return TVL_OK;
    int dev = 0;
    DevInfo info;
    st = current_device(&dev, &info);
    if (st != TVL_OK) return st;
    std::string key(reinterpret_cast<const char *>(&dev), sizeof dev);
    key.append(reinterpret_cast<const char *>(items), sizeof(tvl_item) * (size_t)n);
    // A cached plan is launched under the lock that found it: another
    // thread's eviction (cache full) or tvl_release_workspaces would
    // otherwise free it between the lookup and the launch.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    const hipError_t ce = hipStreamIsCapturing(stream, &cap);
    if (ce != hipSuccess) return fail_hip(ce, "hipStreamIsCapturing");
    const bool capturing = cap != hipStreamCaptureStatusNone;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_cache.find(key);
        if (it != g_cache.end()) {
            // a graph now holds the plan's tables: kept at eviction
            if (capturing) it->second->captured = true;
            return plan_launch(it->second, stream);
        }
    }
    if (capturing)
        return fail(TVL_ERR_ARG, "tvl_gemv_batch_sweep: stream %p is being captured and this item "
                                 "list has no plan yet (building one allocates and uploads); "
                                 "make the same call once before capturing",
                    (void *)stream);
    tvl_plan *fresh = nullptr; // built outside the lock (allocates, uploads)
    st = plan_build(items, n, nullptr, &fresh);
    if (st != TVL_OK) return st;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) { // another thread built the same list meanwhile
        plan_free(fresh);
        return plan_launch(it->second, stream);
    }
    if (g_cache.size() >= kCacheMax) { // plan_free waits for in-flight launches
        for (auto &kv : g_cache) {
            if (kv.second->captured)
                g_plans_retired.push_back(kv.second); // a graph may still launch it
            else
                plan_free(kv.second);
        }
        g_cache.clear();
    }
    g_cache.emplace(key, fresh);
    return plan_launch(fresh, stream);
}

tvl_status tvl_release_workspaces(void)
{
    g_err[0] = 0;
    std::lock_guard<std::mutex> lk(g_mu);
    int cur = -1;
    (void)hipGetDevice(&cur);
    for (auto &kv : g_ws) {
        (void)hipSetDevice(kv.first.first);
        (void)hipDeviceSynchronize();
        (void)hipFree(kv.second.partials);
        (void)hipFree(kv.second.counters);
    }
    g_ws.clear();
    for (auto &dw : g_ws_retired) {
        (void)hipSetDevice(dw.first);
        (void)hipDeviceSynchronize();
        (void)hipFree(dw.second.partials);
        (void)hipFree(dw.second.counters);
    }
    g_ws_retired.clear();
    for (auto &kv : g_cache)
        plan_free(kv.second);
    g_cache.clear();
    for (tvl_plan *p : g_plans_retired)
        plan_free(p);
    g_plans_retired.clear();
    if (cur >= 0) (void)hipSetDevice(cur);
    return TVL_OK;
}

tvl_status tvl_util_read_stream(const void *src, int64_t bytes, float *sink, int64_t sink_len,
                                int64_t *grid_out, hipStream_t stream)
{
    g_err[0] = 0;
    if (!src || !sink) return fail(TVL_ERR_NULL, "tvl_util_read_stream: NULL pointer");
    if (bytes < 16 || bytes % 16 || sink_len < 1 || sink_len > (1 << 20))
        return fail(TVL_ERR_SHAPE, "tvl_util_read_stream: bytes must be a positive multiple of "
                                   "16 and 1 <= sink_len <= 2^20");
    if (reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(sink) % 4)
        return fail(TVL_ERR_ALIGN, "tvl_util_read_stream: src 16-byte, sink 4-byte aligned");
    if (grid_out) *grid_out = sink_len;
    const hipError_t e = tvl::launch_read_stream(src, bytes, sink, (int)sink_len, stream);
    if (e != hipSuccess) return fail_hip(e, "read_stream launch");
    return TVL_OK;
}

tvl_status tvl_util_copy(void *dst, const void *src, int64_t bytes, hipStream_t stream)
{
    g_err[0] = 0;
    if (!src || !dst) return fail(TVL_ERR_NULL, "tvl_util_copy: NULL pointer");
    if (bytes < 16 || bytes % 16) return fail(TVL_ERR_SHAPE, "tvl_util_copy: bytes % 16 != 0");
    if (reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
        return fail(TVL_ERR_ALIGN, "tvl_util_copy: 16-byte alignment required");
    if (overlap(Range{(uintptr_t)src, (uintptr_t)src + (uintptr_t)bytes},
                Range{(uintptr_t)dst, (uintptr_t)dst + (uintptr_t)bytes}))
        return fail(TVL_ERR_ALIAS, "tvl_util_copy: overlap");
    const hipError_t e = tvl::launch_copy(dst, src, bytes, stream);
    if (e != hipSuccess) return fail_hip(e, "copy launch");
    return TVL_OK;
}

const char *tvl_status_str(int32_t status)
{
    switch (status) {
    case TVL_OK: return "TVL_OK";
    case TVL_ERR_NULL: return "TVL_ERR_NULL: a required pointer is NULL";
    case TVL_ERR_SHAPE: return "TVL_ERR_SHAPE: invalid M, K, ldw or count";
    case TVL_ERR_ALIGN: return "TVL_ERR_ALIGN: TVL alignment violated";
    case TVL_ERR_DTYPE: return "TVL_ERR_DTYPE: unknown weight dtype";
    case TVL_ERR_ALIAS: return "TVL_ERR_ALIAS: an output overlaps an input or output";
    case TVL_ERR_HIP: return "TVL_ERR_HIP: HIP runtime error";
    case TVL_ERR_NOMEM: return "TVL_ERR_NOMEM: allocation failed";
    case TVL_ERR_ARG: return "TVL_ERR_ARG: unsupported argument";
    default: return "unknown tvl_status";
    }
}

const char *tvl_last_error(void) { return g_err; }

}  // extern "C"
