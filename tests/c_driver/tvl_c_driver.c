/*
 * tvl_c_driver.c -- TEST INFRASTRUCTURE: the C ABI of include/tvl.h driven
 * from plain C99, with the HIP runtime and no Python or torch.  It links the
 * CPU oracle (oracle/liboracle.so) to check the results, which only tests may
 * do.
 *
 * Steps: allocate dense weights and vectors with hipMalloc, pack them into the
 * 128-byte row layout (tvl_pack_rows), run a three-item plan (fp32 ragged,
 * fp16 ragged, fp32 768 x 768) in one launch, run the same items through
 * tvl_gemv_batch_sweep and tvl_gemv, run two several-vector items (8 fp32 and
 * 16 fp16 beam vectors), and check every output against the oracle (y = W x,
 * Sec. 6.1; normalised error <= 1e-5 fp32, 2e-3 fp16, 1e-5 for the beams).
 * One bad call (a misaligned x) must return TVL_ERR_ALIGN with a message.
 *
 * Exit status: 0 all checks passed, 1 a check failed, 77 no GPU.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "tvl.h"

/* the oracle's entry points (oracle/oracle.c) */
void oracle_gemv_f32(const float *W, int64_t ldw, const float *x, int64_t M, int64_t K,
                     double *y, double *S);
void oracle_gemv_f16(const uint16_t *W, int64_t ldw, const float *x, int64_t M, int64_t K,
                     double *y, double *S);
int64_t oracle_check(const float *y, const double *ref, const double *S, int64_t M, double tol,
                     double *max_err, int64_t *argmax, double *mean_err);

#define HIP_OK(call)                                                                         \
    do {                                                                                     \
        hipError_t e_ = (call);                                                              \
        if (e_ != hipSuccess) {                                                              \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
            exit(1);                                                                         \
        }                                                                                    \
    } while (0)

#define TVL_OK_(call)                                                                        \
    do {                                                                                     \
        tvl_status s_ = (call);                                                              \
        if (s_ != TVL_OK) {                                                                  \
            fprintf(stderr, "%s:%d %s: %s (%s)\n", __FILE__, __LINE__, #call,                \
                    tvl_status_str(s_), tvl_last_error());                                   \
            exit(1);                                                                         \
        }                                                                                    \
    } while (0)

/* SplitMix64 (Steele, Lea & Flood 2014) for the test data */
static uint64_t mix(uint64_t *s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
static float uniform(uint64_t *s, float a, float b)
{
    return a + (b - a) * (float)((double)(mix(s) >> 11) * 0x1.0p-53);
}

/* binary16 bits of a float, round to nearest even in the normal range;
 * magnitudes below 2^-14 (about 0.1 % of these test weights) become +-0.
 * This only shapes the test data: the oracle reads the same bits as the GPU. */
static uint16_t f16_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    const uint32_t sign = (u >> 16) & 0x8000u;
    const int e = (int)((u >> 23) & 0xff) - 127 + 15;
    uint32_t m = u & 0x7fffffu;
    if (e <= 0) return (uint16_t)sign;
    uint32_t h = ((uint32_t)e << 10) | (m >> 13);
    const uint32_t rest = m & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h;
    return (uint16_t)(sign | h);
}

typedef struct {
    int64_t M, K, ldw;
    int32_t dtype;
    void *host;   /* dense M x K (float or uint16_t) */
    void *dense;  /* device copy of host */
    void *packed; /* device, TVL rows */
    float *hx, *dx, *dy;
} case_t;

static void make_case(case_t *c, int64_t M, int64_t K, int32_t dtype, uint64_t seed)
{
    uint64_t s = seed;
    const size_t es = dtype == TVL_F16 ? 2 : 4;
    c->M = M, c->K = K, c->dtype = dtype;
    c->ldw = tvl_row_stride(K, dtype);
    c->host = malloc((size_t)(M * K) * es);
    c->hx = malloc((size_t)K * 4);
    for (int64_t i = 0; i < M * K; ++i) {
        const float w = uniform(&s, -0.05f, 0.05f);
        if (dtype == TVL_F16)
            ((uint16_t *)c->host)[i] = f16_bits(w);
        else
            ((float *)c->host)[i] = w;
    }
    for (int64_t j = 0; j < K; ++j) c->hx[j] = uniform(&s, -2.f, 2.f);
    HIP_OK(hipMalloc(&c->dense, (size_t)(M * K) * es));
    HIP_OK(hipMalloc(&c->packed, (size_t)(M * c->ldw) * es));
    HIP_OK(hipMalloc((void **)&c->dx, (size_t)K * 4));
    HIP_OK(hipMalloc((void **)&c->dy, (size_t)M * 4));
    HIP_OK(hipMemcpy(c->dense, c->host, (size_t)(M * K) * es, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(c->dx, c->hx, (size_t)K * 4, hipMemcpyHostToDevice));
}

static int check_case(const case_t *c, const char *what)
{
    float *y = malloc((size_t)c->M * 4);
    double *ref = malloc((size_t)c->M * 8), *S = malloc((size_t)c->M * 8);
    HIP_OK(hipMemcpy(y, c->dy, (size_t)c->M * 4, hipMemcpyDeviceToHost));
    if (c->dtype == TVL_F16)
        oracle_gemv_f16(c->host, c->K, c->hx, c->M, c->K, ref, S);
    else
        oracle_gemv_f32(c->host, c->K, c->hx, c->M, c->K, ref, S);
    double worst = 0.0, mean = 0.0;
    int64_t at = -1;
    const double tol = c->dtype == TVL_F16 ? 2e-3 : 1e-5;
    const int64_t bad = oracle_check(y, ref, S, c->M, tol, &worst, &at, &mean);
    printf("%s: %lld x %lld %s, max normalised error %.3e (row %lld)%s\n", what,
           (long long)c->M, (long long)c->K, c->dtype == TVL_F16 ? "fp16" : "fp32", worst,
           (long long)at, bad ? "  FAIL" : "");
    free(y), free(ref), free(S);
    return bad != 0;
}

/* A several-vector item (beam search with nrhs hypotheses): nrhs x vectors
 * at a stride of ldx floats (the padding holds NaN, never used), nrhs
 * outputs at a stride of M; every vector against the oracle's GEMV of it,
 * at the fp32 bar (1e-5 of the norm) for both weight types. */
static int run_multi(int64_t M, int64_t K, int32_t dtype, int nrhs, uint64_t seed, int single,
                     hipStream_t st)
{
    case_t c;
    make_case(&c, M, K, dtype, seed);
    TVL_OK_(tvl_pack_rows(c.packed, c.ldw, c.dense, c.M, c.K, c.dtype, st));
    const int64_t ldx = (K + 3) / 4 * 4;
    uint64_t s = seed * 7919u;
    float *hx = malloc((size_t)(nrhs * ldx) * 4);
    for (int64_t i = 0; i < nrhs * ldx; ++i) hx[i] = (i % ldx) < K ? uniform(&s, -2.f, 2.f) : NAN;
    float *dx = NULL, *dy = NULL;
    HIP_OK(hipMalloc((void **)&dx, (size_t)(nrhs * ldx) * 4));
    HIP_OK(hipMalloc((void **)&dy, (size_t)(nrhs * M) * 4));
    HIP_OK(hipMemcpy(dx, hx, (size_t)(nrhs * ldx) * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemsetAsync(dy, 0xff, (size_t)(nrhs * M) * 4, st));
    tvl_item it;
    memset(&it, 0, sizeof it);
    it.W = c.packed, it.ldw = c.ldw, it.x = dx, it.y = dy, it.M = M, it.K = K, it.dtype = dtype;
    it.nrhs = nrhs, it.ldx = ldx, it.ldy = M;
    if (single)
        TVL_OK_(tvl_gemv_item(&it, NULL, st));
    else
        TVL_OK_(tvl_gemv_batch_sweep(&it, 1, st));
    HIP_OK(hipStreamSynchronize(st));
    float *y = malloc((size_t)(nrhs * M) * 4);
    double *ref = malloc((size_t)M * 8), *S = malloc((size_t)M * 8);
    HIP_OK(hipMemcpy(y, dy, (size_t)(nrhs * M) * 4, hipMemcpyDeviceToHost));
    double worst = 0.0;
    int64_t bad = 0;
    for (int b = 0; b < nrhs; ++b) {
        if (dtype == TVL_F16)
            oracle_gemv_f16(c.host, K, hx + b * ldx, M, K, ref, S);
        else
            oracle_gemv_f32(c.host, K, hx + b * ldx, M, K, ref, S);
        double w = 0.0, mean = 0.0;
        int64_t at = -1;
        bad += oracle_check(y + b * M, ref, S, M, 1e-5, &w, &at, &mean);
        if (w > worst) worst = w;
    }
    printf("%s: %lld x %lld %s, %d vectors, max normalised error %.3e%s\n",
           single ? "multi item" : "multi batch", (long long)M, (long long)K,
           dtype == TVL_F16 ? "fp16" : "fp32", nrhs, worst, bad ? "  FAIL" : "");
    free(hx), free(y), free(ref), free(S);
    HIP_OK(hipFree(dx));
    HIP_OK(hipFree(dy));
    HIP_OK(hipFree(c.dense));
    HIP_OK(hipFree(c.packed));
    HIP_OK(hipFree(c.dx));
    HIP_OK(hipFree(c.dy));
    free(c.host);
    free(c.hx);
    return bad != 0;
}

int main(void)
{
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        printf("no GPU\n");
        return 77;
    }
    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));
    case_t cs[3];
    make_case(&cs[0], 300, 1000, TVL_F32, 1);
    make_case(&cs[1], 77, 1001, TVL_F16, 2);
    make_case(&cs[2], 768, 768, TVL_F32, 3);
    tvl_item items[3];
    memset(items, 0, sizeof items);
    for (int k = 0; k < 3; ++k) {
        case_t *c = &cs[k];
        TVL_OK_(tvl_pack_rows(c->packed, c->ldw, c->dense, c->M, c->K, c->dtype, st));
        items[k].W = c->packed, items[k].ldw = c->ldw, items[k].x = c->dx, items[k].y = c->dy;
        items[k].M = c->M, items[k].K = c->K, items[k].dtype = c->dtype;
    }
    int fails = 0;

    /* a plan: exactly one launch for the three GEMVs */
    tvl_plan *plan = NULL;
    TVL_OK_(tvl_sweep_plan_create(items, 3, NULL, &plan));
    int64_t ntiles = 0, grid = 0;
    int32_t rows = 0;
    TVL_OK_(tvl_sweep_plan_info(plan, &ntiles, &grid, &rows));
    for (int k = 0; k < 3; ++k) HIP_OK(hipMemsetAsync(cs[k].dy, 0xff, (size_t)cs[k].M * 4, st));
    TVL_OK_(tvl_sweep_plan_run(plan, st));
    HIP_OK(hipStreamSynchronize(st));
    printf("plan: %lld tiles of %d rows, grid %lld\n", (long long)ntiles, (int)rows,
           (long long)grid);
    for (int k = 0; k < 3; ++k) fails += check_case(&cs[k], "plan");
    TVL_OK_(tvl_sweep_plan_destroy(plan));
    TVL_OK_(tvl_sweep_plan_destroy(NULL)); /* a no-op */

    /* the same items through the batch entry point (plans cached by list) */
    for (int rep = 0; rep < 2; ++rep) {
        for (int k = 0; k < 3; ++k)
            HIP_OK(hipMemsetAsync(cs[k].dy, 0xff, (size_t)cs[k].M * 4, st));
        TVL_OK_(tvl_gemv_batch_sweep(items, 3, st));
        HIP_OK(hipStreamSynchronize(st));
        for (int k = 0; k < 3; ++k) fails += check_case(&cs[k], "batch");
    }

    /* one GEMV at a time */
    for (int k = 0; k < 3; ++k) {
        case_t *c = &cs[k];
        HIP_OK(hipMemsetAsync(c->dy, 0xff, (size_t)c->M * 4, st));
        TVL_OK_(tvl_gemv(c->packed, c->ldw, c->dtype, c->dx, c->dy, c->M, c->K, st));
        HIP_OK(hipStreamSynchronize(st));
        fails += check_case(c, "gemv");
    }

    /* beam search: 8 fp32 vectors through the batch entry point, 16 fp16
     * vectors through the single-item one (the library's default kernels) */
    fails += run_multi(300, 1000, TVL_F32, 8, 4, 0, st);
    fails += run_multi(130, 2050, TVL_F16, 16, 5, 1, st);

    /* an error is returned, not raised, and nothing is enqueued */
    const tvl_status bad = tvl_gemv(cs[0].packed, cs[0].ldw, TVL_F32, cs[0].dx + 1, cs[0].dy,
                                    cs[0].M, cs[0].K, st);
    if (bad != TVL_ERR_ALIGN || tvl_last_error()[0] == 0) {
        printf("misaligned x: got %s, want TVL_ERR_ALIGN  FAIL\n", tvl_status_str(bad));
        ++fails;
    } else {
        printf("misaligned x: %s (%s)\n", tvl_status_str(bad), tvl_last_error());
    }

    TVL_OK_(tvl_release_workspaces());
    for (int k = 0; k < 3; ++k) {
        HIP_OK(hipFree(cs[k].dense));
        HIP_OK(hipFree(cs[k].packed));
        HIP_OK(hipFree(cs[k].dx));
        HIP_OK(hipFree(cs[k].dy));
        free(cs[k].host);
        free(cs[k].hx);
    }
    HIP_OK(hipStreamDestroy(st));
    printf("%s\n", fails ? "FAILED" : "all checks passed");
    return fails ? 1 : 0;
}
