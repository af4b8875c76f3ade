/* Drives the C ABI with plain HIP allocations (no Python, no torch): a plan,
 * the warm-up, three compression steps, then the error state made explicit,
 * each result compared with the CPU oracle on the same inputs.  An optional
 * argument sets the plan's chunk-owner table mode (onebit_plan_set_server_tables:
 * 0 off, 1 auto, 2 on).  Prints "ok" and exits 0 on success. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "onebit.h"

/* oracle (test infrastructure) */
int64_t orc_layout(const int64_t *numel, int32_t K, int32_t n, int64_t *tensor_off,
                   int64_t *seg_begin, int64_t *seg_end);
void orc_warmup_range(int64_t b, int64_t e, float *x, float *m, float *v, const float *g,
                      int64_t g_ld, int32_t n, float lr, float beta1, float beta2, float eps,
                      int32_t bias_correction, int64_t t);
void orc_step(const int64_t *numel, int32_t K, int32_t n, const int64_t *seg_begin,
              const int64_t *seg_end, float *x, float *m, const float *v_frozen, const float *g,
              int64_t g_ld, float *delta, int64_t delta_ld, float *delta_bar, uint64_t *wbits,
              int64_t W, float *wscales, uint64_t *sbits, float *sscales, float lr, float beta1,
              float eps, float *z_scratch);

#define CHECK_HIP(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { \
    fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); return 2; } } while (0)
#define CHECK_OB(x) do { int s_ = (x); if (s_ != ONEBIT_OK) { \
    fprintf(stderr, "%s: %s (%s) at line %d\n", #x, onebit_status_str(s_), onebit_last_error(), __LINE__); \
    return 3; } } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform01(void)
{   /* splitmix64 */
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return ((z >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}
static float normal(float sd)
{
    double u1 = uniform01(), u2 = uniform01();
    return (float)(sd * sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2));
}

static int compare(const char *name, const float *a, const float *b, int64_t len)
{
    int64_t bad = 0;
    for (int64_t i = 0; i < len; ++i) {
        double d = fabs((double)a[i] - (double)b[i]);
        if (d > 1e-6 + 1e-5 * fabs((double)b[i])) ++bad;
    }
    if (bad) fprintf(stderr, "%s: %lld of %lld outside tolerance\n", name, (long long)bad, (long long)len);
    return bad != 0;
}

int main(int argc, char **argv)
{
    const int64_t numel[3] = {70001, 4096, 33};
    const int32_t K = 3, n = 4;
    const float lr = 1e-4f, b1 = 0.9f, b2 = 0.999f, eps = 1e-8f;
    int64_t toff[3], sb[12], se[12];
    const int64_t D = orc_layout(numel, K, n, toff, sb, se), W = D / 64, S = K * n;

    onebit_plan plan;
    CHECK_OB(onebit_plan_create(numel, K, n, &plan));
    if (argc > 1) CHECK_OB(onebit_plan_set_server_tables(plan, atoi(argv[1])));
    onebit_plan_sizes info;
    CHECK_OB(onebit_plan_get_info(plan, &info));
    if (info.padded_len != D || info.num_segments != S) { fprintf(stderr, "layout differs\n"); return 4; }

    size_t fD = (size_t)D * sizeof(float);
    float *hx = calloc(D, 4), *hm = calloc(D, 4), *hv = calloc(D, 4), *hg = calloc((size_t)n * D, 4);
    float *hdelta = calloc((size_t)n * D, 4), *hdbar = calloc(D, 4), *hz = calloc(D, 4);
    uint64_t *hwb = calloc((size_t)n * W, 8), *hsb = calloc(W, 8);
    float *hws = calloc((size_t)n * S, 4), *hss = calloc(S, 4), *back = calloc((size_t)n * D, 4);
    for (int k = 0; k < K; ++k)
        for (int64_t e = 0; e < numel[k]; ++e) hx[toff[k] + e] = normal(0.02f);

    float *x, *m, *v, *g, *werr, *serr, *wsc, *ssc, *dout;
    uint64_t *wb, *sbits;
    void *ws;
    CHECK_HIP(hipMalloc((void **)&x, fD)); CHECK_HIP(hipMalloc((void **)&m, fD));
    CHECK_HIP(hipMalloc((void **)&v, fD)); CHECK_HIP(hipMalloc((void **)&g, n * fD));
    CHECK_HIP(hipMalloc((void **)&werr, n * fD)); CHECK_HIP(hipMalloc((void **)&serr, fD));
    CHECK_HIP(hipMalloc((void **)&wsc, (size_t)n * S * 4)); CHECK_HIP(hipMalloc((void **)&ssc, S * 4));
    CHECK_HIP(hipMalloc((void **)&wb, (size_t)n * W * 8)); CHECK_HIP(hipMalloc((void **)&sbits, W * 8));
    CHECK_HIP(hipMalloc((void **)&dout, n * fD)); CHECK_HIP(hipMalloc(&ws, info.workspace_bytes));
    CHECK_HIP(hipMemcpy(x, hx, fD, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemset(m, 0, fD)); CHECK_HIP(hipMemset(v, 0, fD));
    CHECK_HIP(hipMemset(werr, 0, n * fD)); CHECK_HIP(hipMemset(serr, 0, fD));
    CHECK_HIP(hipMemset(wsc, 0, (size_t)n * S * 4)); CHECK_HIP(hipMemset(ssc, 0, S * 4));

    for (int t = 1; t <= 6; ++t) {
        for (int64_t i = 0; i < (int64_t)n * D; ++i) hg[i] = 0.0f;
        for (int r = 0; r < n; ++r)
            for (int k = 0; k < K; ++k)
                for (int64_t e = 0; e < numel[k]; ++e) hg[(int64_t)r * D + toff[k] + e] = normal(1e-3f);
        CHECK_HIP(hipMemcpy(g, hg, n * fD, hipMemcpyHostToDevice));
        if (t <= 3) {
            for (int k = 0; k < K; ++k)
                orc_warmup_range(toff[k], toff[k] + numel[k], hx, hm, hv, hg, D, n, lr, b1, b2, eps, 0, t);
            CHECK_OB(onebit_warmup_adam_step(plan, x, m, v, g, ONEBIT_GRAD_F32, D, n, lr, b1, b2,
                                             eps, 0, t, 0));
        } else {
            orc_step(numel, K, n, sb, se, hx, hm, hv, hg, D, hdelta, D, hdbar, hwb, W, hws, hsb,
                     hss, lr, b1, eps, hz);
            CHECK_OB(onebit_step(plan, x, t == 4 ? m : NULL, v, g, ONEBIT_GRAD_F32, D, werr, D,
                                 serr, wb, wsc, sbits, ssc, lr, b1, eps, ws, 0));
        }
    }
    CHECK_OB(onebit_error_materialize(plan, werr, D, wsc, S, n, dout, D, 0));
    CHECK_HIP(hipDeviceSynchronize());

    int fails = 0;
    CHECK_HIP(hipMemcpy(back, x, fD, hipMemcpyDeviceToHost));
    fails += compare("x", back, hx, D);
    CHECK_HIP(hipMemcpy(back, dout, n * fD, hipMemcpyDeviceToHost));
    fails += compare("worker delta", back, hdelta, (int64_t)n * D);
    CHECK_OB(onebit_decode(plan, sbits, ssc, dout, 0));
    CHECK_HIP(hipDeviceSynchronize());
    CHECK_HIP(hipMemcpy(back, dout, fD, hipMemcpyDeviceToHost));
    /* padding of the decoded buffer was not written: compare real elements only */
    for (int k = 0; k < K; ++k)
        fails += compare("momentum", back + toff[k], hm + toff[k], numel[k]);
    uint64_t *bb = (uint64_t *)back;
    CHECK_HIP(hipMemcpy(bb, sbits, W * 8, hipMemcpyDeviceToHost));
    if (memcmp(bb, hsb, W * 8) != 0) { fprintf(stderr, "server bits differ\n"); ++fails; }
    /* an error path: a misaligned pointer is rejected without launching */
    if (onebit_decode(plan, sbits, ssc, (float *)((char *)dout + 4), 0) != ONEBIT_EALIGN) {
        fprintf(stderr, "misaligned out accepted\n"); ++fails;
    }
    CHECK_OB(onebit_plan_destroy(plan));
    if (fails) return 1;
    printf("ok\n");
    return 0;
}
