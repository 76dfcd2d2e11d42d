/*
 * A C99 user of libbq through include/bq.h alone: no C++, no PyTorch.
 *
 *   bq_c_example        host-only calls and argument errors (no GPU needed)
 *   bq_c_example gpu    also, on the current HIP device: a block-wise quantize
 *                       round trip and fused 8-bit Adam steps through the
 *                       allocation-free call and through a step plan
 *
 * The GPU results are checked against properties that hold at any size:
 * - each block's absmax is the largest magnitude in the block (Section 3.1);
 * - each dequantized value lies within half the widest gap of the map, scaled
 *   by its block's absmax, of the input (Eq. 4: the nearest code);
 * - Adam's first step moves every param by lr * g / (|g| + eps) from the
 *   unquantized states (Eq. 2 with bias correction), i.e. by lr against the
 *   sign of its gradient when |g| >> eps;
 * - a step plan and the call give identical codes and absmax.
 * Exit status 0 on success; a message and status 1 otherwise.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "bq.h"

static int failures = 0;

#define CHECK(cond, ...)                        \
    do {                                        \
        if (!(cond)) {                          \
            fprintf(stderr, "FAIL: " __VA_ARGS__); \
            fprintf(stderr, "\n");              \
            ++failures;                         \
        }                                       \
    } while (0)

#define HIP(call)                                                           \
    do {                                                                    \
        hipError_t e_ = (call);                                             \
        if (e_ != hipSuccess) {                                             \
            fprintf(stderr, "HIP error %d at %s:%d\n", (int)e_, __FILE__, __LINE__); \
            exit(1);                                                        \
        }                                                                   \
    } while (0)

static void host_calls(void)
{
    float qs[256], qu[256], lin[256];
    CHECK(bq_make_dynamic_codebook(BQ_SIGNED, qs) == BQ_OK, "signed map");
    CHECK(bq_make_dynamic_codebook(BQ_UNSIGNED, qu) == BQ_OK, "unsigned map");
    CHECK(bq_make_codebook(BQ_LINEAR_SIGNED, lin) == BQ_OK, "linear map");
    CHECK(qs[0] == -1.0f && qs[127] == 0.0f && qs[255] == 1.0f, "signed map ends");
    CHECK(qu[0] == 0.0f && qu[255] == 1.0f, "unsigned map ends");
    for (int i = 1; i < 256; ++i)
        CHECK(qs[i - 1] < qs[i] && qu[i - 1] < qu[i], "maps increase at %d", i);
    CHECK(bq_make_dynamic_codebook(BQ_SIGNED, NULL) == BQ_ERR_NULL, "NULL out");
    CHECK(bq_make_codebook((bq_codebook_kind)99, lin) == BQ_ERR_ENUM, "bad kind");
    /* argument errors are returned before any HIP call */
    CHECK(bq_quantize_blockwise(qs, qs, 16, 100, NULL, NULL, 0) == BQ_ERR_BLOCKSIZE, "blocksize");
    CHECK(bq_quantize_blockwise(qs, qs, -1, 2048, NULL, NULL, 0) == BQ_ERR_SIZE, "size");
    CHECK(bq_quantize_blockwise(qs, qs, 0, 2048, NULL, NULL, 0) == BQ_OK, "empty is a no-op");
    CHECK(bq_optimizer8bit_step(BQ_ADAM, 2048, (bq_dtype)7, NULL, 1, NULL, NULL, NULL, 0) ==
              BQ_ERR_DTYPE,
          "grad dtype");
    CHECK(bq_step_plan_run_prepared(NULL, NULL, NULL, 0) == BQ_ERR_NULL, "NULL plan");
    CHECK(strcmp(bq_status_string(BQ_ERR_ALIGN), "ok") != 0, "status string");
    CHECK(bq_quantile_workspace_bytes(0) == 0, "workspace of nothing");
}

/* deterministic inputs: a sine with a few large outliers */
static float value_at(int64_t i)
{
    float v = 0.01f * sinf(0.37f * (float)i) * (1.0f + (float)(i % 7));
    if (i % 997 == 0)
        v *= 50.0f;
    return v;
}

static void gpu_quantize(const float *qs)
{
    const int64_t n = 3 * 2048 + 77;
    const int32_t B = 2048;
    const int64_t nb = (n + B - 1) / B;
    float *x = malloc(n * sizeof(float)), *out = malloc(n * sizeof(float));
    float *absmax = malloc(nb * sizeof(float));
    for (int64_t i = 0; i < n; ++i)
        x[i] = value_at(i);
    float *x_d, *out_d, *absmax_d, *q_d;
    uint8_t *codes_d;
    HIP(hipMalloc((void **)&x_d, n * sizeof(float)));
    HIP(hipMalloc((void **)&out_d, n * sizeof(float)));
    HIP(hipMalloc((void **)&codes_d, n));
    HIP(hipMalloc((void **)&absmax_d, nb * sizeof(float)));
    HIP(hipMalloc((void **)&q_d, 256 * sizeof(float)));
    HIP(hipMemcpy(x_d, x, n * sizeof(float), hipMemcpyHostToDevice));
    HIP(hipMemcpy(q_d, qs, 256 * sizeof(float), hipMemcpyHostToDevice));
    CHECK(bq_quantize_blockwise(q_d, x_d, n, B, codes_d, absmax_d, 0) == BQ_OK, "quantize");
    CHECK(bq_dequantize_blockwise(q_d, codes_d, absmax_d, n, B, out_d, 0) == BQ_OK, "dequantize");
    HIP(hipDeviceSynchronize());
    HIP(hipMemcpy(out, out_d, n * sizeof(float), hipMemcpyDeviceToHost));
    HIP(hipMemcpy(absmax, absmax_d, nb * sizeof(float), hipMemcpyDeviceToHost));
    float gap = 0.0f;
    for (int i = 1; i < 256; ++i)
        gap = fmaxf(gap, qs[i] - qs[i - 1]);
    for (int64_t b = 0; b < nb; ++b) {
        float m = 0.0f;
        for (int64_t i = b * B; i < n && i < (b + 1) * B; ++i)
            m = fmaxf(m, fabsf(x[i]));
        CHECK(absmax[b] == m, "absmax of block %lld", (long long)b);
    }
    for (int64_t i = 0; i < n; ++i) {
        const float bound = absmax[i / B] * gap * 0.5f * 1.0001f;
        CHECK(fabsf(out[i] - x[i]) <= bound, "round trip at %lld: %g vs %g", (long long)i,
              out[i], x[i]);
    }
    HIP(hipFree(x_d));
    HIP(hipFree(out_d));
    HIP(hipFree(codes_d));
    HIP(hipFree(absmax_d));
    HIP(hipFree(q_d));
    free(x);
    free(out);
    free(absmax);
}

struct dev_state {
    float *w, *g, *a1, *a2;
    uint8_t *s1, *s2;
};

static void make_state(struct dev_state *d, const float *w, const float *g, int64_t n, int64_t nb)
{
    HIP(hipMalloc((void **)&d->w, n * sizeof(float)));
    HIP(hipMalloc((void **)&d->g, n * sizeof(float)));
    HIP(hipMalloc((void **)&d->s1, n));
    HIP(hipMalloc((void **)&d->s2, n));
    HIP(hipMalloc((void **)&d->a1, nb * sizeof(float)));
    HIP(hipMalloc((void **)&d->a2, nb * sizeof(float)));
    HIP(hipMemcpy(d->w, w, n * sizeof(float), hipMemcpyHostToDevice));
    HIP(hipMemcpy(d->g, g, n * sizeof(float), hipMemcpyHostToDevice));
    HIP(hipMemset(d->s1, 127, n)); /* the signed map's zero code */
    HIP(hipMemset(d->s2, 0, n));   /* the unsigned map's zero code */
    HIP(hipMemset(d->a1, 0, nb * sizeof(float)));
    HIP(hipMemset(d->a2, 0, nb * sizeof(float)));
}

static bq_tensor as_tensor(const struct dev_state *d, int64_t n)
{
    bq_tensor t;
    memset(&t, 0, sizeof(t));
    t.param = d->w;
    t.grad = d->g;
    t.state1 = d->s1;
    t.state2 = d->s2;
    t.absmax1 = d->a1;
    t.absmax2 = d->a2;
    t.numel = n;
    return t;
}

static int same_bytes(const void *a_d, const void *b_d, size_t bytes)
{
    unsigned char *a = malloc(bytes), *b = malloc(bytes);
    HIP(hipMemcpy(a, a_d, bytes, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(b, b_d, bytes, hipMemcpyDeviceToHost));
    const int same = memcmp(a, b, bytes) == 0;
    free(a);
    free(b);
    return same;
}

static void gpu_adam(const float *qs, const float *qu)
{
    const int64_t n = 2 * 4096 + 333;
    const int32_t B = 2048;
    const int64_t nb = (n + B - 1) / B;
    float *w = malloc(n * sizeof(float)), *g = malloc(n * sizeof(float));
    float *w1 = malloc(n * sizeof(float));
    for (int64_t i = 0; i < n; ++i) {
        w[i] = 0.05f * cosf(0.11f * (float)i);
        g[i] = value_at(i) + (value_at(i) >= 0.0f ? 1e-3f : -1e-3f); /* |g| >= 1e-3 */
    }
    float *qs_d, *qu_d;
    HIP(hipMalloc((void **)&qs_d, 256 * sizeof(float)));
    HIP(hipMalloc((void **)&qu_d, 256 * sizeof(float)));
    HIP(hipMemcpy(qs_d, qs, 256 * sizeof(float), hipMemcpyHostToDevice));
    HIP(hipMemcpy(qu_d, qu, 256 * sizeof(float), hipMemcpyHostToDevice));
    struct dev_state call, plan_state;
    make_state(&call, w, g, n, nb);
    make_state(&plan_state, w, g, n, nb);
    bq_hparams hp;
    memset(&hp, 0, sizeof(hp));
    hp.lr = 1e-3f;
    hp.beta1 = 0.9f;
    hp.beta2 = 0.995f;
    hp.eps = 1e-8f;
    hp.weight_decay = 0.0f;
    const bq_tensor tc = as_tensor(&call, n), tp = as_tensor(&plan_state, n);
    bq_step_plan plan = NULL;
    CHECK(bq_step_plan_create(BQ_ADAM, B, BQ_F32, &tp, 1, &plan) == BQ_OK, "plan create");
    for (int64_t t = 1; t <= 2; ++t) {
        hp.step = t;
        CHECK(bq_optimizer8bit_step(BQ_ADAM, B, BQ_F32, &tc, 1, &hp, qs_d, qu_d, 0) == BQ_OK,
              "step call t=%lld", (long long)t);
        CHECK(bq_step_plan_run(plan, &hp, qs_d, qu_d, 0) == BQ_OK, "plan run t=%lld",
              (long long)t);
        HIP(hipDeviceSynchronize());
        if (t == 1) {
            HIP(hipMemcpy(w1, call.w, n * sizeof(float), hipMemcpyDeviceToHost));
            for (int64_t i = 0; i < n; ++i) {
                const double step = (double)w[i] - (double)w1[i];
                const double expect = 1e-3 * (double)g[i] / (fabs((double)g[i]) + 1e-8);
                CHECK(fabs(step - expect) <= 1e-6 * 1e-3 + 1e-7 * fabs((double)w[i]),
                      "Adam's first step at %lld: %g, expected %g", (long long)i, step, expect);
            }
        }
        CHECK(same_bytes(call.s1, plan_state.s1, n) && same_bytes(call.s2, plan_state.s2, n),
              "plan and call codes differ at t=%lld", (long long)t);
        CHECK(same_bytes(call.a1, plan_state.a1, nb * sizeof(float)) &&
                  same_bytes(call.a2, plan_state.a2, nb * sizeof(float)),
              "plan and call absmax differ at t=%lld", (long long)t);
    }
    CHECK(bq_step_plan_destroy(plan) == BQ_OK, "plan destroy");
    struct dev_state *all[2] = {&call, &plan_state};
    for (int k = 0; k < 2; ++k) {
        HIP(hipFree(all[k]->w));
        HIP(hipFree(all[k]->g));
        HIP(hipFree(all[k]->s1));
        HIP(hipFree(all[k]->s2));
        HIP(hipFree(all[k]->a1));
        HIP(hipFree(all[k]->a2));
    }
    HIP(hipFree(qs_d));
    HIP(hipFree(qu_d));
    free(w);
    free(g);
    free(w1);
}

int main(int argc, char **argv)
{
    host_calls();
    if (argc > 1 && strcmp(argv[1], "gpu") == 0) {
        float qs[256], qu[256];
        bq_make_dynamic_codebook(BQ_SIGNED, qs);
        bq_make_dynamic_codebook(BQ_UNSIGNED, qu);
        printf("bq_c_example: quantize round trip\n");
        fflush(stdout);
        gpu_quantize(qs);
        printf("bq_c_example: 8-bit Adam, call and plan\n");
        fflush(stdout);
        gpu_adam(qs, qu);
    }
    if (failures) {
        fprintf(stderr, "bq_c_example: %d checks failed\n", failures);
        return 1;
    }
    printf("bq_c_example ok\n");
    return 0;
}
