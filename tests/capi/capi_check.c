/*
 * A plain C client of libsbw: include/sbw.h compiles as C (C11), and the library
 * links and runs with no Python or torch in the process.  Test infrastructure: it
 * links the CPU oracle (oracle/sbw_oracle.c) to check the results.
 *
 *   capi_check cpu   version string, status texts, and the argument checks that
 *                    return before any HIP call (no GPU needed).
 *   capi_check gpu   watermark (context and self-salt, window of 4, fp32), greedy
 *                    decoding (with a workspace and without: sbw_watermark_argmax_noalloc),
 *                    Gumbel-max sampling and detection on HIP device
 *                    buffers, each compared bit for bit with the oracle (z within
 *                    1e-6 relative).
 *
 * Inputs come from a xorshift64* generator seeded per case.  Prints one line per
 * check and exits non-zero on the first mismatch.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "sbw.h"

/* The oracle's C entry points used here (oracle/sbw_oracle.c). */
void oracle_watermark_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                            const int32_t *context, int64_t width, uint64_t key, double gamma,
                            float delta, int seeding);
void oracle_watermark_argmax_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, int32_t *tokens,
                                   float *values);
void oracle_watermark_sample_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, const uint64_t *seeds,
                                   float inv_temperature, int32_t *tokens, float *scores);
void oracle_detect_w(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                     int64_t width, uint64_t key, double gamma, int seeding,
                     int32_t *green_counts, double *z);
void oracle_green_mask_w(uint32_t *bits, int64_t B, int64_t V, const int32_t *context,
                         int64_t width, uint64_t key, double gamma, int seeding);
void oracle_watermark_candidates_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                                       const int32_t *cand, int64_t k, const int32_t *context,
                                       int64_t width, uint64_t key, double gamma, float delta,
                                       int seeding);
void oracle_detect_ex(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                      const int32_t *lengths, int64_t width, uint64_t key, double gamma,
                      int seeding, int ignore_repeated, int32_t *green_counts, int32_t *scored,
                      double *z);

static uint64_t rng_state;
static uint64_t next_u64(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1DULL;
}
static float next_logit(void) { return (float)((double)(next_u64() >> 11) * 0x1p-53 * 8.0 - 4.0); }

#define CHECK(cond, ...)                                                   \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "capi_check: FAILED: " __VA_ARGS__);           \
            fprintf(stderr, "\n");                                         \
            exit(1);                                                       \
        }                                                                  \
    } while (0)
#define HIP(call) CHECK((call) == hipSuccess, "%s", #call)
#define SBW(call) do { sbw_status_t s_ = (call); CHECK(s_ == SBW_OK, "%s -> %s", #call, sbw_strerror(s_)); } while (0)

static int cpu_checks(void)
{
    const char *v = sbw_version();
    CHECK(v != NULL && strlen(v) >= 5, "version");
    CHECK(strlen(sbw_strerror(SBW_ERR_GAMMA)) > 0 && strlen(sbw_strerror((sbw_status_t)99)) > 0, "strerror");
    float dummy = 0.0f;
    int32_t prev = 0;
    /* each of these fails its argument check before any HIP call */
    CHECK(sbw_watermark(NULL, SBW_F32, 1, 1, 1, &prev, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_INVALID_ARG, "null logits");
    CHECK(sbw_watermark(&dummy, SBW_F32, 1, 2, 1, &prev, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_INVALID_ARG, "row_stride < V");
    CHECK(sbw_watermark(&dummy, SBW_F32, 1, 1, 1, &prev, 1, 1.5, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_GAMMA, "gamma > 1");
    CHECK(sbw_watermark(&dummy, SBW_F32, 1, 1, 1, &prev, 1, 0.25, INFINITY, SBW_SEED_CONTEXT, NULL) == SBW_ERR_DELTA, "delta inf");
    CHECK(sbw_watermark(&dummy, (sbw_dtype_t)7, 1, 1, 1, &prev, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_UNSUPPORTED, "dtype");
    CHECK(sbw_watermark(&dummy, SBW_F32, 0, 1, 1, &prev, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_OK, "B = 0 is a no-op");
    CHECK(sbw_watermark_shard(&dummy, SBW_F32, 1, 1, 1, &prev, 1, -1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_INVALID_ARG, "negative v_offset");
    CHECK(sbw_watermark_shard(&dummy, SBW_F32, 1, 2, 2, &prev, 1, (int64_t)1 << 32, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL) == SBW_ERR_UNSUPPORTED, "ids past 2^32");
    CHECK(sbw_watermark_argmax_workspace(256, 152064) == 256 * 75, "workspace size");
    CHECK(sbw_watermark_argmax_workspace(0, 5) == 0, "workspace of nothing");
    /* the other entry points' host checks (unknown enum values included) */
    int32_t tok = 0, cnt = 0, cand = 0;
    uint32_t bits = 0;
    uint64_t ws = 0, seed = 1;
    double z = 0.0;
    CHECK(sbw_watermark_window(&dummy, SBW_BF16, 1, 1, 1, &prev, 9, 1, 0.25, 2.0f, SBW_SEED_SELF_SALT, NULL) == SBW_ERR_UNSUPPORTED, "width 9");
    CHECK(sbw_watermark_window(&dummy, SBW_F32, 1, 1, 1, &prev, 0, 1, 0.25, 2.0f, SBW_SEED_SELF_SALT, NULL) == SBW_ERR_INVALID_ARG, "width 0");
    CHECK(sbw_green_mask(&bits, 1, 1, &prev, 1, 0.25, (sbw_seeding_t)5, NULL) == SBW_ERR_UNSUPPORTED, "seeding 5");
    CHECK(sbw_green_mask_window(&bits, -1, 1, &prev, 1, 1, 0.25, SBW_SEED_CONTEXT, NULL) == SBW_ERR_INVALID_ARG, "mask B < 0");
    CHECK(sbw_detect(&tok, 1, 2, 2, 1, 0.0, SBW_SEED_CONTEXT, &cnt, &z, NULL) == SBW_ERR_GAMMA, "detect gamma 0");
    CHECK(sbw_detect(&tok, 1, 2, 1, 1, 0.25, SBW_SEED_CONTEXT, &cnt, &z, NULL) == SBW_ERR_INVALID_ARG, "detect stride < L");
    CHECK(sbw_detect(NULL, 0, 5, 5, 1, 0.25, SBW_SEED_CONTEXT, NULL, NULL, NULL) == SBW_OK, "detect N = 0");
    CHECK(sbw_detect_window(&tok, 1, (int64_t)1 << 31, (int64_t)1 << 31, 1, 1, 0.25, SBW_SEED_CONTEXT, &cnt, &z, NULL) == SBW_ERR_UNSUPPORTED, "L = 2^31");
    CHECK(sbw_detect_ex(&tok, 1, 2, 2, NULL, 1, 1, 0.25, SBW_SEED_CONTEXT, 2u, &cnt, NULL, &z, NULL) == SBW_ERR_UNSUPPORTED, "unknown flag");
    CHECK(sbw_detect_ex(&tok, 1, 5000, 5000, NULL, 1, 1, 0.25, SBW_SEED_CONTEXT, SBW_DETECT_IGNORE_REPEATED, &cnt, NULL, &z, NULL) == SBW_ERR_UNSUPPORTED, "repeat rule beyond 4096");
    CHECK(sbw_watermark_candidates(&dummy, SBW_F32, 1, 1, 1, &cand, 1025, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_SELF_SALT, NULL) == SBW_ERR_UNSUPPORTED, "k > 1024");
    CHECK(sbw_watermark_candidates(&dummy, SBW_F32, 1, 1, 1, &cand, -1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_SELF_SALT, NULL) == SBW_ERR_INVALID_ARG, "k < 0");
    CHECK(sbw_watermark_argmax(&dummy, SBW_F32, 1, 1, 1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &tok, NULL, NULL, NULL) == SBW_ERR_INVALID_ARG, "argmax without workspace");
    CHECK(sbw_watermark_argmax(&dummy, SBW_F32, 1, 0, 0, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &tok, NULL, &ws, NULL) == SBW_ERR_INVALID_ARG, "argmax V = 0");
    CHECK(sbw_watermark_sample(&dummy, SBW_F32, 1, 1, 1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &seed, 0.0f, &tok, NULL, &ws, NULL) == SBW_ERR_INVALID_ARG, "1/T = 0");
    CHECK(sbw_watermark_sample(&dummy, SBW_F32, 1, 1, 1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, NULL, 1.0f, &tok, NULL, &ws, NULL) == SBW_ERR_INVALID_ARG, "no seeds");
    CHECK(sbw_watermark_argmax_noalloc(&dummy, SBW_F32, 3496, 152064, 152064, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &tok, NULL, NULL) == SBW_ERR_UNSUPPORTED, "noalloc beyond its array");
    CHECK(sbw_watermark_argmax_noalloc(&dummy, (sbw_dtype_t)2, 1, 1, 1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &tok, NULL, NULL) == SBW_ERR_UNSUPPORTED, "noalloc dtype 2");
    CHECK(sbw_watermark_argmax_noalloc(&dummy, SBW_F32, 0, 1, 1, &prev, 1, 1, 0.25, 2.0f, SBW_SEED_CONTEXT, &tok, NULL, NULL) == SBW_OK, "noalloc B = 0");
    printf("capi cpu ok: libsbw %s\n", v);
    return 0;
}

static int gpu_checks(void)
{
    const int64_t B = 8, V = 50001, W = 4, N = 16, L = 300;
    const uint64_t key = 0x243F6A8885A308D3ULL;
    const double gamma = 0.25;
    const float delta = 2.0f, inv_t = 0.8f;
    size_t nl = (size_t)(B * V);
    float *x = malloc(nl * sizeof(float)), *expect = malloc(nl * sizeof(float)),
          *got = malloc(nl * sizeof(float));
    int32_t ctx[8 * 4], tok[16 * 300], etok[8], gtok[8], ecount[16], gcount[16];
    float evals[8], gvals[8];
    uint64_t seeds[8];
    double ez[16], gz[16];
    CHECK(x && expect && got, "host allocation");
    rng_state = 0x9E3779B97F4A7C15ULL;
    for (size_t i = 0; i < nl; ++i) x[i] = next_logit();
    x[3 * V + 777] = NAN;                           /* a NaN row: its first NaN wins */
    for (int i = 0; i < B * W; ++i) ctx[i] = (int32_t)(next_u64() % (uint64_t)V);
    for (int i = 0; i < B; ++i) seeds[i] = next_u64();
    for (int i = 0; i < N * L; ++i) tok[i] = (int32_t)(next_u64() % (uint64_t)V);

    float *d_x, *d_vals;
    int32_t *d_ctx, *d_tok, *d_tokens, *d_count;
    uint64_t *d_seeds, *d_ws;
    double *d_z;
    const int64_t ws = sbw_watermark_argmax_workspace(B, V);
    HIP(hipMalloc((void **)&d_x, nl * sizeof(float)));
    HIP(hipMalloc((void **)&d_vals, B * sizeof(float)));
    HIP(hipMalloc((void **)&d_ctx, sizeof ctx));
    HIP(hipMalloc((void **)&d_tok, sizeof tok));
    HIP(hipMalloc((void **)&d_tokens, B * sizeof(int32_t)));
    HIP(hipMalloc((void **)&d_count, N * sizeof(int32_t)));
    HIP(hipMalloc((void **)&d_seeds, sizeof seeds));
    HIP(hipMalloc((void **)&d_ws, (size_t)ws * sizeof(uint64_t)));
    HIP(hipMalloc((void **)&d_z, N * sizeof(double)));
    HIP(hipMemcpy(d_ctx, ctx, sizeof ctx, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_tok, tok, sizeof tok, hipMemcpyHostToDevice));
    HIP(hipMemcpy(d_seeds, seeds, sizeof seeds, hipMemcpyHostToDevice));

    for (int seeding = 0; seeding < 2; ++seeding) {
        const sbw_seeding_t sd = (sbw_seeding_t)seeding;
        /* greedy decoding and sampling read the unmodified logits */
        HIP(hipMemcpy(d_x, x, nl * sizeof(float), hipMemcpyHostToDevice));
        SBW(sbw_watermark_argmax(d_x, SBW_F32, B, V, V, d_ctx, W, key, gamma, delta, sd,
                                 d_tokens, d_vals, d_ws, NULL));
        HIP(hipMemcpy(gtok, d_tokens, sizeof gtok, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(gvals, d_vals, sizeof gvals, hipMemcpyDeviceToHost));
        oracle_watermark_argmax_f32_w(x, B, V, V, ctx, W, key, gamma, delta, seeding, etok, evals);
        CHECK(memcmp(gtok, etok, sizeof etok) == 0 && memcmp(gvals, evals, sizeof evals) == 0,
              "argmax, seeding %d", seeding);
        /* the same through the call that keeps its partials in the library's own array */
        HIP(hipMemset(d_tokens, 0xFF, B * sizeof(int32_t)));
        SBW(sbw_watermark_argmax_noalloc(d_x, SBW_F32, B, V, V, d_ctx, W, key, gamma, delta, sd,
                                         d_tokens, d_vals, NULL));
        HIP(hipMemcpy(gtok, d_tokens, sizeof gtok, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(gvals, d_vals, sizeof gvals, hipMemcpyDeviceToHost));
        CHECK(memcmp(gtok, etok, sizeof etok) == 0 && memcmp(gvals, evals, sizeof evals) == 0,
              "argmax without a workspace, seeding %d", seeding);
        SBW(sbw_watermark_sample(d_x, SBW_F32, B, V, V, d_ctx, W, key, gamma, delta, sd, d_seeds,
                                 inv_t, d_tokens, d_vals, d_ws, NULL));
        HIP(hipMemcpy(gtok, d_tokens, sizeof gtok, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(gvals, d_vals, sizeof gvals, hipMemcpyDeviceToHost));
        oracle_watermark_sample_f32_w(x, B, V, V, ctx, W, key, gamma, delta, seeding, seeds, inv_t,
                                      etok, evals);
        CHECK(memcmp(gtok, etok, sizeof etok) == 0 && memcmp(gvals, evals, sizeof evals) == 0,
              "sample, seeding %d", seeding);
        CHECK(gtok[3] == 777, "the NaN logit wins the sample");
        /* the same draw from two vocabulary shards, [0, S) and [S, V), reduced here:
           the larger score, the smaller id among equal ones, a NaN above all */
        {
            const int64_t S = 20003;
            int32_t t0[8], t1[8];
            float s0[8], s1[8];
            SBW(sbw_watermark_sample_shard(d_x, SBW_F32, B, S, V, d_ctx, W, 0, key, gamma, delta, sd,
                                           d_seeds, inv_t, d_tokens, d_vals, d_ws, NULL));
            HIP(hipMemcpy(t0, d_tokens, sizeof t0, hipMemcpyDeviceToHost));
            HIP(hipMemcpy(s0, d_vals, sizeof s0, hipMemcpyDeviceToHost));
            SBW(sbw_watermark_sample_shard(d_x + S, SBW_F32, B, V - S, V, d_ctx, W, S, key, gamma,
                                           delta, sd, d_seeds, inv_t, d_tokens, d_vals, d_ws, NULL));
            HIP(hipMemcpy(t1, d_tokens, sizeof t1, hipMemcpyDeviceToHost));
            HIP(hipMemcpy(s1, d_vals, sizeof s1, hipMemcpyDeviceToHost));
            for (int b = 0; b < B; ++b) {
                const int second = !isnan(s0[b]) && (isnan(s1[b]) || s1[b] > s0[b]);
                const int32_t t = second ? t1[b] : t0[b];
                const float sc = second ? s1[b] : s0[b];
                CHECK(t == etok[b] && memcmp(&sc, &evals[b], sizeof sc) == 0,
                      "sample from shards, row %d, seeding %d", b, seeding);
            }
        }
        /* then the watermark in place */
        SBW(sbw_watermark_window(d_x, SBW_F32, B, V, V, d_ctx, W, key, gamma, delta, sd, NULL));
        HIP(hipMemcpy(got, d_x, nl * sizeof(float), hipMemcpyDeviceToHost));
        memcpy(expect, x, nl * sizeof(float));
        oracle_watermark_f32_w(expect, B, V, V, ctx, W, key, gamma, delta, seeding);
        CHECK(memcmp(got, expect, nl * sizeof(float)) == 0, "watermark, seeding %d", seeding);
        /* detection */
        SBW(sbw_detect_window(d_tok, N, L, L, W, key, gamma, sd, d_count, d_z, NULL));
        HIP(hipMemcpy(gcount, d_count, sizeof gcount, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(gz, d_z, sizeof gz, hipMemcpyDeviceToHost));
        oracle_detect_w(tok, N, L, L, W, key, gamma, seeding, ecount, ez);
        CHECK(memcmp(gcount, ecount, sizeof ecount) == 0, "detect counts, seeding %d", seeding);
        for (int i = 0; i < N; ++i)
            CHECK(fabs(gz[i] - ez[i]) <= 1e-6 * fabs(ez[i]) + 1e-12, "detect z, seeding %d", seeding);
        /* green masks */
        {
            const int64_t words = (V + 31) / 32;
            uint32_t *gbits = malloc((size_t)(B * words) * sizeof(uint32_t)),
                     *ebits = malloc((size_t)(B * words) * sizeof(uint32_t)), *d_bits;
            CHECK(gbits && ebits, "host allocation");
            HIP(hipMalloc((void **)&d_bits, (size_t)(B * words) * sizeof(uint32_t)));
            SBW(sbw_green_mask_window(d_bits, B, V, d_ctx, W, key, gamma, sd, NULL));
            HIP(hipMemcpy(gbits, d_bits, (size_t)(B * words) * sizeof(uint32_t), hipMemcpyDeviceToHost));
            oracle_green_mask_w(ebits, B, V, ctx, W, key, gamma, seeding);
            CHECK(memcmp(gbits, ebits, (size_t)(B * words) * sizeof(uint32_t)) == 0,
                  "green mask, seeding %d", seeding);
            HIP(hipFree(d_bits));
            free(gbits); free(ebits);
        }
        /* the watermark on 40 candidate ids per row (one out of range, one repeated) */
        {
            int32_t cand[8 * 40], *d_cand;
            for (int i = 0; i < B * 40; ++i) cand[i] = (int32_t)(next_u64() % (uint64_t)V);
            cand[5] = (int32_t)V;
            cand[7] = cand[6];
            HIP(hipMalloc((void **)&d_cand, sizeof cand));
            HIP(hipMemcpy(d_cand, cand, sizeof cand, hipMemcpyHostToDevice));
            HIP(hipMemcpy(d_x, x, nl * sizeof(float), hipMemcpyHostToDevice));
            SBW(sbw_watermark_candidates(d_x, SBW_F32, B, V, V, d_cand, 40, d_ctx, W, key, gamma,
                                         delta, sd, NULL));
            HIP(hipMemcpy(got, d_x, nl * sizeof(float), hipMemcpyDeviceToHost));
            memcpy(expect, x, nl * sizeof(float));
            oracle_watermark_candidates_f32_w(expect, B, V, V, cand, 40, ctx, W, key, gamma, delta,
                                              seeding);
            CHECK(memcmp(got, expect, nl * sizeof(float)) == 0, "candidates, seeding %d", seeding);
            HIP(hipFree(d_cand));
        }
        /* detection with per-text lengths and the repeated-n-gram rule */
        {
            int32_t lens[16], *d_lens, gscored[16], escored[16], *d_scored;
            for (int i = 0; i < N; ++i) lens[i] = (int32_t)(next_u64() % (uint64_t)(L + 1));
            for (int i = 0; i < L / 2; ++i) tok[3 * L + L / 2 + i] = tok[3 * L + i];  /* repeats */
            HIP(hipMemcpy(d_tok, tok, sizeof tok, hipMemcpyHostToDevice));
            HIP(hipMalloc((void **)&d_lens, sizeof lens));
            HIP(hipMalloc((void **)&d_scored, sizeof gscored));
            HIP(hipMemcpy(d_lens, lens, sizeof lens, hipMemcpyHostToDevice));
            for (int rule = 0; rule < 2; ++rule) {
                SBW(sbw_detect_ex(d_tok, N, L, L, d_lens, W, key, gamma, sd,
                                  rule ? (uint32_t)SBW_DETECT_IGNORE_REPEATED : 0u, d_count,
                                  d_scored, d_z, NULL));
                HIP(hipMemcpy(gcount, d_count, sizeof gcount, hipMemcpyDeviceToHost));
                HIP(hipMemcpy(gscored, d_scored, sizeof gscored, hipMemcpyDeviceToHost));
                HIP(hipMemcpy(gz, d_z, sizeof gz, hipMemcpyDeviceToHost));
                oracle_detect_ex(tok, N, L, L, lens, W, key, gamma, seeding, rule, ecount, escored, ez);
                CHECK(memcmp(gcount, ecount, sizeof ecount) == 0 &&
                      memcmp(gscored, escored, sizeof escored) == 0,
                      "detect_ex counts, rule %d, seeding %d", rule, seeding);
                for (int i = 0; i < N; ++i)
                    CHECK((isnan(gz[i]) && isnan(ez[i])) ||
                          fabs(gz[i] - ez[i]) <= 1e-6 * fabs(ez[i]) + 1e-12,
                          "detect_ex z, rule %d, seeding %d", rule, seeding);
            }
            HIP(hipFree(d_lens));
            HIP(hipFree(d_scored));
        }
        printf("capi gpu seeding %d ok\n", seeding);
    }
    HIP(hipFree(d_x)); HIP(hipFree(d_vals)); HIP(hipFree(d_ctx)); HIP(hipFree(d_tok));
    HIP(hipFree(d_tokens)); HIP(hipFree(d_count)); HIP(hipFree(d_seeds)); HIP(hipFree(d_ws));
    HIP(hipFree(d_z));
    free(x); free(expect); free(got);
    printf("capi gpu ok\n");
    return 0;
}

int main(int argc, char **argv)
{
    if (argc == 2 && strcmp(argv[1], "cpu") == 0) return cpu_checks();
    if (argc == 2 && strcmp(argv[1], "gpu") == 0) return gpu_checks();
    fprintf(stderr, "usage: capi_check cpu|gpu\n");
    return 2;
}
