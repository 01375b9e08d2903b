/*
 * Every entry point of the C oracle (oracle/sbw_oracle.c) on edge shapes, for a build
 * with AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_sanitize_cpu.py):
 * a vocabulary of one token, rows whose length is not a multiple of 32, padded rows,
 * texts of 0, 1 and 2 tokens, windows of 8, lengths below 0 and beyond L, candidate
 * ids -1, V and 2^31 - 1, repeated candidates, empty arrays.  Every buffer is
 * allocated at its exact size, so that a read or write one element too far is caught.
 * A few results with a closed form are checked too; the sanitizers do the rest.
 * Prints "oracle edges ok" and exits 0 when nothing was reported.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_philox4x32_10(const uint32_t counter[4], const uint32_t key[2], uint32_t out[4]);
uint32_t oracle_cbrng(uint32_t v, uint64_t r);
uint64_t oracle_threshold(double gamma);
uint32_t oracle_jenkins32(uint32_t a);
uint64_t oracle_seed_context(uint64_t key, uint32_t prev);
uint64_t oracle_seed_self_salt(uint64_t key, uint32_t prev, uint32_t cand);
uint64_t oracle_seed(uint64_t key, uint32_t prev, uint32_t cand, int seeding);
int oracle_is_green(uint64_t key, uint32_t prev, uint32_t cand, uint64_t threshold, int seeding);
void oracle_is_green_many(uint64_t key, const int32_t *prev, const int32_t *cand, int64_t n,
                          double gamma, int seeding, uint8_t *out);
uint16_t oracle_f32_to_bf16(float f);
float oracle_bias_f32(float logit, float delta);
uint16_t oracle_bias_bf16(uint16_t logit, float delta);
void oracle_watermark_f32(float *logits, int64_t B, int64_t V, int64_t row_stride,
                          const int32_t *prev, uint64_t key, double gamma, float delta,
                          int seeding);
void oracle_watermark_bf16(uint16_t *logits, int64_t B, int64_t V, int64_t row_stride,
                           const int32_t *prev, uint64_t key, double gamma, float delta,
                           int seeding);
void oracle_green_mask(uint32_t *bits, int64_t B, int64_t V, const int32_t *prev, uint64_t key,
                       double gamma, int seeding);
double oracle_z_score(int64_t green_count, int64_t T, double gamma);
void oracle_detect(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride, uint64_t key,
                   double gamma, int seeding, int32_t *green_counts, double *z);
void oracle_cbrng_many(const uint32_t *v, const uint64_t *r, int64_t n, uint32_t *out);
void oracle_jenkins32_many(const uint32_t *a, int64_t n, uint32_t *out);
void oracle_seed_many(uint64_t key, const int32_t *prev, const int32_t *cand, int64_t n,
                      int seeding, uint64_t *out);
void oracle_bias_f32_many(const float *in, int64_t n, float delta, float *out);
void oracle_bias_bf16_many(const uint16_t *in, int64_t n, float delta, uint16_t *out);
void oracle_f32_to_bf16_many(const float *in, int64_t n, uint16_t *out);
uint64_t oracle_seed_context_w(uint64_t key, const int32_t *context, int64_t width);
uint64_t oracle_seed_self_salt_w(uint64_t key, const int32_t *context, int64_t width,
                                 uint32_t cand);
uint64_t oracle_seed_w(uint64_t key, const int32_t *context, int64_t width, uint32_t cand,
                       int seeding);
int oracle_is_green_w(uint64_t key, const int32_t *context, int64_t width, uint32_t cand,
                      uint64_t threshold, int seeding);
void oracle_watermark_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                            const int32_t *context, int64_t width, uint64_t key, double gamma,
                            float delta, int seeding);
void oracle_watermark_bf16_w(uint16_t *logits, int64_t B, int64_t V, int64_t row_stride,
                             const int32_t *context, int64_t width, uint64_t key, double gamma,
                             float delta, int seeding);
void oracle_green_mask_w(uint32_t *bits, int64_t B, int64_t V, const int32_t *context,
                         int64_t width, uint64_t key, double gamma, int seeding);
void oracle_detect_w(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                     int64_t width, uint64_t key, double gamma, int seeding,
                     int32_t *green_counts, double *z);
void oracle_seed_w_many(uint64_t key, const int32_t *context, int64_t width, const int32_t *cand,
                        int64_t n, int seeding, uint64_t *out);
void oracle_is_green_w_many(uint64_t key, const int32_t *context, int64_t width,
                            const int32_t *cand, int64_t n, double gamma, int seeding,
                            uint8_t *out);
void oracle_watermark_argmax_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, int32_t *tokens,
                                   float *values);
void oracle_watermark_argmax_bf16_w(const uint16_t *logits, int64_t B, int64_t V,
                                    int64_t row_stride, const int32_t *context, int64_t width,
                                    uint64_t key, double gamma, float delta, int seeding,
                                    int32_t *tokens, float *values);
void oracle_watermark_candidates_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                                       const int32_t *cand, int64_t k, const int32_t *context,
                                       int64_t width, uint64_t key, double gamma, float delta,
                                       int seeding);
void oracle_watermark_candidates_bf16_w(uint16_t *logits, int64_t B, int64_t V,
                                        int64_t row_stride, const int32_t *cand, int64_t k,
                                        const int32_t *context, int64_t width, uint64_t key,
                                        double gamma, float delta, int seeding);
void oracle_detect_ex(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                      const int32_t *lengths, int64_t width, uint64_t key, double gamma,
                      int seeding, int ignore_repeated, int32_t *green_counts, int32_t *scored,
                      double *z);
float oracle_sample_log(float x);
float oracle_gumbel_of_draw(uint32_t x);
float oracle_gumbel(uint32_t v, uint64_t seed);
void oracle_watermark_sample_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, const uint64_t *seeds,
                                   float inv_temperature, int32_t *tokens, float *scores);
void oracle_watermark_sample_bf16_w(const uint16_t *logits, int64_t B, int64_t V,
                                    int64_t row_stride, const int32_t *context, int64_t width,
                                    uint64_t key, double gamma, float delta, int seeding,
                                    const uint64_t *seeds, float inv_temperature,
                                    int32_t *tokens, float *scores);
void oracle_sample_log_many(const float *x, int64_t n, float *out);
void oracle_gumbel_many(const uint32_t *v, const uint64_t *seed, int64_t n, float *out);
void oracle_gumbel_of_draws(const uint32_t *x, int64_t n, float *out);

static const uint64_t KEYS[] = {15485863ull, 0x243F6A8885A308D3ull, 0ull, ~0ull};
static const double GAMMAS[] = {0.0, 5e-324, 0.25, 0.5, 1.0 - 1e-10, 1.0};
static const float DELTAS[] = {2.0f, -3.0f, 0.0f, 3e38f};

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1DULL;
}

static int failures = 0;
#define CHECK(cond)                                                                  \
    do {                                                                             \
        if (!(cond)) {                                                               \
            printf("check failed at line %d: %s\n", __LINE__, #cond);                \
            ++failures;                                                              \
        }                                                                            \
    } while (0)

/* Exact-size buffers: the sanitizer sees one element past the end. */
static void *xalloc(size_t n, size_t size)
{
    void *p = malloc(n ? n * size : 1);
    if (!p) {
        printf("out of memory\n");
        exit(2);
    }
    return p;
}

static float *logits_f32(int64_t n)
{
    float *x = xalloc((size_t)n, sizeof(float));
    for (int64_t i = 0; i < n; ++i)
        x[i] = (float)((double)(next_u64() >> 11) * 0x1p-53 * 8.0 - 4.0);
    if (n > 2) {
        x[0] = INFINITY;
        x[1] = NAN;
        x[2] = -0.0f;
    }
    return x;
}

static uint16_t *logits_bf16(int64_t n)
{
    uint16_t *x = xalloc((size_t)n, sizeof(uint16_t));
    for (int64_t i = 0; i < n; ++i) x[i] = (uint16_t)next_u64();
    return x;
}

static int32_t *tokens_of(int64_t n, int64_t V)
{
    int32_t *t = xalloc((size_t)n, sizeof(int32_t));
    for (int64_t i = 0; i < n; ++i) t[i] = V > 0 ? (int32_t)(next_u64() % (uint64_t)V) : 0;
    return t;
}

static void scalars(void)
{
    const uint32_t ctr[4] = {0u, 0u, 0u, 0u}, key[2] = {0u, 0u};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    /* Random123's known answer for the zero counter and key */
    CHECK(out[0] == 0x6627e8d5u && out[1] == 0xe169c58du && out[2] == 0xbc57ac4cu &&
          out[3] == 0x9b00dbd8u);
    for (int k = 0; k < 4; ++k) {
        const uint32_t vs[] = {0u, 1u, 3u, 4u, 0x7FFFFFFFu, 0xFFFFFFFFu};
        for (int i = 0; i < 6; ++i) {
            (void)oracle_cbrng(vs[i], KEYS[k]);
            (void)oracle_seed_context(KEYS[k], vs[i]);
            (void)oracle_seed_self_salt(KEYS[k], vs[i], vs[5 - i]);
            for (int s = 0; s < 2; ++s) {
                (void)oracle_seed(KEYS[k], vs[i], vs[5 - i], s);
                (void)oracle_is_green(KEYS[k], vs[i], vs[5 - i], 1ull << 30, s);
                (void)oracle_is_green(KEYS[k], vs[i], vs[5 - i], 1ull << 32, s);
            }
        }
    }
    CHECK(oracle_threshold(0.0) == 0 && oracle_threshold(1.0) == (1ull << 32));
    CHECK(oracle_threshold(0.25) == (1ull << 30) && oracle_threshold(5e-324) == 1);
    for (int g = 0; g < 6; ++g) (void)oracle_threshold(GAMMAS[g]);
    (void)oracle_jenkins32(0u);
    (void)oracle_jenkins32(0xFFFFFFFFu);
    CHECK(oracle_f32_to_bf16(1.0f) == 0x3F80u);
    CHECK(oracle_f32_to_bf16(NAN) != 0u);
    (void)oracle_bias_f32(INFINITY, -3e38f);
    (void)oracle_bias_bf16(0x7F80u, 2.0f);
    (void)oracle_bias_bf16(0xFFC1u, 2.0f);
    CHECK(isnan(oracle_z_score(0, 0, 0.25)));
    (void)oracle_z_score(0, 1, 0.5);
    (void)oracle_z_score(511, 511, 0.25);
    (void)oracle_sample_log(1.0f);
    (void)oracle_sample_log(0x1p-126f);
    (void)oracle_sample_log(3.4e38f);
    (void)oracle_gumbel_of_draw(0u);
    (void)oracle_gumbel_of_draw(0xFFFFFFFFu);
    (void)oracle_gumbel(0xFFFFFFFFu, ~0ull);
    const int32_t ctx8[8] = {0, -1, 2147483647, 5, 5, 7, 0, 1};
    for (int64_t w = 1; w <= 8; ++w) {
        (void)oracle_seed_context_w(KEYS[1], ctx8, w);
        (void)oracle_seed_self_salt_w(KEYS[1], ctx8, w, 0xFFFFFFFFu);
        for (int s = 0; s < 2; ++s) {
            (void)oracle_seed_w(KEYS[1], ctx8, w, 3u, s);
            (void)oracle_is_green_w(KEYS[1], ctx8, w, 3u, 1ull << 31, s);
        }
    }
}

static void many(void)
{
    for (int64_t n = 0; n <= 37; n += 37) {
        uint32_t *v = xalloc((size_t)n, sizeof(uint32_t)), *o32 = xalloc((size_t)n, sizeof(uint32_t));
        uint64_t *r = xalloc((size_t)n, sizeof(uint64_t)), *o64 = xalloc((size_t)n, sizeof(uint64_t));
        int32_t *p = tokens_of(n, 1000), *c = tokens_of(n, 1000);
        uint8_t *g = xalloc((size_t)n, 1);
        float *f = logits_f32(n), *of = xalloc((size_t)n, sizeof(float));
        uint16_t *h = logits_bf16(n), *oh = xalloc((size_t)n, sizeof(uint16_t));
        for (int64_t i = 0; i < n; ++i) {
            v[i] = (uint32_t)next_u64();
            r[i] = next_u64();
        }
        oracle_cbrng_many(v, r, n, o32);
        oracle_jenkins32_many(v, n, o32);
        for (int s = 0; s < 2; ++s) {
            oracle_seed_many(KEYS[0], p, c, n, s, o64);
            oracle_is_green_many(KEYS[0], p, c, n, 0.25, s, g);
            oracle_seed_w_many(KEYS[0], p, 1, c, n, s, o64);
            oracle_is_green_w_many(KEYS[0], p, 1, c, n, 0.5, s, g);
        }
        oracle_bias_f32_many(f, n, 2.0f, of);
        oracle_bias_bf16_many(h, n, 2.0f, oh);
        oracle_f32_to_bf16_many(f, n, oh);
        for (int64_t i = 0; i < n; ++i) f[i] = fabsf(f[i]) + 1e-3f;
        oracle_sample_log_many(f, n, of);
        oracle_gumbel_many(v, r, n, of);
        oracle_gumbel_of_draws(v, n, of);
        free(v); free(o32); free(r); free(o64); free(p); free(c); free(g);
        free(f); free(of); free(h); free(oh);
    }
}

/* Watermark, green masks, decoding and candidates on one shape. */
static void logits_shape(int64_t B, int64_t V, int64_t pad, int64_t width)
{
    const int64_t stride = V + pad, n = B * stride;
    int32_t *ctx = tokens_of(B * width, V > 0 ? V : 1);
    int32_t *ctx1 = tokens_of(B, V > 0 ? V : 1);
    const int64_t words = (V + 31) / 32;
    uint32_t *bits = xalloc((size_t)(B * words), sizeof(uint32_t));
    int32_t *tok = xalloc((size_t)B, sizeof(int32_t));
    float *val = xalloc((size_t)B, sizeof(float));
    uint64_t *seeds = xalloc((size_t)B, sizeof(uint64_t));
    for (int64_t b = 0; b < B; ++b) seeds[b] = next_u64();
    for (int s = 0; s < 2; ++s) {
        for (int gi = 0; gi < 6; ++gi) {
            const double gamma = GAMMAS[gi];
            const float delta = DELTAS[gi % 4];
            float *x = logits_f32(n);
            uint16_t *y = logits_bf16(n);
            oracle_watermark_f32(x, B, V, stride, ctx1, KEYS[gi % 4], gamma, delta, s);
            oracle_watermark_bf16(y, B, V, stride, ctx1, KEYS[gi % 4], gamma, delta, s);
            oracle_watermark_f32_w(x, B, V, stride, ctx, width, KEYS[gi % 4], gamma, delta, s);
            oracle_watermark_bf16_w(y, B, V, stride, ctx, width, KEYS[gi % 4], gamma, delta, s);
            oracle_green_mask(bits, B, V, ctx1, KEYS[gi % 4], gamma, s);
            if (gamma == 0.0)
                for (int64_t i = 0; i < B * words; ++i) CHECK(bits[i] == 0u);
            oracle_green_mask_w(bits, B, V, ctx, width, KEYS[gi % 4], gamma, s);
            if (V > 0) {
                oracle_watermark_argmax_f32_w(x, B, V, stride, ctx, width, KEYS[gi % 4], gamma,
                                              delta, s, tok, val);
                for (int64_t b = 0; b < B; ++b) CHECK(tok[b] >= 0 && tok[b] < V);
                oracle_watermark_argmax_bf16_w(y, B, V, stride, ctx, width, KEYS[gi % 4], gamma,
                                               delta, s, tok, val);
                oracle_watermark_sample_f32_w(x, B, V, stride, ctx, width, KEYS[gi % 4], gamma,
                                              delta, s, seeds, 0.37f, tok, val);
                for (int64_t b = 0; b < B; ++b) CHECK(tok[b] >= 0 && tok[b] < V);
                oracle_watermark_sample_bf16_w(y, B, V, stride, ctx, width, KEYS[gi % 4], gamma,
                                               delta, s, seeds, 1e30f, tok, val);
            }
            /* candidates: out-of-range ids, repeats, a full row of the vocabulary */
            const int64_t k = 7 + (V > 0 ? V : 0);
            int32_t *cand = xalloc((size_t)(B * k), sizeof(int32_t));
            for (int64_t b = 0; b < B; ++b) {
                int32_t *c = cand + b * k;
                c[0] = -1;
                c[1] = (int32_t)V;
                c[2] = 2147483647;
                c[3] = V > 0 ? (int32_t)(V - 1) : 0;
                c[4] = c[3];
                c[5] = 0;
                c[6] = -2147483647 - 1;
                for (int64_t i = 7; i < k; ++i) c[i] = (int32_t)(i - 7);
            }
            oracle_watermark_candidates_f32_w(x, B, V, stride, cand, k, ctx, width, KEYS[gi % 4],
                                              gamma, delta, s);
            oracle_watermark_candidates_bf16_w(y, B, V, stride, cand, k, ctx, width,
                                               KEYS[gi % 4], gamma, delta, s);
            free(cand);
            free(x);
            free(y);
        }
    }
    free(ctx); free(ctx1); free(bits); free(tok); free(val); free(seeds);
}

/* Detection on one shape: every entry point, lengths outside [0, L], both rules. */
static void detect_shape(int64_t N, int64_t L, int64_t width, int64_t V)
{
    const int64_t stride = L + 3;
    int32_t *t = tokens_of(N * stride, V);
    if (N > 1 && L > 4)   /* a repeated stretch for the repeat rule */
        memcpy(t + stride + L / 2, t + stride, (size_t)(L / 2 - 1) * sizeof(int32_t));
    int32_t *counts = xalloc((size_t)N, sizeof(int32_t)), *scored = xalloc((size_t)N, sizeof(int32_t));
    double *z = xalloc((size_t)N, sizeof(double));
    int32_t *lengths = xalloc((size_t)N, sizeof(int32_t));
    const int32_t pick[] = {-5, 0, 1, (int32_t)L, (int32_t)L + 7, 2147483647, (int32_t)(L / 2)};
    for (int64_t n = 0; n < N; ++n) lengths[n] = pick[n % 7];
    for (int s = 0; s < 2; ++s) {
        oracle_detect(t, N, L, stride, KEYS[0], 0.25, s, counts, z);
        for (int64_t n = 0; n < N; ++n) CHECK(counts[n] >= 0 && counts[n] <= (L > 1 ? L - 1 : 0));
        oracle_detect_w(t, N, L, stride, width, KEYS[1], 0.5, s, counts, z);
        for (int rep = 0; rep < 2; ++rep) {
            oracle_detect_ex(t, N, L, stride, NULL, width, KEYS[0], 0.25, s, rep, counts, scored, z);
            oracle_detect_ex(t, N, L, stride, lengths, width, KEYS[0], 0.25, s, rep, counts, scored,
                             z);
            for (int64_t n = 0; n < N; ++n) {
                CHECK(scored[n] >= 0 && scored[n] <= (L > width ? L - width : 0));
                CHECK(counts[n] >= 0 && counts[n] <= scored[n]);
                CHECK(scored[n] > 0 || isnan(z[n]));
            }
        }
    }
    free(t); free(counts); free(scored); free(z); free(lengths);
}

int main(void)
{
    scalars();
    many();
    const int64_t shapes[][4] = {
        /* B, V, pad, width */
        {1, 1, 0, 1}, {3, 1, 2, 8}, {2, 37, 0, 4}, {2, 33, 5, 1}, {4, 64, 3, 8}, {1, 0, 4, 2},
        {5, 257, 1, 2},
    };
    for (size_t i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i)
        logits_shape(shapes[i][0], shapes[i][1], shapes[i][2], shapes[i][3]);
    const int64_t dshapes[][4] = {
        /* N, L, width, V */
        {2, 0, 1, 5}, {3, 1, 1, 5}, {3, 2, 1, 5}, {7, 9, 8, 3}, {7, 8, 8, 50}, {7, 200, 4, 128256},
        {14, 63, 1, 2}, {7, 130, 2, 1},
    };
    for (size_t i = 0; i < sizeof(dshapes) / sizeof(dshapes[0]); ++i)
        detect_shape(dshapes[i][0], dshapes[i][1], dshapes[i][2], dshapes[i][3]);
    if (failures) {
        printf("%d checks failed\n", failures);
        return 1;
    }
    printf("oracle edges ok\n");
    return 0;
}
