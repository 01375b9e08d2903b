/*
 * CPU oracle for Stateless Bernoulli Watermarking (SBW).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the watermark and detect hot path compute.  Only the test
 * suite, the smoke check and the CPU-baseline leg of the benchmark load it.  It
 * shares no source, header, table or helper with the HIP library, and the HIP
 * library never calls it.
 *
 * Every function evaluates the paper's definitions element by element, in the
 * order the paper states them, with no blocking, fusion or reuse between
 * elements.  Integer arithmetic is exact (uint32/uint64 wraparound is the
 * modular arithmetic the definitions use); floating point follows the
 * precision the definitions fix (one fp32 add; fp64 for the z-score).
 *
 * Readings taken where the paper is silent (each one is listed, with its
 * alternatives, in the design notes of the repository):
 *   R1  CBRNG(v, r) is the v-th 32-bit output of the Philox4x32-10 stream with
 *       key r and counter starting at 0: word (v mod 4) of the block at
 *       counter (floor(v/4), 0, 0, 0).
 *   R2  "CBRNG(v, r) < gamma" is the exact real comparison x * 2^-32 < gamma,
 *       i.e. x < ceil(gamma * 2^32).
 *   R3  Context seed ("additive" PRF, width 1): r = K * p mod 2^64.
 *   R4  The Jenkins integer hash is Robert Jenkins' six-step 32-bit mix.
 *   R5  Self-salt seed ("anchored minhash" over {p, v}, anchored on the
 *       candidate v): r = min_u64(K*J(p)*J(v), K*J(v)*J(v)), products mod 2^64,
 *       unsigned minimum.
 *   R6  Detection scores positions 1..L-1, T = L-1, no de-duplication.
 *   R7  bf16 bias: exact upcast, one fp32 add rounded to nearest even, one
 *       round-to-nearest-even down-conversion; NaN stays NaN.
 *   R8  Tokens are taken as their 32-bit pattern (no range check).
 *
 * Parity unpinned: jenkins32() has no printed value in the paper and no
 * independent implementation is available to compare against; it is checked
 * only through its properties (bijectivity, avalanche, uniformity).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as    */
/* easy as 1, 2, 3", SC'11), the CBRNG named in Sec. 2.2.                      */
/* ------------------------------------------------------------------------- */

/* Round multipliers and key-schedule (Weyl) increments as published. */
static const uint32_t PHILOX_MULT_A = 0xD2511F53u; /* applied to counter word 0 */
static const uint32_t PHILOX_MULT_B = 0xCD9E8D57u; /* applied to counter word 2 */
static const uint32_t PHILOX_WEYL_0 = 0x9E3779B9u; /* golden ratio */
static const uint32_t PHILOX_WEYL_1 = 0xBB67AE85u; /* sqrt(3) - 1  */

/* One Philox S-box: the full 64-bit product of two 32-bit words, split. */
static void mul_hi_lo(uint32_t a, uint32_t b, uint32_t *hi, uint32_t *lo)
{
    uint64_t product = (uint64_t)a * (uint64_t)b;
    *hi = (uint32_t)(product >> 32);
    *lo = (uint32_t)product;
}

/* Ten rounds; the key is bumped by the Weyl constants before rounds 2..10. */
void oracle_philox4x32_10(const uint32_t counter[4], const uint32_t key[2],
                          uint32_t out[4])
{
    uint32_t c0 = counter[0], c1 = counter[1], c2 = counter[2], c3 = counter[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_WEYL_0;
            k1 += PHILOX_WEYL_1;
        }
        uint32_t hi_a, lo_a, hi_b, lo_b;
        mul_hi_lo(PHILOX_MULT_A, c0, &hi_a, &lo_a);
        mul_hi_lo(PHILOX_MULT_B, c2, &hi_b, &lo_b);
        uint32_t n0 = hi_b ^ c1 ^ k0;
        uint32_t n1 = lo_b;
        uint32_t n2 = hi_a ^ c3 ^ k1;
        uint32_t n3 = lo_a;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* CBRNG(v, r), Sec. 2.2: the value at position v of the stream seeded by r,
 * without computing any earlier position (reading R1). */
uint32_t oracle_cbrng(uint32_t v, uint64_t r)
{
    uint32_t counter[4] = { v / 4u, 0u, 0u, 0u };
    uint32_t key[2] = { (uint32_t)r, (uint32_t)(r >> 32) };
    uint32_t block[4];
    oracle_philox4x32_10(counter, key, block);
    return block[v % 4u];
}

/* Membership threshold for "CBRNG(v, r) < gamma", Sec. 2.2, Eq. 1 (reading R2):
 * ceil(gamma * 2^32), clamped to [0, 2^32].  gamma * 2^32 is exact in binary64. */
uint64_t oracle_threshold(double gamma)
{
    double scaled = ceil(gamma * 4294967296.0);
    if (!(scaled > 0.0)) return 0u;               /* also catches NaN */
    if (scaled >= 4294967296.0) return 4294967296ull;
    return (uint64_t)scaled;
}

/* ------------------------------------------------------------------------- */
/* Seeds, Sec. 2.2 (seed from the preceding context via a PRF) and Sec. 2.3    */
/* (Jenkins integer hash for token ids).                                       */
/* ------------------------------------------------------------------------- */

/* Robert Jenkins' 32-bit integer hash (reading R4).  Parity unpinned. */
uint32_t oracle_jenkins32(uint32_t a)
{
    a = (a + 0x7ed55d16u) + (a << 12);
    a = (a ^ 0xc761c23cu) ^ (a >> 19);
    a = (a + 0x165667b1u) + (a << 5);
    a = (a + 0xd3a2646cu) ^ (a << 9);
    a = (a + 0xfd7046c5u) + (a << 3);
    a = (a ^ 0xb55a4f09u) ^ (a >> 16);
    return a;
}

/* Context seeding, additive PRF of width 1 (SBW-1; scheme table in App. D):
 * r = K * p mod 2^64 (reading R3). */
uint64_t oracle_seed_context(uint64_t key, uint32_t prev)
{
    return key * (uint64_t)prev;
}

/* Full-vocabulary self-salt seeding (Sec. 5.2; "anchored minhash" in App. D),
 * at width 1 over the window {p, v}, anchored on the candidate v (reading R5). */
uint64_t oracle_seed_self_salt(uint64_t key, uint32_t prev, uint32_t cand)
{
    uint64_t hp = (uint64_t)oracle_jenkins32(prev);
    uint64_t hv = (uint64_t)oracle_jenkins32(cand);
    uint64_t with_prev = key * hp * hv;
    uint64_t with_self = key * hv * hv;
    return with_prev < with_self ? with_prev : with_self;
}

/* Seeding scheme codes (the oracle's own; numerically equal to the library's
 * by agreement, checked by the tests, not by sharing a header). */
enum { ORACLE_SEED_CONTEXT = 0, ORACLE_SEED_SELF_SALT = 1 };

uint64_t oracle_seed(uint64_t key, uint32_t prev, uint32_t cand, int seeding)
{
    if (seeding == ORACLE_SEED_SELF_SALT) return oracle_seed_self_salt(key, prev, cand);
    return oracle_seed_context(key, prev);
}

/* v in G_t  <=>  CBRNG(v, r_t) < gamma   (Sec. 2.2, Eq. 1). */
int oracle_is_green(uint64_t key, uint32_t prev, uint32_t cand, uint64_t threshold,
                    int seeding)
{
    uint64_t r = oracle_seed(key, prev, cand, seeding);
    return (uint64_t)oracle_cbrng(cand, r) < threshold;
}

/* Array form of oracle_is_green for the workload sampler and the tests. */
void oracle_is_green_many(uint64_t key, const int32_t *prev, const int32_t *cand,
                          int64_t n, double gamma, int seeding, uint8_t *out)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t i = 0; i < n; ++i)
        out[i] = (uint8_t)oracle_is_green(key, (uint32_t)prev[i], (uint32_t)cand[i],
                                          threshold, seeding);
}

/* ------------------------------------------------------------------------- */
/* Logit bias, Sec. 2.2, Eq. 2: l' = l + delta on G_t, l' = l elsewhere.       */
/* ------------------------------------------------------------------------- */

static float f32_from_bits(uint32_t bits) { float f; memcpy(&f, &bits, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* fp32 -> bf16, round to nearest, ties to even; NaN stays NaN (reading R7). */
uint16_t oracle_f32_to_bf16(float f)
{
    uint32_t bits = bits_from_f32(f);
    if (isnan(f)) return (uint16_t)((bits >> 16) | 0x0040u);
    uint32_t upper = bits >> 16;
    uint32_t lower = bits & 0xFFFFu;
    if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
    return (uint16_t)upper;
}

float oracle_bias_f32(float logit, float delta) { return logit + delta; }

uint16_t oracle_bias_bf16(uint16_t logit, float delta)
{
    float widened = f32_from_bits((uint32_t)logit << 16);
    return oracle_f32_to_bf16(widened + delta);
}

/* In place over logits[b * row_stride + v], b < B, v < V. */
void oracle_watermark_f32(float *logits, int64_t B, int64_t V, int64_t row_stride,
                          const int32_t *prev, uint64_t key, double gamma, float delta,
                          int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t v = 0; v < V; ++v) {
            if (oracle_is_green(key, (uint32_t)prev[b], (uint32_t)v, threshold, seeding)) {
                float *l = &logits[b * row_stride + v];
                *l = oracle_bias_f32(*l, delta);
            }
        }
    }
}

void oracle_watermark_bf16(uint16_t *logits, int64_t B, int64_t V, int64_t row_stride,
                           const int32_t *prev, uint64_t key, double gamma, float delta,
                           int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t v = 0; v < V; ++v) {
            if (oracle_is_green(key, (uint32_t)prev[b], (uint32_t)v, threshold, seeding)) {
                uint16_t *l = &logits[b * row_stride + v];
                *l = oracle_bias_bf16(*l, delta);
            }
        }
    }
}

/* Green list G_t as a bit set: bit (v % 32) of word bits[b * ceil(V/32) + v/32]. */
void oracle_green_mask(uint32_t *bits, int64_t B, int64_t V, const int32_t *prev,
                       uint64_t key, double gamma, int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    int64_t words = (V + 31) / 32;
    for (int64_t i = 0; i < B * words; ++i) bits[i] = 0u;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t v = 0; v < V; ++v)
            if (oracle_is_green(key, (uint32_t)prev[b], (uint32_t)v, threshold, seeding))
                bits[b * words + v / 32] |= 1u << (v % 32);
}

/* ------------------------------------------------------------------------- */
/* Detection, Sec. 2.2 (O(1) per-token test) and Sec. 3 (z-score).             */
/* ------------------------------------------------------------------------- */

/* z = (W - T*gamma) / sqrt(T*gamma*(1-gamma)) in binary64, Sec. 3. */
double oracle_z_score(int64_t green_count, int64_t T, double gamma)
{
    double t = (double)T;
    double numerator = (double)green_count - t * gamma;
    double denominator = sqrt(t * gamma * (1.0 - gamma));
    return numerator / denominator;
}

/* For each sequence n: W = #{ i in 1..L-1 : tok[i] in G(tok[i-1]) } (R6). */
void oracle_detect(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                   uint64_t key, double gamma, int seeding, int32_t *green_counts,
                   double *z)
{
    uint64_t threshold = oracle_threshold(gamma);
    int64_t T = L > 1 ? L - 1 : 0;
    for (int64_t n = 0; n < N; ++n) {
        const int32_t *row = tokens + n * row_stride;
        int64_t count = 0;
        for (int64_t i = 1; i < L; ++i)
            count += oracle_is_green(key, (uint32_t)row[i - 1], (uint32_t)row[i],
                                     threshold, seeding);
        green_counts[n] = (int32_t)count;
        z[n] = oracle_z_score(count, T, gamma);
    }
}

/* ------------------------------------------------------------------------- */
/* Array forms of the scalar definitions above, for the tests.                 */
/* ------------------------------------------------------------------------- */

void oracle_cbrng_many(const uint32_t *v, const uint64_t *r, int64_t n, uint32_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_cbrng(v[i], r[i]);
}

void oracle_jenkins32_many(const uint32_t *a, int64_t n, uint32_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_jenkins32(a[i]);
}

void oracle_seed_many(uint64_t key, const int32_t *prev, const int32_t *cand, int64_t n,
                      int seeding, uint64_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_seed(key, (uint32_t)prev[i], (uint32_t)cand[i], seeding);
}

void oracle_bias_f32_many(const float *in, int64_t n, float delta, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bias_f32(in[i], delta);
}

void oracle_bias_bf16_many(const uint16_t *in, int64_t n, float delta, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bias_bf16(in[i], delta);
}

void oracle_f32_to_bf16_many(const float *in, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_bf16(in[i]);
}

/* ------------------------------------------------------------------------- */
/* Context width h (SBW-4 and SBW-ss-V in the scheme table of App. D; the      */
/* isolated benchmark of App. E).  The window is the h tokens before position   */
/* t, context[0..h-1]; both PRFs are symmetric in the window, so its order does */
/* not matter.                                                                   */
/*   R3h  additive PRF:   r = K * (p_1 + ... + p_h) mod 2^64, p_i as uint32      */
/*   R5h  anchored minhash with self-salt over {p_1..p_h, v}, anchored on v:     */
/*        r = min_u64( min_i K*J(p_i)*J(v), K*J(v)*J(v) )                        */
/*   R6h  detection scores positions h..L-1 (T = L - h) under the h tokens       */
/*        before each position.                                                 */
/* Width 1 is exactly the definitions above.                                     */
/* ------------------------------------------------------------------------- */

uint64_t oracle_seed_context_w(uint64_t key, const int32_t *context, int64_t width)
{
    uint64_t sum = 0;
    for (int64_t i = 0; i < width; ++i) sum += (uint64_t)(uint32_t)context[i];
    return key * sum;
}

uint64_t oracle_seed_self_salt_w(uint64_t key, const int32_t *context, int64_t width,
                                 uint32_t cand)
{
    uint64_t hv = (uint64_t)oracle_jenkins32(cand);
    uint64_t best = key * hv * hv;                       /* the candidate itself */
    for (int64_t i = 0; i < width; ++i) {
        uint64_t term = key * (uint64_t)oracle_jenkins32((uint32_t)context[i]) * hv;
        if (term < best) best = term;
    }
    return best;
}

uint64_t oracle_seed_w(uint64_t key, const int32_t *context, int64_t width, uint32_t cand,
                       int seeding)
{
    if (seeding == ORACLE_SEED_SELF_SALT)
        return oracle_seed_self_salt_w(key, context, width, cand);
    return oracle_seed_context_w(key, context, width);
}

int oracle_is_green_w(uint64_t key, const int32_t *context, int64_t width, uint32_t cand,
                      uint64_t threshold, int seeding)
{
    uint64_t r = oracle_seed_w(key, context, width, cand, seeding);
    return (uint64_t)oracle_cbrng(cand, r) < threshold;
}

/* context: [B, width] int32, row-major. */
void oracle_watermark_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                            const int32_t *context, int64_t width, uint64_t key, double gamma,
                            float delta, int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t v = 0; v < V; ++v)
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding)) {
                float *l = &logits[b * row_stride + v];
                *l = oracle_bias_f32(*l, delta);
            }
}

void oracle_watermark_bf16_w(uint16_t *logits, int64_t B, int64_t V, int64_t row_stride,
                             const int32_t *context, int64_t width, uint64_t key, double gamma,
                             float delta, int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t v = 0; v < V; ++v)
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding)) {
                uint16_t *l = &logits[b * row_stride + v];
                *l = oracle_bias_bf16(*l, delta);
            }
}

void oracle_green_mask_w(uint32_t *bits, int64_t B, int64_t V, const int32_t *context,
                         int64_t width, uint64_t key, double gamma, int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    int64_t words = (V + 31) / 32;
    for (int64_t i = 0; i < B * words; ++i) bits[i] = 0u;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t v = 0; v < V; ++v)
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding))
                bits[b * words + v / 32] |= 1u << (v % 32);
}

void oracle_detect_w(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                     int64_t width, uint64_t key, double gamma, int seeding,
                     int32_t *green_counts, double *z)
{
    uint64_t threshold = oracle_threshold(gamma);
    int64_t T = L > width ? L - width : 0;
    for (int64_t n = 0; n < N; ++n) {
        const int32_t *row = tokens + n * row_stride;
        int64_t count = 0;
        for (int64_t i = width; i < L; ++i)
            count += oracle_is_green_w(key, row + i - width, width, (uint32_t)row[i], threshold,
                                       seeding);
        green_counts[n] = (int32_t)count;
        z[n] = oracle_z_score(count, T, gamma);
    }
}

void oracle_seed_w_many(uint64_t key, const int32_t *context, int64_t width, const int32_t *cand,
                        int64_t n, int seeding, uint64_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_seed_w(key, context + i * width, width, (uint32_t)cand[i], seeding);
}

void oracle_is_green_w_many(uint64_t key, const int32_t *context, int64_t width,
                            const int32_t *cand, int64_t n, double gamma, int seeding, uint8_t *out)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t i = 0; i < n; ++i)
        out[i] = (uint8_t)oracle_is_green_w(key, context + i * width, width, (uint32_t)cand[i],
                                            threshold, seeding);
}

/* ------------------------------------------------------------------------- */
/* Greedy decoding of the watermarked logits (Eq. 2 followed by argmax): the   */
/* index of the largest watermarked logit per row.  Ties go to the smallest    */
/* index, a NaN counts as larger than any number (the first NaN wins), and     */
/* -0 equals +0.  The value returned is the watermarked logit at that index    */
/* (bf16 widened exactly to fp32).                                             */
/* ------------------------------------------------------------------------- */

static void argmax_update(float value, int64_t v, float *best, int64_t *best_v, int *best_nan)
{
    if (*best_nan) return;
    if (isnan(value)) {
        *best = value; *best_v = v; *best_nan = 1;
        return;
    }
    if (*best_v < 0 || value > *best) { *best = value; *best_v = v; }
}

void oracle_watermark_argmax_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, int32_t *tokens,
                                   float *values)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        float best = 0.0f; int64_t best_v = -1; int best_nan = 0;
        for (int64_t v = 0; v < V; ++v) {
            float l = logits[b * row_stride + v];
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding))
                l = oracle_bias_f32(l, delta);
            argmax_update(l, v, &best, &best_v, &best_nan);
        }
        tokens[b] = (int32_t)best_v;
        values[b] = best;
    }
}

void oracle_watermark_argmax_bf16_w(const uint16_t *logits, int64_t B, int64_t V,
                                    int64_t row_stride, const int32_t *context, int64_t width,
                                    uint64_t key, double gamma, float delta, int seeding,
                                    int32_t *tokens, float *values)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        float best = 0.0f; int64_t best_v = -1; int best_nan = 0;
        for (int64_t v = 0; v < V; ++v) {
            uint16_t l = logits[b * row_stride + v];
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding))
                l = oracle_bias_bf16(l, delta);
            argmax_update(f32_from_bits((uint32_t)l << 16), v, &best, &best_v, &best_nan);
        }
        tokens[b] = (int32_t)best_v;
        values[b] = best;
    }
}

/* ------------------------------------------------------------------------- */
/* Watermark restricted to candidate tokens: SBW-ss of the scheme table       */
/* (Sec. 4), the width-4 self-salt watermark applied to the top-40 candidates */
/* of a step only, the rest of the vocabulary left unbiased.  Row b's         */
/* candidates are cand[b*k .. b*k+k-1] (any order).  A candidate id outside   */
/* [0, V) is ignored and a repeated id is biased once; every other logit      */
/* keeps its bits.                                                            */
/* ------------------------------------------------------------------------- */

static int first_valid_candidate(const int32_t *row_cand, int64_t j, int64_t V)
{
    if (row_cand[j] < 0 || (int64_t)row_cand[j] >= V) return 0;
    for (int64_t i = 0; i < j; ++i)
        if (row_cand[i] == row_cand[j]) return 0;
    return 1;
}

void oracle_watermark_candidates_f32_w(float *logits, int64_t B, int64_t V, int64_t row_stride,
                                       const int32_t *cand, int64_t k, const int32_t *context,
                                       int64_t width, uint64_t key, double gamma, float delta,
                                       int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t j = 0; j < k; ++j) {
            if (!first_valid_candidate(cand + b * k, j, V)) continue;
            uint32_t v = (uint32_t)cand[b * k + j];
            if (oracle_is_green_w(key, context + b * width, width, v, threshold, seeding)) {
                float *l = &logits[b * row_stride + v];
                *l = oracle_bias_f32(*l, delta);
            }
        }
}

void oracle_watermark_candidates_bf16_w(uint16_t *logits, int64_t B, int64_t V, int64_t row_stride,
                                        const int32_t *cand, int64_t k, const int32_t *context,
                                        int64_t width, uint64_t key, double gamma, float delta,
                                        int seeding)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t j = 0; j < k; ++j) {
            if (!first_valid_candidate(cand + b * k, j, V)) continue;
            uint32_t v = (uint32_t)cand[b * k + j];
            if (oracle_is_green_w(key, context + b * width, width, v, threshold, seeding)) {
                uint16_t *l = &logits[b * row_stride + v];
                *l = oracle_bias_bf16(*l, delta);
            }
        }
}

/* ------------------------------------------------------------------------- */
/* Detection with per-sequence lengths and, optionally, each distinct n-gram  */
/* scored once.  Sequence n holds len_n = lengths[n] tokens (clamped to       */
/* [0, L]; all L when lengths is NULL) and positions width..len_n-1 are        */
/* scored under the width tokens before each, as in oracle_detect_w.  With    */
/* ignore_repeated, a position whose (width+1)-gram (its window and itself)   */
/* already occurred at an earlier scored position of the sequence is left     */
/* out of both T and the green count; a repeat has the same colour, so only   */
/* the number of trials changes.  z as in Sec. 3 with that T.                 */
/* ------------------------------------------------------------------------- */

static int same_ngram(const int32_t *seq, int64_t a, int64_t b, int64_t width)
{
    for (int64_t k = 0; k <= width; ++k)
        if (seq[a - width + k] != seq[b - width + k]) return 0;
    return 1;
}

void oracle_detect_ex(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                      const int32_t *lengths, int64_t width, uint64_t key, double gamma,
                      int seeding, int ignore_repeated, int32_t *green_counts, int32_t *scored,
                      double *z)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t n = 0; n < N; ++n) {
        const int32_t *seq = tokens + n * row_stride;
        int64_t len = L;
        if (lengths != 0) {
            len = lengths[n];
            if (len < 0) len = 0;
            if (len > L) len = L;
        }
        int64_t green = 0, T = 0;
        for (int64_t i = width; i < len; ++i) {
            if (ignore_repeated) {
                int seen = 0;
                for (int64_t j = width; j < i && !seen; ++j) seen = same_ngram(seq, j, i, width);
                if (seen) continue;
            }
            ++T;
            green += oracle_is_green_w(key, seq + i - width, width, (uint32_t)seq[i], threshold,
                                       seeding);
        }
        green_counts[n] = (int32_t)green;
        if (scored != 0) scored[n] = (int32_t)T;
        z[n] = oracle_z_score(green, T, gamma);
    }
}

/* ------------------------------------------------------------------------- */
/* Sampling from the watermarked distribution by the Gumbel-max trick: the    */
/* token argmax_v (l'_v / T + G_v) with G_v i.i.d. standard Gumbel is a draw  */
/* from softmax(l' / T), l' the watermarked logits of Eq. 2.  G_v is derived  */
/* from a caller-given seed per row through the same counter-based stream as  */
/* the watermark: u = ((CBRNG(v, seed) >> 9) + 1/2) * 2^-23, exact in fp32   */
/* and strictly inside (0, 1), G = -log(-log(u)).                             */
/*                                                                            */
/* The logarithm is computed from fp32 adds, multiplies and one divide, each  */
/* rounded once, in a fixed order, so every IEEE-754 implementation returns   */
/* the same bits: x = 2^e m with m in [sqrt(1/2), sqrt(2)), s = (m-1)/(m+1),  */
/* log m = 2 (s + s^3/3 + s^5/5 + s^7/7 + s^9/9) (the atanh series; |s| <=    */
/* 0.172, so the next term is below 2^-30), log x = e ln 2 + log m.  Valid    */
/* for finite normal x > 0, which is all it is given here.                    */
/* ------------------------------------------------------------------------- */

float oracle_sample_log(float x)
{
    uint32_t b = bits_from_f32(x);
    int e = (int)((b >> 23) & 0xFFu) - 127;
    float m = f32_from_bits((b & 0x007FFFFFu) | 0x3F800000u);    /* [1, 2) */
    if (m > 1.41421356f) {       /* to [sqrt(1/2), sqrt(2)): halving is exact */
        m = m * 0.5f;
        e = e + 1;
    }
    float s = (m - 1.0f) / (m + 1.0f);
    float s2 = s * s;
    float poly = 1.0f / 9.0f;
    poly = 1.0f / 7.0f + s2 * poly;
    poly = 1.0f / 5.0f + s2 * poly;
    poly = 1.0f / 3.0f + s2 * poly;
    poly = s + (s * s2) * poly;
    return (float)e * 0.693147180559945309f + 2.0f * poly;
}

float oracle_gumbel_of_draw(uint32_t x)
{
    float u = ((float)(x >> 9) + 0.5f) * 1.1920928955078125e-7f;   /* 2^-23 */
    return -oracle_sample_log(-oracle_sample_log(u));
}

float oracle_gumbel(uint32_t v, uint64_t seed)
{
    return oracle_gumbel_of_draw(oracle_cbrng(v, seed));
}

void oracle_watermark_sample_f32_w(const float *logits, int64_t B, int64_t V, int64_t row_stride,
                                   const int32_t *context, int64_t width, uint64_t key,
                                   double gamma, float delta, int seeding, const uint64_t *seeds,
                                   float inv_temperature, int32_t *tokens, float *scores)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        float best = 0.0f; int64_t best_v = -1; int best_nan = 0;
        for (int64_t v = 0; v < V; ++v) {
            float l = logits[b * row_stride + v];
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding))
                l = oracle_bias_f32(l, delta);
            float score = l * inv_temperature + oracle_gumbel((uint32_t)v, seeds[b]);
            argmax_update(score, v, &best, &best_v, &best_nan);
        }
        tokens[b] = (int32_t)best_v;
        scores[b] = best;
    }
}

void oracle_watermark_sample_bf16_w(const uint16_t *logits, int64_t B, int64_t V,
                                    int64_t row_stride, const int32_t *context, int64_t width,
                                    uint64_t key, double gamma, float delta, int seeding,
                                    const uint64_t *seeds, float inv_temperature, int32_t *tokens,
                                    float *scores)
{
    uint64_t threshold = oracle_threshold(gamma);
    for (int64_t b = 0; b < B; ++b) {
        float best = 0.0f; int64_t best_v = -1; int best_nan = 0;
        for (int64_t v = 0; v < V; ++v) {
            uint16_t l = logits[b * row_stride + v];
            if (oracle_is_green_w(key, context + b * width, width, (uint32_t)v, threshold, seeding))
                l = oracle_bias_bf16(l, delta);
            float score = f32_from_bits((uint32_t)l << 16) * inv_temperature +
                          oracle_gumbel((uint32_t)v, seeds[b]);
            argmax_update(score, v, &best, &best_v, &best_nan);
        }
        tokens[b] = (int32_t)best_v;
        scores[b] = best;
    }
}

void oracle_sample_log_many(const float *x, int64_t n, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_sample_log(x[i]);
}

void oracle_gumbel_many(const uint32_t *v, const uint64_t *seed, int64_t n, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_gumbel(v[i], seed[i]);
}

void oracle_gumbel_of_draws(const uint32_t *x, int64_t n, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_gumbel_of_draw(x[i]);
}
