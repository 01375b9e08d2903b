/*
 * sbw.h -- C ABI of libsbw, the MI355X (gfx950) hot path of Stateless Bernoulli
 * Watermarking ("Flip, Don't Shuffle", arXiv 2609.03844).
 *
 * Operations, each hand-written HIP kernels launched on the caller's stream:
 *
 *   watermark  For every row b of a decode batch and every token v of the
 *              vocabulary: derive the seed r from the row's previous token (or
 *              window of tokens; and, for self-salt, from v), draw x = CBRNG(v, r),
 *              and add delta to the logit when x < gamma (Sec. 2.2, Eq. 1 and
 *              Eq. 2; full-vocabulary self-salt, Sec. 5.2).  In place, one read and
 *              one write per logit.
 *   watermark_argmax     greedy decoding fused with the watermark: the index of
 *              the largest watermarked logit per row, the logits read once;
 *              watermark_argmax_noalloc the same for callers that cannot allocate
 *              (its scratch in a static device array).
 *   watermark_sample     sampling fused with the watermark (Gumbel-max).
 *   watermark_candidates the watermark on caller-given candidate ids only (the
 *              top-k self-salt scheme of Sec. 4).
 *   watermark_shard, watermark_argmax_shard, watermark_sample_shard
 *              the three logits calls on one slice of the vocabulary (a tensor-
 *              parallel LM head), column c being token v_offset + c.
 *   green_mask the green lists as bit sets (a parity and debugging aid).
 *   detect     For every sequence: count the positions whose token is green
 *              under the seed of the token(s) before it (O(1) per token, Sec. 2.2)
 *              and return the count W and z = (W - T gamma)/sqrt(T gamma (1-gamma))
 *              with T = L - 1 (Sec. 3); detect_window and detect_ex for windows,
 *              per-sequence lengths and repeated n-grams.
 *
 * Definitions fixed by this library where the paper leaves them open:
 *   CBRNG(v, r)   the v-th 32-bit output of the Philox4x32-10 stream keyed by r:
 *                 word (v mod 4) of Philox4x32-10(key = (lo32 r, hi32 r),
 *                 counter = (floor(v/4), 0, 0, 0))  (Sec. 2.2).
 *   x < gamma     x < ceil(gamma * 2^32), the exact comparison x * 2^-32 < gamma.
 *   context seed  r = key * p mod 2^64, p = previous token as uint32
 *                 ("additive" PRF of width 1, scheme table of App. D).
 *   self-salt     r = min_u64(key*J(p)*J(v), key*J(v)*J(v)) mod 2^64, J = Robert
 *                 Jenkins' 32-bit integer hash (Sec. 2.3), unsigned minimum
 *                 ("anchored minhash" over {p, v} anchored on v, App. D).
 *   bias          fp32: l + delta, one fp32 add rounded to nearest even.
 *                 bf16: round-to-nearest-even bf16 of (fp32(l) + delta); NaN
 *                 stays NaN.  Tokens not in the green list keep their bits.
 *
 * Conventions shared by every entry point:
 *   - Buffers belong to the caller.  Device pointers are HIP device (or managed)
 *     memory of the current device; they are not checked (a host pointer makes
 *     the kernel fault).  The library allocates nothing, on host or device
 *     (App. E, memory).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and the
 *     call returns without synchronising the host.  Functions hold no global
 *     mutable state and are reentrant, except sbw_watermark_argmax_noalloc, whose
 *     scratch array is shared by all of its calls on a device.
 *   - All arguments are checked on the host before any HIP call, so an error
 *     return means nothing was enqueued.  Token values are not checked (that
 *     would need a device read): every definition holds for any 32-bit pattern.
 *   - Empty work (B, V, N == 0) returns SBW_OK without a HIP call.
 *   - SBW_ERR_NO_DEVICE: no usable HIP device.  SBW_ERR_HIP: a HIP call or the
 *     kernel launch failed; sbw_last_hip_error() then names the HIP error of the
 *     calling thread.
 */
#ifndef SBW_H
#define SBW_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* In C++ the enumerations have the fixed underlying type int32_t, so that every value a
 * C caller can pass is a value of the type (the library answers an unknown one with
 * SBW_ERR_UNSUPPORTED); in C they are plain enumerations of the same size. */
#ifdef __cplusplus
#define SBW_ENUM_TYPE : int32_t
#else
#define SBW_ENUM_TYPE
#endif

typedef enum SBW_ENUM_TYPE {
    SBW_SEED_CONTEXT = 0,   /* seed from the previous token only          */
    SBW_SEED_SELF_SALT = 1  /* seed from the previous token and candidate */
} sbw_seeding_t;

typedef enum SBW_ENUM_TYPE {
    SBW_F32 = 0,            /* IEEE binary32 logits                        */
    SBW_BF16 = 1            /* bfloat16 logits (upper half of binary32)    */
} sbw_dtype_t;

typedef enum SBW_ENUM_TYPE {
    SBW_OK = 0,
    SBW_ERR_INVALID_ARG = 1, /* null pointer, negative size, stride too small */
    SBW_ERR_GAMMA = 2,       /* gamma outside the allowed range              */
    SBW_ERR_DELTA = 3,       /* delta not finite                            */
    SBW_ERR_UNSUPPORTED = 4, /* unknown enum value, or sizes beyond limits   */
    SBW_ERR_NO_DEVICE = 5,   /* no HIP device                                */
    SBW_ERR_HIP = 6          /* HIP runtime or launch error                  */
} sbw_status_t;

/*
 * sbw_watermark -- bias the green tokens of every row, in place
 * (Sec. 2.2, Eq. 1 and Eq. 2; full-vocabulary self-salt, Sec. 5.2).
 *
 *   logits       device, [B, row_stride] elements of `dtype`; element (b, v) is
 *                logits[b * row_stride + v] for b < B, v < V.  Read and written.
 *                Elements with v >= V are neither read nor written.
 *   dtype        SBW_F32 or SBW_BF16.
 *   B, V         rows and vocabulary size; 0 is a no-op.  V < 2^32 (token ids are
 *                32-bit), else SBW_ERR_UNSUPPORTED.
 *   row_stride   elements between row starts, >= V.
 *   prev_tokens  device, [B] int32: the token generated before this step, per row.
 *   key          the 64-bit watermark key.
 *   gamma        green-list fraction, 0 <= gamma <= 1 (0: nothing is green, the
 *                call is a no-op; 1: everything is green).  Else SBW_ERR_GAMMA.
 *   delta        bias added to green logits; must be finite, else SBW_ERR_DELTA.
 *   seeding      SBW_SEED_CONTEXT or SBW_SEED_SELF_SALT.
 *   stream       hipStream_t to enqueue on.
 *
 * Rows whose start is 16-byte aligned take 128-bit loads and stores; other
 * layouts are correct but slower.
 */
sbw_status_t sbw_watermark(void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                           int64_t row_stride, const int32_t *prev_tokens, uint64_t key,
                           double gamma, float delta, sbw_seeding_t seeding, void *stream);

/*
 * sbw_green_mask -- the green list G_t of every row as a bit set (Sec. 2.2, Eq. 1).
 * A parity and debugging aid: the watermark never materialises it.
 *
 *   bits         device, [B, ceil(V/32)] uint32, written: bit (v % 32) of word
 *                bits[b * ceil(V/32) + v / 32] is 1 iff v is green in row b.
 *                Bits for v >= V in the last word of a row are 0.
 *   B, V, prev_tokens, key, seeding   as for sbw_watermark.
 *   gamma        0 <= gamma <= 1, else SBW_ERR_GAMMA.
 */
sbw_status_t sbw_green_mask(uint32_t *bits, int64_t B, int64_t V, const int32_t *prev_tokens,
                            uint64_t key, double gamma, sbw_seeding_t seeding, void *stream);

/*
 * sbw_detect -- green count and z-score of every sequence (Sec. 2.2, O(1)
 * membership per token; Sec. 3, z-score).
 *
 *   tokens       device, [N, row_stride] int32; sequence n is tokens[n*row_stride
 *                + i], i < L.  May be NULL when L == 0.
 *   N, L         sequences and tokens per sequence; N == 0 is a no-op.  Positions
 *                1..L-1 are scored, each under the seed of the token before it,
 *                so T = L - 1; for L < 2, T = 0, the count is 0 and z is NaN.
 *   row_stride   elements between sequence starts, >= L.
 *   key, seeding as for sbw_watermark.
 *   gamma        0 < gamma < 1 (the z-score is undefined otherwise), else
 *                SBW_ERR_GAMMA.
 *   green_counts device, [N] int32, written: W per sequence.
 *   z            device, [N] double, written: (W - T*gamma) / sqrt(T*gamma*(1-gamma)),
 *                evaluated in binary64 in that order.
 *   L is limited to 2^31 - 1 (SBW_ERR_UNSUPPORTED beyond).
 */
sbw_status_t sbw_detect(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                        uint64_t key, double gamma, sbw_seeding_t seeding,
                        int32_t *green_counts, double *z, void *stream);

/*
 * Context windows of width h (the full-vocabulary schemes SBW-4 and SBW-ss-V of
 * the paper's scheme table and isolated benchmark, App. D and E).  The seed of a
 * step is derived from the h tokens before it:
 *   context seeding  r = key * (p_1 + ... + p_h) mod 2^64   ("additive" PRF)
 *   self-salt        r = min_u64( min_i key*J(p_i)*J(v), key*J(v)*J(v) )
 *                    ("anchored minhash" over the window and the candidate v)
 * Both are symmetric in the window.  Width 1 gives exactly sbw_watermark,
 * sbw_green_mask and sbw_detect, which are these calls with width = 1.
 *
 *   context      device, [B, width] int32 row-major: row b's window is
 *                context[b*width .. b*width + width-1] (any order).
 *   width        1 <= width <= 8; width < 1 is SBW_ERR_INVALID_ARG, width > 8
 *                SBW_ERR_UNSUPPORTED.
 * Other arguments, layouts and errors as for the width-1 calls.
 */
sbw_status_t sbw_watermark_window(void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t *context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  void *stream);

sbw_status_t sbw_green_mask_window(uint32_t *bits, int64_t B, int64_t V, const int32_t *context,
                                   int64_t width, uint64_t key, double gamma,
                                   sbw_seeding_t seeding, void *stream);

/*
 * Windowed detection: position i (width <= i < L) is scored under the window
 * tokens[n*row_stride + i-width .. i-1], so T = L - width; for L <= width the
 * count is 0 and z is NaN.
 */
sbw_status_t sbw_detect_window(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                               int64_t width, uint64_t key, double gamma, sbw_seeding_t seeding,
                               int32_t *green_counts, double *z, void *stream);

/* Flags of sbw_detect_ex. */
typedef enum SBW_ENUM_TYPE {
    SBW_DETECT_IGNORE_REPEATED = 1   /* score each distinct (width+1)-gram once */
} sbw_detect_flags_t;

/*
 * sbw_detect_ex -- detection for a batch of texts of different lengths, optionally
 * scoring every distinct n-gram once (a production extension of the z-test of
 * Sec. 3; the paper scores every position and fixes neither rule).
 *
 *   tokens, N, L, row_stride, width, key, gamma, seeding
 *                as for sbw_detect_window; L is the longest length (row capacity).
 *   lengths      device, [N] int32 or NULL: sequence n holds lengths[n] tokens,
 *                clamped to [0, L] (all L when NULL).  Positions width..len-1 are
 *                scored, T = max(len - width, 0).
 *   flags        0 or SBW_DETECT_IGNORE_REPEATED: then a position whose window and
 *                token (its (width+1)-gram) already occurred at an earlier scored
 *                position of the same sequence is left out of T and of the green
 *                count (a repeat has the same colour).  Supported for
 *                L - width <= 4096 (else SBW_ERR_UNSUPPORTED); other bits are
 *                SBW_ERR_UNSUPPORTED.
 *   green_counts device, [N] int32, written.
 *   scored       device, [N] int32 or NULL: T of each sequence, written.
 *   z            device, [N] double, written; NaN when T == 0.
 * One kernel on `stream`: one wavefront per sequence, or, with the repeat rule, one
 * workgroup per sequence with an LDS hash set (no global memory is allocated).
 */
sbw_status_t sbw_detect_ex(const int32_t *tokens, int64_t N, int64_t L, int64_t row_stride,
                           const int32_t *lengths, int64_t width, uint64_t key, double gamma,
                           sbw_seeding_t seeding, uint32_t flags, int32_t *green_counts,
                           int32_t *scored, double *z, void *stream);

/*
 * sbw_watermark_candidates -- the watermark restricted to given candidate tokens:
 * SBW-ss of the paper's scheme table (Sec. 4; self-salt, width 4, top-40
 * candidates), where only the top-k candidates of a step are tested and biased and
 * the rest of the vocabulary keeps its logits.  The caller's sampler supplies the
 * candidates (for example its top-k); membership and bias are as for
 * sbw_watermark_window with the same window, so a candidate is biased exactly when
 * the full-vocabulary watermark would bias it.
 *
 *   logits, dtype, B, V, row_stride, context, width, key, gamma, delta, seeding
 *                as for sbw_watermark_window (logits mutated in place).
 *   candidates   device, [B, k] int32 row-major: row b's candidate token ids, in any
 *                order.  An id outside [0, V) is ignored; an id repeated within a
 *                row is biased once.
 *   k            candidates per row, 0 <= k <= 1024 (k > 1024: SBW_ERR_UNSUPPORTED;
 *                k < 0: SBW_ERR_INVALID_ARG; k == 0: no-op).
 * One kernel on `stream` (one workgroup per row); nothing is allocated.
 */
sbw_status_t sbw_watermark_candidates(void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                      int64_t row_stride, const int32_t *candidates, int64_t k,
                                      const int32_t *context, int64_t width, uint64_t key,
                                      double gamma, float delta, sbw_seeding_t seeding,
                                      void *stream);

/*
 * sbw_watermark_argmax -- greedy decoding fused with the watermark: for every row,
 * the index of the largest watermarked logit (Eq. 2 applied on the fly; the logits
 * are only read, never written).  One read of each logit instead of a read and a
 * write plus a separate argmax pass.  (A decoding epilogue of the paper's logits
 * processor, Sec. 5.1, fused into the watermark pass.)
 *
 *   logits, dtype, B, V, row_stride, context, width, key, gamma, delta, seeding
 *                as for sbw_watermark_window, except that logits is read-only and
 *                V == 0 with B > 0 is SBW_ERR_INVALID_ARG (no token to choose).
 *   tokens       device, [B] int32, written: the chosen token of each row.  Among
 *                equal maxima the smallest index wins; a NaN counts as larger than
 *                any number (the first NaN wins); -0 and +0 are equal.
 *   values       device, [B] float, written (may be NULL): the watermarked logit at
 *                the chosen index (bf16 logits widened exactly to fp32).
 *   workspace    device, at least sbw_watermark_argmax_workspace(B, V) uint64
 *                elements, caller-owned scratch (partial results per row segment);
 *                its contents on entry do not matter and are undefined on return.
 *                Calls that share a workspace must be ordered (same stream);
 *                concurrent calls race.
 * Enqueues two kernels on `stream` (the fused pass, then a per-row read-out) and no
 * memset, so the call can be captured in a HIP graph.
 */
sbw_status_t sbw_watermark_argmax(const void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t *context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  int32_t *tokens, float *values, uint64_t *workspace,
                                  void *stream);

/*
 * sbw_watermark_sample -- sampling fused with the watermark: for every row, one draw
 * from softmax(l' * inv_temperature), l' the watermarked logits (Eq. 2), by the
 * Gumbel-max trick: the token maximising l'_v * inv_temperature + G_v, with the
 * noise G_v = -log(-log(u_v)), u_v = ((CBRNG(v, seeds[b]) >> 9) + 1/2) * 2^-23 (the
 * watermark's counter-based stream keyed by the row's seed).  The logarithm is the
 * atanh series on the reduced mantissa in fp32 adds, multiplies and one divide, in a
 * fixed order, so the draw is reproducible bit for bit (a decoding epilogue of the
 * logits processor, Sec. 5.1; the paper leaves sampling to the serving stack).
 *
 *   logits, dtype, B, V, row_stride, context, width, key, gamma, delta, seeding
 *                as for sbw_watermark_argmax (logits only read).
 *   seeds        device, [B] uint64: the noise seed of each row; draws with equal
 *                seeds and inputs are equal.
 *   inv_temperature  1/T, finite and > 0 (else SBW_ERR_INVALID_ARG).
 *   tokens       device, [B] int32, written: the drawn token (ties and NaN as for
 *                sbw_watermark_argmax; a NaN logit always wins).
 *   scores       device, [B] float, written (may be NULL): the winning score
 *                l'_v * inv_temperature + G_v.
 *   workspace    as for sbw_watermark_argmax, same size.
 * Enqueues two kernels on `stream` and no memset (graph-capturable).
 */
sbw_status_t sbw_watermark_sample(const void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t *context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  const uint64_t *seeds, float inv_temperature, int32_t *tokens,
                                  float *scores, uint64_t *workspace, void *stream);

/* Workspace size, in uint64 elements, that sbw_watermark_argmax needs for B rows of
 * V logits: B * ceil(V / 2048) (0 when B or V is not positive). */
int64_t sbw_watermark_argmax_workspace(int64_t B, int64_t V);

/* Capacity, in uint64 elements, of the scratch array of sbw_watermark_argmax_noalloc
 * (2 MiB per device). */
#define SBW_NOALLOC_SCRATCH_ELEMS 262144

/*
 * sbw_watermark_argmax_noalloc -- sbw_watermark_argmax without a workspace argument,
 * for callers that cannot allocate device memory at all: code being captured into a
 * HIP graph, tight serving loops, harnesses that forbid hipMalloc.  The per-segment
 * partials go to a scratch array that the library holds in its own code object
 * (one copy per device, kept until the process ends); the call itself allocates
 * nothing, on host or device, and makes no hipMalloc or hipFree.
 *
 *   logits, dtype, B, V, row_stride, context, width, key, gamma, delta, seeding,
 *   tokens, values, stream   as for sbw_watermark_argmax, with the same results.
 *   Limit: sbw_watermark_argmax_workspace(B, V) <= SBW_NOALLOC_SCRATCH_ELEMS (for
 *   example B <= 3495 rows of 152064 logits), else SBW_ERR_UNSUPPORTED, before any
 *   HIP call.
 *   Sharing: every call on a device uses that device's one array, so calls that
 *   overlap in time on one device race (keep them on one stream, or ordered); calls on
 *   different devices do not interact.  Nothing needs to be cleared between calls.
 *   First call: the first call made on a device looks up the array's address on that
 *   device (hipGetSymbolAddress); make it outside graph capture.  Later calls can be
 *   captured.
 */
sbw_status_t sbw_watermark_argmax_noalloc(const void *logits, sbw_dtype_t dtype, int64_t B,
                                          int64_t V, int64_t row_stride, const int32_t *context,
                                          int64_t width, uint64_t key, double gamma, float delta,
                                          sbw_seeding_t seeding, int32_t *tokens, float *values,
                                          void *stream);

/*
 * Vocabulary shards.  A token's colour depends only on the row's seed and on its own
 * id (Sec. 2.2: membership is one CBRNG draw at counter v, with no list to build), and
 * so does its sampling noise.  A slice of the vocabulary can therefore be watermarked,
 * and its best token found, on its own: this is what a tensor-parallel LM head holds
 * on each device.  These calls treat column c of each row as token v_offset + c.
 *
 *   logits       device, [B, row_stride]: the shard's columns, V of them per row.
 *   v_offset     global id of column 0, >= 0 (else SBW_ERR_INVALID_ARG), with
 *                v_offset + V <= 2^32 (else SBW_ERR_UNSUPPORTED).
 *   tokens       (argmax, sample) written as global ids, v_offset + c (an id of 2^31
 *                or more comes back as its 32-bit pattern, as a negative int32).
 * Every other argument, layout and error as for the unsharded call, which is the
 * same call with v_offset = 0.  The rows of all shards of a vocabulary, put side by
 * side, are biased exactly as the full rows are.  For decoding, the full row's token
 * is the shards' winner with the largest value (or score), the smallest global id
 * among equal ones, a NaN above everything: the reduction the unsharded call makes
 * over its own segments.  Rows whose first id is not a multiple of 4 (fp32) or 8
 * (bf16) take the element-wise kernels, which give the same results.
 */
sbw_status_t sbw_watermark_shard(void *logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                 int64_t row_stride, const int32_t *context, int64_t width,
                                 int64_t v_offset, uint64_t key, double gamma, float delta,
                                 sbw_seeding_t seeding, void *stream);

sbw_status_t sbw_watermark_argmax_shard(const void *logits, sbw_dtype_t dtype, int64_t B,
                                        int64_t V, int64_t row_stride, const int32_t *context,
                                        int64_t width, int64_t v_offset, uint64_t key,
                                        double gamma, float delta, sbw_seeding_t seeding,
                                        int32_t *tokens, float *values, uint64_t *workspace,
                                        void *stream);

sbw_status_t sbw_watermark_sample_shard(const void *logits, sbw_dtype_t dtype, int64_t B,
                                        int64_t V, int64_t row_stride, const int32_t *context,
                                        int64_t width, int64_t v_offset, uint64_t key,
                                        double gamma, float delta, sbw_seeding_t seeding,
                                        const uint64_t *seeds, float inv_temperature,
                                        int32_t *tokens, float *scores, uint64_t *workspace,
                                        void *stream);

/* Static description of a status code (never NULL). */
const char *sbw_strerror(sbw_status_t status);

/* Name of the last HIP error seen by an sbw_* call on the calling thread, or
 * "hipSuccess".  Thread-local; not reset by later successful calls. */
const char *sbw_last_hip_error(void);

/* Library version string, "MAJOR.MINOR.PATCH". */
const char *sbw_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SBW_H */
