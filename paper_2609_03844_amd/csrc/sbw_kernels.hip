// HIP kernels and C ABI of libsbw (declared in include/sbw.h) for MI355X / gfx950.
//
// watermark   one streaming pass over the logits: each lane owns 16-byte vectors
//             of a row (4 fp32 or 8 bf16 logits), loads them, derives the green
//             decision in registers (seed, Philox4x32-10 draw, threshold compare)
//             and stores them back.  Row-uniform values (the window of previous
//             tokens, the context seed, key * J(p_i)) sit in scalar registers.
//             Context seeding shares one Philox block between the 4 tokens of a
//             counter; self-salt needs one block per token, and its workgroups
//             share each candidate's hash and self term across up to 4 rows.  Large
//             self-salt launches (window of one token) instead draw each
//             column's self-term block once per slab of 12, 8 or 6 rows and queue in
//             LDS only the pairs whose row term is the smaller one (about half).
// argmax      greedy decoding of the watermarked logits without writing them: one
//             read of each logit, a per-segment (value, index) partial, a read-out
//             kernel per row.  Colours are drawn only for logits that can still
//             reach the segment's maximum.
// candidates  the watermark restricted to caller-given candidate ids per row (the
//             top-k self-salt scheme): one workgroup per row.
// green_mask  one lane per 32-token word of the bit set.
// detect      one wavefront per sequence; each lane scores positions i, i+64, ...
//             and the wave counts green positions with a ballot + popcount.  With
//             repeated n-grams scored once: one workgroup per sequence and an LDS
//             hash set of first occurrences.
//
// The context window: row b of a watermark call sees the `width` tokens
// context[b*width .. b*width+width-1] (the tokens before the step); position i of a
// detected sequence sees tokens i-width .. i-1.  Width 1 is the previous token.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "sbw.h"
#include "sbw_device.hpp"

namespace sbw {
namespace {

// Launch-shape tuning knobs (compile-time; the defaults are the measured best).
#ifndef SBW_CONTEXT_UNROLL
#define SBW_CONTEXT_UNROLL 2   // 16-byte vectors per lane, context seeding (HBM-bound)
#endif
#ifndef SBW_CONTEXT_UNROLL_BF16
#define SBW_CONTEXT_UNROLL_BF16 2
#endif
#ifndef SBW_SELF_SALT_UNROLL
#define SBW_SELF_SALT_UNROLL 2 // 16-byte vectors per lane, self-salt fp32 (Philox-bound)
#endif
#ifndef SBW_SELF_SALT_UNROLL_BF16
#define SBW_SELF_SALT_UNROLL_BF16 1
#endif
// Self-salt rows per workgroup (sharing the candidate terms) are chosen per launch,
// for width 1 only (with a wider window the window terms dominate and sharing does
// not pay): the most rows, up to 4 for fp32 and 2 for bf16 (register pressure), that
// still leave SBW_SELF_SALT_MIN_GROUPS workgroups.
// A self-salt workgroup may also take several row groups (at most ..._GROUP_ITERS,
// while SBW_SELF_SALT_MIN_GROUPS workgroups remain), computing the candidate terms
// once, and load the next group while drawing the current one (..._PREFETCH).
#ifndef SBW_SELF_SALT_GROUP_ITERS
#define SBW_SELF_SALT_GROUP_ITERS 1
#endif
#ifndef SBW_SELF_SALT_PREFETCH
#define SBW_SELF_SALT_PREFETCH 0
#endif
#ifndef SBW_SELF_SALT_GROUP_ITERS_BF16
#define SBW_SELF_SALT_GROUP_ITERS_BF16 4
#endif
#ifndef SBW_SELF_SALT_PREFETCH_BF16
#define SBW_SELF_SALT_PREFETCH_BF16 1
#endif
// Self-salt, width 1 (fp32 and bf16): the split-term slab kernel with 12-row slabs when
// that makes at least SBW_SLAB12_MIN_GROUPS workgroups, else with 8-row, else with 6-row
// slabs when that makes at least SBW_SLAB_MIN_GROUPS (below that its long-lived waves
// leave the chip underfilled and the row-group kernel is faster).  12-row slabs need
// more workgroups than the others: with fewer than ~1.7 rounds of the ~1800 that fit
// at once, the last round's tail costs more than the shorter slabs' extra self terms.
// 0 = off.
#ifndef SBW_SELF_SALT_SLAB
#define SBW_SELF_SALT_SLAB 1
#endif
// Context seeding: launches of at least SBW_XCD_ROWS_MIN rows (a multiple of 8) and
// SBW_XCD_ROWS_MIN_BYTES of logits, more than the 256 MB Infinity Cache holds, give
// each XCD whole rows (fp32 B = 512 / 1024 of 152064: 1 / 3 % faster, bf16 B = 1024:
// 3 %; B = 256 even, B = 128 and bf16 B = 512 of 128256 up to 1 % slower).
#ifndef SBW_XCD_ROWS_MIN
#define SBW_XCD_ROWS_MIN 512
#endif
#ifndef SBW_XCD_ROWS_MIN_BYTES
#define SBW_XCD_ROWS_MIN_BYTES (int64_t{256} << 20)
#endif
#ifndef SBW_SLAB_MIN_GROUPS
#define SBW_SLAB_MIN_GROUPS 2000
#endif
#ifndef SBW_SLAB12_MIN_GROUPS
#define SBW_SLAB12_MIN_GROUPS 3000
#endif
#ifndef SBW_SELF_SALT_MIN_GROUPS
#define SBW_SELF_SALT_MIN_GROUPS 1024  // 2048 measured 5 % slower for B * V of 5-10 M logits
#endif

constexpr int kThreads = 256;            // 4 wavefronts of 64
constexpr int kMaxWidth = 8;             // longest context window
constexpr int kMidWidth = 4;             // windows of 2-4 (the paper's 4): own instantiations
constexpr int64_t kMaxGrid = 1ll << 20;  // blocks; grid-stride loops cover the rest
constexpr int64_t kMaxGridY = 65535;

// Native vector types (the non-temporal builtins take these, not HIP's float4/uint4).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename V>
__device__ __forceinline__ V stream_load(const V* p) { return __builtin_nontemporal_load(p); }
template <typename V>
__device__ __forceinline__ void stream_store(V* p, V v) { __builtin_nontemporal_store(v, p); }

// ---------------------------------------------------------------------------
// Seeds.  kW is the compile-time bound on the window width: 1 for the
// previous-token path, kMaxWidth for wider windows (runtime width <= kW).
// ---------------------------------------------------------------------------
template <int kW>
struct RowSeed {
  uint64_t key;        // the watermark key
  uint64_t seed;       // context seeding: key * (sum of the window)
  uint64_t kjp[kW];    // self-salt: key * J(p_i) for the window tokens
  int width;
};

template <int kSeeding, int kW>
__device__ __forceinline__ RowSeed<kW> row_seed(uint64_t key, const int32_t* window, int width) {
  RowSeed<kW> rs;
  rs.key = key;
  rs.width = width;
  rs.seed = 0u;
  if (kSeeding == kContext) {
    uint64_t sum = 0u;
    for (int i = 0; i < (kW == 1 ? 1 : width); ++i) sum += static_cast<uint32_t>(window[i]);
    rs.seed = key * sum;
  } else {
#pragma unroll
    for (int i = 0; i < kW; ++i)
      rs.kjp[i] = (kW == 1 || i < width)
                      ? key * static_cast<uint64_t>(jenkins32(static_cast<uint32_t>(window[i])))
                      : 0u;
  }
  return rs;
}

// Self-salt seed of candidate v: the minimum over the window and v itself of
// key*J(w)*J(v).  Split in two: the candidate's terms J(v) and key*J(v)*J(v), which
// do not depend on the row, then the row's minimum.
struct CandTerm {
  uint32_t jv;     // J(v)
  uint64_t self;   // key * J(v) * J(v)
};

__device__ __forceinline__ CandTerm cand_term(uint64_t key, uint32_t v) {
  const uint32_t jv = jenkins32(v);
  return CandTerm{jv, mul_64x64(key, wide_mul(jv, jv))};
}

// The self-salt seed of a candidate from its terms and the row's key*J(p_i).
template <int kW>
__device__ __forceinline__ uint64_t self_salt_seed_t(const RowSeed<kW>& rs, const CandTerm& t) {
  uint64_t best = t.self;
#pragma unroll
  for (int i = 0; i < kW; ++i) {
    if (kW == 1 || i < rs.width) {
      const uint64_t x = lane_mul_64x32(rs.kjp[i], t.jv);
      best = x < best ? x : best;
    }
  }
  return best;
}

template <int kW>
__device__ __forceinline__ uint64_t self_salt_seed_w(const RowSeed<kW>& rs, uint32_t v) {
  return self_salt_seed_t(rs, cand_term(rs.key, v));
}

template <int kSeeding, int kW>
__device__ __forceinline__ uint32_t draw(const RowSeed<kW>& rs, uint32_t v) {
  if (kSeeding == kContext) return cbrng(v, rs.seed);
  return cbrng(v, self_salt_seed_w(rs, v));
}

// ---------------------------------------------------------------------------
// Context-seeded watermark vectors: one row seed, so the tokens of a Philox block
// share it.  fp32: a vector is the 4 tokens 4j..4j+3, exactly the 4 words of the
// block at counter j.  bf16: the 8 tokens 8j..8j+7 = blocks 2j and 2j+1.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 bias_vec_context(f32x4 l, uint32_t j, uint64_t seed, uint32_t tm1,
                                                  float delta) {
  const Block blk = philox_block(j, key_of(seed));
  f32x4 o;
  o.x = bias_f32(l.x, delta, is_green(blk.w0, tm1));
  o.y = bias_f32(l.y, delta, is_green(blk.w1, tm1));
  o.z = bias_f32(l.z, delta, is_green(blk.w2, tm1));
  o.w = bias_f32(l.w, delta, is_green(blk.w3, tm1));
  return o;
}

__device__ __forceinline__ u32x4 bias_vec_context(u32x4 raw, uint32_t j, uint64_t seed, uint32_t tm1,
                                                  float delta) {
  const Key k = key_of(seed);
  const Block a = philox_block(2u * j, k);
  const Block b = philox_block(2u * j + 1u, k);
  const uint32_t x[8] = {a.w0, a.w1, a.w2, a.w3, b.w0, b.w1, b.w2, b.w3};
  const uint32_t in[4] = {raw.x, raw.y, raw.z, raw.w};
  uint32_t out[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    out[q] = bias_bf16x2(in[q], delta, is_green(x[2 * q], tm1), is_green(x[2 * q + 1], tm1));
  return u32x4{out[0], out[1], out[2], out[3]};
}

// One element of either dtype (row tails and unaligned rows).
__device__ __forceinline__ float bias_elem(float l, float d, bool g) { return bias_f32(l, d, g); }
__device__ __forceinline__ uint16_t bias_elem(uint16_t l, float d, bool g) {
  return bias_bf16(l, d, g);
}

// One token: column v of the row, token id vbase + v.
template <typename T, int kSeeding, int kW>
__device__ __forceinline__ void bias_one(T* row, uint32_t v, const RowSeed<kW>& rs, uint32_t tm1,
                                         float delta, uint32_t vbase) {
  const uint32_t x = draw<kSeeding>(rs, vbase + v);
  row[v] = bias_elem(row[v], delta, is_green(x, tm1));
}

// Context-seeded watermark for rows whose start is 16-byte aligned.  Grid: x = tile
// of kThreads * kU vectors within a row, y = row (grid-stride over rows beyond
// 65535).  Each lane issues its logits load before reading the row's window, so the
// scalar loads of the window overlap the HBM stream.  With xcd_rows (one row per y,
// B a multiple of 8) the workgroups are renumbered so that each of the 8 XCDs, which
// take workgroups in turn, streams whole rows: workgroup n goes to row
// 8 * (n / 8 / tiles) + n % 8, tile n / 8 % tiles.
template <typename T, int kU, int kW>
__global__ void __launch_bounds__(kThreads)
watermark_vec_kernel(T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                     const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                     float delta, uint32_t vbase, uint32_t xcd_rows) {
  using VecT = typename std::conditional<sizeof(T) == 4, f32x4, u32x4>::type;
  constexpr uint32_t kPer = 16u / sizeof(T);  // elements per 16-byte vector
  const uint32_t full = V / kPer;             // complete vectors in a row
  const uint32_t tail = V % kPer;
  const uint32_t jbase = vbase / kPer;        // vector index of the first column (vbase % 8 == 0)
  uint32_t first = blockIdx.x * (kThreads * kU);
  int64_t row0 = blockIdx.y;
  if (xcd_rows != 0u) {
    const uint32_t n = blockIdx.y * gridDim.x + blockIdx.x;
    const uint32_t q = n >> 3;
    row0 = static_cast<int64_t>(q / gridDim.x) * 8 + (n & 7u);
    first = (q % gridDim.x) * (kThreads * kU);
  }
  for (int64_t row = row0; row < B; row += gridDim.y) {
    T* row_ptr = logits + row * row_stride;
    VecT* vec = reinterpret_cast<VecT*>(row_ptr);
    const int32_t* window = context + row * width;
    VecT buf[kU];
    if (first + kThreads * kU <= full) {
      // Whole tile inside the row: no per-vector guards, all loads in flight at once.
#pragma unroll
      for (int u = 0; u < kU; ++u) buf[u] = stream_load(vec + first + u * kThreads + threadIdx.x);
      const RowSeed<kW> rs = row_seed<kContext, kW>(key, window, width);
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const uint32_t j = first + u * kThreads + threadIdx.x;
        stream_store(vec + j, bias_vec_context(buf[u], j + jbase, rs.seed, tm1, delta));
      }
    } else {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const uint32_t j = first + u * kThreads + threadIdx.x;
        if (j < full) buf[u] = stream_load(vec + j);
      }
      const RowSeed<kW> rs = row_seed<kContext, kW>(key, window, width);
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const uint32_t j = first + u * kThreads + threadIdx.x;
        if (j < full) stream_store(vec + j, bias_vec_context(buf[u], j + jbase, rs.seed, tm1, delta));
      }
      // The partial vector at the end of the row, element by element, by lane 0 of
      // the tile that covers vector index `full`.
      if (tail != 0u && threadIdx.x == 0 && full >= first &&
          full - first < static_cast<uint32_t>(kThreads * kU)) {
        for (uint32_t e = 0; e < tail; ++e)
          bias_one<T, kContext>(row_ptr, full * kPer + e, rs, tm1, delta, vbase);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Self-salt watermark over kRows rows per workgroup.  The rows of a workgroup share
// their columns, so a candidate's J(v) and the row-independent term key*J(v)*J(v)
// of its seed are computed once per lane and reused for every row; the window terms
// key*J(p_i)*J(v), the minimum and the Philox draw are per row.
// ---------------------------------------------------------------------------
template <int kW>
__device__ __forceinline__ f32x4 bias_vec_terms(f32x4 l, uint32_t j, const CandTerm (&ct)[4],
                                                const RowSeed<kW>& rs, uint32_t tm1, float delta) {
  const uint32_t x0 = philox_block_lane<6>(j, key_of(self_salt_seed_t(rs, ct[0]))).w0;
  const uint32_t x1 = philox_block_lane<6>(j, key_of(self_salt_seed_t(rs, ct[1]))).w1;
  const uint32_t x2 = philox_block_lane<6>(j, key_of(self_salt_seed_t(rs, ct[2]))).w2;
  const uint32_t x3 = philox_block_lane<6>(j, key_of(self_salt_seed_t(rs, ct[3]))).w3;
  f32x4 o;
  o.x = bias_f32(l.x, delta, is_green(x0, tm1));
  o.y = bias_f32(l.y, delta, is_green(x1, tm1));
  o.z = bias_f32(l.z, delta, is_green(x2, tm1));
  o.w = bias_f32(l.w, delta, is_green(x3, tm1));
  return o;
}

template <int kW>
__device__ __forceinline__ u32x4 bias_vec_terms(u32x4 raw, uint32_t j, const CandTerm (&ct)[8],
                                                const RowSeed<kW>& rs, uint32_t tm1, float delta) {
  uint32_t x[8];
#pragma unroll
  for (int e = 0; e < 8; ++e)
    x[e] = block_word(philox_block_lane<6>(2u * j + static_cast<uint32_t>(e >> 2),
                                           key_of(self_salt_seed_t(rs, ct[e]))),
                      static_cast<uint32_t>(e & 3));
  const uint32_t in[4] = {raw.x, raw.y, raw.z, raw.w};
  uint32_t out[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)
    out[q] = bias_bf16x2(in[q], delta, is_green(x[2 * q], tm1), is_green(x[2 * q + 1], tm1));
  return u32x4{out[0], out[1], out[2], out[3]};
}

// Grid: x = tile of kThreads * kU vectors of a row, y = a slot that takes groups of
// kRows rows y, y + gridDim.y, ...  The candidate terms depend on the columns only, so
// a workgroup computes them once, while its first group's loads are in flight, and
// uses them for every group it takes.  With kPrefetch the next group's logits are
// loaded while the current group is drawn.
template <typename T, int kU, int kW, int kRows, bool kPrefetch>
__global__ void __launch_bounds__(kThreads)
watermark_ss_rows_kernel(T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                         const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                         float delta, uint32_t vbase) {
  using VecT = typename std::conditional<sizeof(T) == 4, f32x4, u32x4>::type;
  constexpr uint32_t kPer = 16u / sizeof(T);
  const uint32_t full = V / kPer;
  const uint32_t tail = V % kPer;
  const uint32_t first = blockIdx.x * (kThreads * kU);
  // the tile's first vector counted in token ids (vbase is a multiple of kPer)
  const uint32_t id_first = first + vbase / kPer;
  const bool whole = first + kThreads * kU <= full;
  const int64_t groups = (B + kRows - 1) / kRows;
  auto load_group = [&](VecT (&buf)[kRows][kU], int64_t g) {
    const int64_t row0 = g * kRows;
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      if (row0 + r < B) {
        const VecT* vec = reinterpret_cast<const VecT*>(logits + (row0 + r) * row_stride);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const uint32_t j = first + u * kThreads + threadIdx.x;
          if (whole || j < full) buf[r][u] = stream_load(vec + j);
        }
      }
    }
  };
  CandTerm ct[kU][kPer];
  auto draw_group = [&](const VecT (&buf)[kRows][kU], int64_t g) {
    const int64_t row0 = g * kRows;
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      if (row0 + r < B) {
        const int64_t row = row0 + r;
        T* row_ptr = logits + row * row_stride;
        VecT* vec = reinterpret_cast<VecT*>(row_ptr);
        const RowSeed<kW> rs = row_seed<kSelfSalt, kW>(key, context + row * width, width);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const uint32_t j = first + u * kThreads + threadIdx.x;
          if (whole || j < full)
            stream_store(vec + j, bias_vec_terms(buf[r][u], id_first + u * kThreads + threadIdx.x,
                                                 ct[u], rs, tm1, delta));
        }
        // the row's partial last vector, by lane 0 of the tile that covers it
        if (!whole && tail != 0u && threadIdx.x == 0 && full >= first &&
            full - first < static_cast<uint32_t>(kThreads * kU)) {
          for (uint32_t e = 0; e < tail; ++e)
            bias_one<T, kSelfSalt>(row_ptr, full * kPer + e, rs, tm1, delta, vbase);
        }
      }
    }
  };
  int64_t g = blockIdx.y;
  if (g >= groups) return;
  VecT buf0[kRows][kU];
  load_group(buf0, g);
#pragma unroll
  for (int u = 0; u < kU; ++u)
#pragma unroll
    for (uint32_t e = 0; e < kPer; ++e)
      ct[u][e] = cand_term(key, (id_first + u * kThreads + threadIdx.x) * kPer + e);
  if constexpr (!kPrefetch) {
    for (;;) {
      draw_group(buf0, g);
      g += gridDim.y;
      if (g >= groups) break;
      load_group(buf0, g);
    }
  } else {
    VecT buf1[kRows][kU];
    for (;;) {
      const int64_t g1 = g + gridDim.y;
      if (g1 < groups) load_group(buf1, g1);
      draw_group(buf0, g);
      if (g1 >= groups) break;
      const int64_t g2 = g1 + gridDim.y;
      if (g2 < groups) load_group(buf0, g2);
      draw_group(buf1, g1);
      if (g2 >= groups) break;
      g = g2;
    }
  }
}

// ---------------------------------------------------------------------------
// Self-salt watermark, fp32 or bf16, window of one token, by split terms over a slab
// of rows.  The seed of (row, v) is the smaller of the row term key*J(p)*J(v) and the
// self term key*J(v)*J(v) (Sec. 2.3 with the window {p, v}); the self term, and so
// the draw whenever it is the smaller one (about half of the pairs), is the same in
// every row.  A wave owns 64 16-byte vectors of a row (one per lane: 256 fp32 or 512
// bf16 columns) over a slab of up to kRows rows (12, or 8 or 6 for launches that
// taller slabs would leave with too few workgroups):
//  1. each lane draws its vector's self-term blocks (4 or 8) once and writes those
//     decisions into the slab's decision map (a byte per row and column, a lane's
//     columns in one word, or two for bf16) for every row;
//  2. one token position q of the vector at a time, the lanes whose row term is
//     smaller append (row term, map word, lane) to the wave's queue (ballot + mbcnt
//     give consecutive entries), and a queue holding 64 pairs is drained at once: 64
//     Philox draws side by side, each decision written over its map byte; the last
//     partial chunk is drained after the slab's last row;
//  3. each row's vector is biased from its map word and stored.
// The Philox counter and word are compile-time functions of q in every draw (q is a
// template argument), so each block keeps only the work its word needs.  Per logit this
// draws about 0.57 blocks instead of 1; the queueing costs about 9 instructions.
// ---------------------------------------------------------------------------
constexpr uint32_t kSlabQueue = 128;   // queue entries: fewer than 64 left + one row's 64
// Map words per row: one more than the lanes, so that the same lane's words in
// adjacent rows fall in different LDS banks.
constexpr uint32_t kSlabMapStride = 65;
constexpr int kSlabLoadRows = 4;       // rows whose logits are loaded together in step 3

// l + delta where bit `bit` of `bits` is set, l's own bits elsewhere: the bit widened
// to a full mask by a sign-extending field extract, then a bitwise select.
__device__ __forceinline__ float bias_bit(float l, float delta, uint32_t bits, int bit) {
  const uint32_t m = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(bits), bit, 1));
  return __uint_as_float(
      __builtin_amdgcn_bitop3_b32(m, __float_as_uint(l + delta), __float_as_uint(l), 0xCA));
}

template <int kQ>
__device__ __forceinline__ uint32_t word_of(const Block& b) {
  return kQ == 0 ? b.w0 : kQ == 1 ? b.w1 : kQ == 2 ? b.w2 : b.w3;
}

// A queued pair: the row term (the Philox key, two words), its map word and the lane
// that queued it; one 16-byte record, one address and one LDS operation each way.
typedef uint32_t SlabEntry __attribute__((ext_vector_type(4)));

// One wave's LDS: the queue, the decision map (kPer bytes per row and lane: the
// decisions of a lane's kPer tokens), and each row's key * J(p).
template <int kRows, int kPer>
struct SlabLds {
  SlabEntry queue[kSlabQueue];
  uint32_t map[kRows * kSlabMapStride * (kPer / 4)];
  alignas(16) uint64_t kjp[kRows + 2];  // two spares for the read-ahead
};

// Draws the first n (<= 64) queue entries of token position kE (of the kPer tokens
// of a lane's vector), one per lane, writes each decision over its map byte, and
// moves entries 64 .. pending-1 to the front.  Lanes past n read entries inside the
// queue and store nothing.
template <int kE, int kRows, int kPer>
__device__ __forceinline__ void slab_drain(SlabLds<kRows, kPer>& s, uint32_t n, uint32_t pending,
                                           uint32_t lane, uint32_t jid0, uint32_t tm1) {
  const SlabEntry e = s.queue[lane];
  SlabEntry e2;  // read and written back only where `move` holds
  const bool move = lane + 64u < pending;
  if (move) e2 = s.queue[lane + 64u];
  // the pair's token is kPer * (jid0 + lane that queued it) + kE: Philox counter
  // (kPer / 4) * (jid0 + lane) + kE / 4, word kE mod 4
  const uint32_t x = word_of<kE % 4>(philox_block_lane<6>(
      (kPer / 4) * (jid0 + e.w) + static_cast<uint32_t>(kE / 4), Key{e.x, e.y}));
  if (lane < n)
    reinterpret_cast<uint8_t*>(s.map)[kPer * e.z + kE] = static_cast<uint8_t>(is_green(x, tm1));
  if (move) s.queue[lane] = e2;
}

// Queues the pairs of one row and token position kE whose row term kjp * J(v) is
// below `bound`, and drains the queue when it holds 64.
template <int kE, int kRows, int kPer>
__device__ __forceinline__ void slab_enqueue(SlabLds<kRows, kPer>& s, uint32_t& pending, uint64_t kjp,
                                             uint32_t jv, uint64_t bound, uint32_t map_word,
                                             uint32_t lane, uint32_t jid0, uint32_t tm1) {
  const uint64_t t = lane_mul_64x32(kjp, jv);
  // the lanes with t < bound, as one wave mask (the compiler shares the compare
  // with the branch below)
  const uint64_t mask = __builtin_amdgcn_uicmpl(t, bound, 36 /* unsigned less than */);
  if (t < bound) {
    const uint32_t at = pending + __builtin_amdgcn_mbcnt_hi(
                                      static_cast<uint32_t>(mask >> 32),
                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
    s.queue[at] = SlabEntry{static_cast<uint32_t>(t), static_cast<uint32_t>(t >> 32), map_word, lane};
  }
  pending += static_cast<uint32_t>(__builtin_popcountll(mask));
  // LDS operations of one wave complete in order; the barriers only keep the
  // compiler from moving them across the passes.
  __builtin_amdgcn_wave_barrier();
  if (pending >= 64u) {
    slab_drain<kE, kRows, kPer>(s, 64u, pending, lane, jid0, tm1);
    pending -= 64u;
    __builtin_amdgcn_wave_barrier();
  }
}

// Token position kE over the rows of the slab: queue, drain at 64, drain the rest.
template <int kE, int kRows, int kPer>
__device__ __forceinline__ void slab_position(SlabLds<kRows, kPer>& s, int rows, uint32_t jv, uint64_t bound,
                                              uint32_t lane, uint32_t jid0, uint32_t tm1) {
  uint32_t pending = 0u;  // wave-uniform
  // four rows per iteration, their key * J(p) by two broadcast LDS reads of two rows
  // each, each pair read one pair ahead into the registers the pair before it has
  // just freed (entries past the last row are spares: read, never used)
  typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
  u64x2 a = *reinterpret_cast<const u64x2*>(&s.kjp[0]);
  int r = 0;
#pragma nounroll
  for (; r + 3 < rows; r += 4) {
    const u64x2 b = *reinterpret_cast<const u64x2*>(&s.kjp[r + 2]);
    const uint32_t w0 = static_cast<uint32_t>(r) * kSlabMapStride + lane;
    slab_enqueue<kE, kRows, kPer>(s, pending, a.x, jv, bound, w0, lane, jid0, tm1);
    slab_enqueue<kE, kRows, kPer>(s, pending, a.y, jv, bound, w0 + kSlabMapStride, lane, jid0, tm1);
    a = *reinterpret_cast<const u64x2*>(&s.kjp[r + 4]);
    slab_enqueue<kE, kRows, kPer>(s, pending, b.x, jv, bound, w0 + 2 * kSlabMapStride, lane, jid0, tm1);
    slab_enqueue<kE, kRows, kPer>(s, pending, b.y, jv, bound, w0 + 3 * kSlabMapStride, lane, jid0, tm1);
  }
  if (r + 1 < rows) {
    const uint32_t w0 = static_cast<uint32_t>(r) * kSlabMapStride + lane;
    slab_enqueue<kE, kRows, kPer>(s, pending, a.x, jv, bound, w0, lane, jid0, tm1);
    slab_enqueue<kE, kRows, kPer>(s, pending, a.y, jv, bound, w0 + kSlabMapStride, lane, jid0, tm1);
    r += 2;
    a = *reinterpret_cast<const u64x2*>(&s.kjp[r]);
  }
  if (r < rows)
    slab_enqueue<kE, kRows, kPer>(s, pending, a.x, jv, bound,
                                  static_cast<uint32_t>(r) * kSlabMapStride + lane, lane, jid0, tm1);
  if (pending != 0u) slab_drain<kE, kRows, kPer>(s, pending, pending, lane, jid0, tm1);
  __builtin_amdgcn_wave_barrier();
}

// The bias of a bf16 pair from its two map bytes (bits blo and bhi of the decision
// word d): one fp32 add each, one rounding, the non-green half's bits kept.
__device__ __forceinline__ uint32_t bias_pair_bits(uint32_t pair, float delta, uint32_t d, int blo,
                                                   int bhi) {
  const uint32_t mlo = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(d), blo, 1));
  const uint32_t mhi = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(d), bhi, 1));
  const uint32_t take = __builtin_amdgcn_bitop3_b32(0x0000FFFFu, mlo, mhi, 0xCA);
  const uint32_t biased = to_bf16x2(__uint_as_float(pair << 16) + delta,
                                    __uint_as_float(pair & 0xFFFF0000u) + delta);
  return __builtin_amdgcn_bitop3_b32(take, biased, pair, 0xCA);
}

// Step 3 of a row's vector: the bias from the row's kPer map bytes.
__device__ __forceinline__ f32x4 slab_bias(f32x4 o, float delta, const uint32_t (&d)[1]) {
  o.x = bias_bit(o.x, delta, d[0], 0);
  o.y = bias_bit(o.y, delta, d[0], 8);
  o.z = bias_bit(o.z, delta, d[0], 16);
  o.w = bias_bit(o.w, delta, d[0], 24);
  return o;
}
__device__ __forceinline__ u32x4 slab_bias(u32x4 o, float delta, const uint32_t (&d)[2]) {
  o.x = bias_pair_bits(o.x, delta, d[0], 0, 8);
  o.y = bias_pair_bits(o.y, delta, d[0], 16, 24);
  o.z = bias_pair_bits(o.z, delta, d[1], 0, 8);
  o.w = bias_pair_bits(o.w, delta, d[1], 16, 24);
  return o;
}

// The kPer token positions of a lane's vector, one after another.
template <int kE, int kRows, int kPer>
__device__ __forceinline__ void slab_positions(SlabLds<kRows, kPer>& s, int rows,
                                               const uint32_t (&jv)[kPer],
                                               const uint64_t (&bound)[kPer], uint32_t lane,
                                               uint32_t jid0, uint32_t tm1) {
  if constexpr (kE < kPer) {
    slab_position<kE, kRows, kPer>(s, rows, jv[kE], bound[kE], lane, jid0, tm1);
    slab_positions<kE + 1, kRows, kPer>(s, rows, jv, bound, lane, jid0, tm1);
  }
}

// Grid: x = tile of kThreads vectors (4 waves of 256 vectors), y = a slot taking the
// slabs y, y + gridDim.y, ... of kRows rows.  T: float (4 tokens a vector) or bf16
// bits (8).  Rows 16-byte aligned; vbase a multiple of the tokens per vector.
template <typename T, int kRows>
__global__ void __launch_bounds__(kThreads)
watermark_ss_slab_kernel(T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                         const int32_t* __restrict__ context, uint64_t key, uint32_t tm1,
                         float delta, uint32_t vbase) {
  using VecT = typename std::conditional<sizeof(T) == 4, f32x4, u32x4>::type;
  constexpr int kPer = 16 / sizeof(T);  // tokens a vector
  constexpr int kWords = kPer / 4;      // map words (and Philox counters) a vector
  __shared__ SlabLds<kRows, kPer> lds[kThreads / 64];
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  SlabLds<kRows, kPer>& s = lds[wave];
  const uint32_t full = V / kPer;
  const uint32_t tail = V % kPer;
  const uint32_t j0 = blockIdx.x * kThreads + wave * 64u;  // the wave's first vector
  const uint32_t j = j0 + lane;
  const bool active = j < full;
  const uint32_t jid0 = j0 + vbase / kPer;  // in token ids / kPer
  const uint32_t jid = jid0 + lane;
  // the lane's tokens: J(v), and the self term as the queueing bound (0, which no row
  // term is below, for a lane past the row's last whole vector)
  uint32_t jv[kPer];
  uint64_t bound[kPer];
  uint32_t self_word[kWords];
  {
    uint64_t self[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      jv[e] = jenkins32(jid * kPer + static_cast<uint32_t>(e));
      self[e] = mul_64x64(key, wide_mul(jv[e], jv[e]));
      bound[e] = active ? self[e] : 0u;
    }
#pragma unroll
    for (int w = 0; w < kWords; ++w) {
      const uint32_t c = jid * kWords + static_cast<uint32_t>(w);  // Philox counter
      self_word[w] =
          static_cast<uint32_t>(is_green(word_of<0>(philox_block_lane<6>(c, key_of(self[4 * w]))), tm1)) |
          static_cast<uint32_t>(is_green(word_of<1>(philox_block_lane<6>(c, key_of(self[4 * w + 1]))), tm1)) << 8 |
          static_cast<uint32_t>(is_green(word_of<2>(philox_block_lane<6>(c, key_of(self[4 * w + 2]))), tm1)) << 16 |
          static_cast<uint32_t>(is_green(word_of<3>(philox_block_lane<6>(c, key_of(self[4 * w + 3]))), tm1)) << 24;
    }
  }
  const int64_t slabs = (B + kRows - 1) / kRows;
  for (int64_t g = blockIdx.y; g < slabs; g += gridDim.y) {
    const int64_t row0 = g * kRows;
    const int rows = static_cast<int>(B - row0 < kRows ? B - row0 : kRows);
    // step 1: the self decisions for every row, and each row's key * J(p)
#pragma nounroll
    for (int r = 0; r < rows; ++r) {
#pragma unroll
      for (int w = 0; w < kWords; ++w)
        s.map[(static_cast<uint32_t>(r) * kSlabMapStride + lane) * kWords + w] = self_word[w];
    }
    if (lane < static_cast<uint32_t>(rows))
      s.kjp[lane] = key * static_cast<uint64_t>(jenkins32(static_cast<uint32_t>(context[row0 + lane])));
    __builtin_amdgcn_wave_barrier();
    // step 2: the pairs whose row term is smaller, one token position at a time
    slab_positions<0, kRows, kPer>(s, rows, jv, bound, lane, jid0, tm1);
    // step 3: bias and store, kSlabLoadRows rows' loads in flight at a time
    if (active) {
      for (int r0 = 0; r0 < rows; r0 += kSlabLoadRows) {
        VecT buf[kSlabLoadRows];
        uint32_t dec[kSlabLoadRows][kWords];
#pragma unroll
        for (int k = 0; k < kSlabLoadRows; ++k) {
          if (r0 + k < rows) {
            buf[k] = stream_load(reinterpret_cast<const VecT*>(logits + (row0 + r0 + k) * row_stride) + j);
#pragma unroll
            for (int w = 0; w < kWords; ++w)
              dec[k][w] = s.map[(static_cast<uint32_t>(r0 + k) * kSlabMapStride + lane) * kWords + w];
          }
        }
#pragma unroll
        for (int k = 0; k < kSlabLoadRows; ++k) {
          if (r0 + k < rows)
            stream_store(reinterpret_cast<VecT*>(logits + (row0 + r0 + k) * row_stride) + j,
                         slab_bias(buf[k], delta, dec[k]));
        }
      }
    }
    // the rows' partial last vector, by lane 0 of the wave that covers it
    if (tail != 0u && lane == 0u && full >= j0 && full - j0 < 64u) {
      for (int r = 0; r < rows; ++r) {
        const RowSeed<1> rs = row_seed<kSelfSalt, 1>(key, context + row0 + r, 1);
        for (uint32_t e = 0; e < tail; ++e)
          bias_one<T, kSelfSalt>(logits + (row0 + r) * row_stride, full * kPer + e, rs, tm1,
                                 delta, vbase);
      }
    }
    __builtin_amdgcn_wave_barrier();  // the next slab rewrites the map
  }
}

// Element-wise watermark for rows that are not 16-byte aligned.
template <typename T, int kSeeding, int kW>
__global__ void __launch_bounds__(kThreads)
watermark_elem_kernel(T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                      const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                      float delta, uint32_t vbase) {
  const uint32_t v = blockIdx.x * kThreads + threadIdx.x;
  for (int64_t row = blockIdx.y; row < B; row += gridDim.y) {
    if (v >= V) continue;
    const RowSeed<kW> rs = row_seed<kSeeding, kW>(key, context + row * width, width);
    bias_one<T, kSeeding>(logits + row * row_stride, v, rs, tm1, delta, vbase);
  }
}

// ---------------------------------------------------------------------------
// Greedy decoding fused with the watermark: the argmax of each watermarked row in
// one read-only pass.  A row is cut into segments; one workgroup scans a segment,
// keeps a running (value, index) per lane, reduces them and writes one partial
// (value bits, index) to the workspace.  A read-out kernel then reduces the
// partials of each row.  Candidates compare through a 64-bit key: the high word
// orders the values (every NaN above +inf, -0 equal to +0), the low word is
// ~index, so the maximum key is the largest value at its smallest index.
// ---------------------------------------------------------------------------
// 16-byte vectors per lane in a sub-batch of the fused decoding pass (greedy and
// sampling), and sub-batches per workgroup segment.  A longer segment gives each wave
// a larger sample for its bounds; every lane holds a sub-batch in registers, and bf16
// takes fewer vectors to hold its 8-token bounds.
#ifndef SBW_DECODE_VECS_F32_GREEDY
#define SBW_DECODE_VECS_F32_GREEDY 6   // greedy decoding, fp32 (sampling keeps 8)
#endif
#ifndef SBW_DECODE_VECS_F32
#define SBW_DECODE_VECS_F32 8
#endif
#ifndef SBW_DECODE_VECS_BF16
#define SBW_DECODE_VECS_BF16 4
#endif
#ifndef SBW_DECODE_VECS_BF16_SAMPLE
#define SBW_DECODE_VECS_BF16_SAMPLE 5   // sampling, bf16 (greedy keeps 4)
#endif
#ifndef SBW_DECODE_SUBS
#define SBW_DECODE_SUBS 1
#endif
constexpr int kElemSegSteps = 8;                                // element kernel
constexpr int64_t kArgmaxSegElems = kThreads * kElemSegSteps;   // element-kernel segment

__device__ __forceinline__ uint32_t order_bits(float f) {
  uint32_t b = __float_as_uint(f);
  if (f != f) return 0xFFFFFFFFu;
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t arg_key(float f, uint32_t v) {
  return (static_cast<uint64_t>(order_bits(f)) << 32) | static_cast<uint32_t>(~v);
}

// Running argmax of one lane, which visits its indices in increasing order: a strict
// greater-than keeps the first of equal values (and -0 == +0); the first NaN wins and
// then stays.  `any` is false until the lane has seen an element.  (Measured faster
// than a NaN-seeded form with fewer operations, and than a form without NaN handling.)
struct LaneBest {
  float v;
  uint32_t i;
  bool any;
};

__device__ __forceinline__ LaneBest lane_best_init() { return LaneBest{0.0f, 0u, false}; }

__device__ __forceinline__ void consider(LaneBest& b, float x, uint32_t i) {
  // Bitwise, not short-circuit, operators keep the update branch-free.
  const bool take = static_cast<bool>(static_cast<int>(!b.any) | static_cast<int>(x > b.v) |
                                      (static_cast<int>(x != x) & static_cast<int>(b.v == b.v)));
  b.v = take ? x : b.v;
  b.i = take ? i : b.i;
  b.any = true;
}

// The same argmax for a lane that sees its indices in any order: equal values and
// NaNs go to the smaller index.
__device__ __forceinline__ void consider_any_order(LaneBest& b, float x, uint32_t i) {
  const int xn = static_cast<int>(x != x), bn = static_cast<int>(b.v != b.v);
  const int first = static_cast<int>(i < b.i);
  const bool take = static_cast<bool>(static_cast<int>(!b.any) | static_cast<int>(x > b.v) |
                                      (static_cast<int>(x == b.v) & first) |
                                      (xn & ((1 - bn) | first)));
  b.v = take ? x : b.v;
  b.i = take ? i : b.i;
  b.any = true;
}

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(uint16_t x) { return __uint_as_float(static_cast<uint32_t>(x) << 16); }

// A partial result: value bits in the high word, index in the low word (0 = none is
// never produced: a workgroup's segment always holds at least one element).
__device__ __forceinline__ uint64_t pack_partial(float v, uint32_t i) {
  return (static_cast<uint64_t>(__float_as_uint(v)) << 32) | i;
}
__device__ __forceinline__ uint64_t partial_key(uint64_t p) {
  return arg_key(__uint_as_float(static_cast<uint32_t>(p >> 32)), static_cast<uint32_t>(p));
}

// Wave-wide maximum of 64-bit keys with their 64-bit payloads, by DPP moves (quad
// permutes, row mirrors, then row broadcasts that carry the maximum to lane 63); no
// index arithmetic or LDS round trips.  Lanes a move does not reach see key 0, which
// never wins.  The result is read from lane 63 into every lane.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ void dpp_argmax_step(uint64_t& k, uint64_t& p) {
  const uint32_t k0 = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      0, static_cast<int>(static_cast<uint32_t>(k)), kCtrl, kRowMask, 0xF, false));
  const uint32_t k1 = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      0, static_cast<int>(static_cast<uint32_t>(k >> 32)), kCtrl, kRowMask, 0xF, false));
  const uint32_t p0 = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      0, static_cast<int>(static_cast<uint32_t>(p)), kCtrl, kRowMask, 0xF, false));
  const uint32_t p1 = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      0, static_cast<int>(static_cast<uint32_t>(p >> 32)), kCtrl, kRowMask, 0xF, false));
  const uint64_t ok = (static_cast<uint64_t>(k1) << 32) | k0;
  if (ok > k) {
    k = ok;
    p = (static_cast<uint64_t>(p1) << 32) | p0;
  }
}
__device__ __forceinline__ uint64_t readlane63(uint64_t x) {
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x)), 63));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x >> 32)), 63));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ void wave_argmax(uint64_t& k, uint64_t& p) {
  dpp_argmax_step<0xB1, 0xF>(k, p);    // quad_perm [1,0,3,2]
  dpp_argmax_step<0x4E, 0xF>(k, p);    // quad_perm [2,3,0,1]
  dpp_argmax_step<0x141, 0xF>(k, p);   // row_half_mirror
  dpp_argmax_step<0x140, 0xF>(k, p);   // row_mirror
  dpp_argmax_step<0x142, 0xA>(k, p);   // row_bcast:15 into rows 1 and 3
  dpp_argmax_step<0x143, 0xC>(k, p);   // row_bcast:31 into rows 2 and 3
  k = readlane63(k);
  p = readlane63(p);
}

// Block-wide argmax of the lanes' running bests; thread 0 stores the partial.
__device__ __forceinline__ void block_argmax_store(const LaneBest& lb, uint64_t* out,
                                                   uint64_t* lds_key, uint64_t* lds_part) {
  uint64_t k = lb.any ? arg_key(lb.v, lb.i) : 0u;
  uint64_t p = pack_partial(lb.v, lb.i);
  wave_argmax(k, p);
  if (threadIdx.x % 64 == 0) {
    lds_key[threadIdx.x / 64] = k;
    lds_part[threadIdx.x / 64] = p;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t bk = lds_key[0], bp = lds_part[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w)
      if (lds_key[w] > bk) { bk = lds_key[w]; bp = lds_part[w]; }
    *out = bp;
  }
  __syncthreads();  // the LDS slots are reused by the next row of this workgroup
}

// Skipping elements that cannot win.  An element's watermarked value is either its
// logit x or bias(x) (the value it takes when green), and bias is non-decreasing in
// x for both dtypes (one rounded add; bf16 rounding is monotone too).  So if m is
// the largest logit of some set of elements, one of them ends at least at
// lb = min(m, bias(m)), and an element with x < lb and bias(x) < lb can be neither
// the maximum nor tied with it: its colour need not be drawn.  A NaN compares false
// and is always kept (it wins), so NaN logits never make the test skip anything;
// delta is finite, so bias(x) is NaN only when x is.
// The lower bound from the largest logit m (-inf when there is none).
__device__ __forceinline__ float reach_bound(float m, float delta, float) {
  return fminf(m, m + delta);
}
__device__ __forceinline__ float reach_bound(float m, float delta, uint16_t) {
  const uint32_t b = __float_as_uint(m) >> 16;   // m is a widened bf16
  return fminf(m, widen(bias_bf16(static_cast<uint16_t>(b), delta, true)));
}

// The 8 bf16 elements of a vector as (x, bias(x)) pairs: each token's two candidate
// values, widened.
__device__ __forceinline__ void green_values(u32x4 o, float delta, float (&x)[8], float (&gv)[8]) {
  const uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t g = bias_bf16x2(w[q], delta, true, true);
    x[2 * q] = __uint_as_float(w[q] << 16);
    x[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
    gv[2 * q] = __uint_as_float(g << 16);
    gv[2 * q + 1] = __uint_as_float(g & 0xFFFF0000u);
  }
}

// What a pass maximises: the watermarked logit (greedy decoding), or, for sampling,
// that logit times 1/T plus the token's Gumbel noise (the Gumbel-max trick).
template <bool kSample>
struct Score {
  uint64_t seed;    // sampling: the row's noise seed
  float inv_t;      // sampling: 1 / temperature
  __device__ __forceinline__ float of(float l, uint32_t v) const {
    if constexpr (kSample) return l * inv_t + gumbel_of(cbrng(v, seed));
    return l;
  }
};

// Each token's larger candidate logit, max(x, bias(x)), times 1/T.  fp32: bias(x)
// is x + delta rounded, so the larger one is x + max(delta, 0) (x + 0 only turns -0
// into +0).  bf16: bias rounds to bf16, so both candidates are formed.
__device__ __forceinline__ void upper_logits(f32x4 o, float, float dplus, float inv_t, float (&phi)[4]) {
  phi[0] = (o.x + dplus) * inv_t;
  phi[1] = (o.y + dplus) * inv_t;
  phi[2] = (o.z + dplus) * inv_t;
  phi[3] = (o.w + dplus) * inv_t;
}
__device__ __forceinline__ void upper_logits(u32x4 o, float delta, float, float inv_t, float (&phi)[8]) {
  float x[8], gv[8];
  green_values(o, delta, x, gv);
#pragma unroll
  for (int e = 0; e < 8; ++e) phi[e] = (delta >= 0.0f ? gv[e] : x[e]) * inv_t;
}

// The same without the temperature (greedy decoding).
__device__ __forceinline__ void upper_logits(f32x4 o, float, float dplus, float (&phi)[4]) {
  phi[0] = o.x + dplus;
  phi[1] = o.y + dplus;
  phi[2] = o.z + dplus;
  phi[3] = o.w + dplus;
}
__device__ __forceinline__ void upper_logits(u32x4 o, float delta, float, float (&phi)[8]) {
  float x[8], gv[8];
  green_values(o, delta, x, gv);
#pragma unroll
  for (int e = 0; e < 8; ++e) phi[e] = delta >= 0.0f ? gv[e] : x[e];
}

// Largest raw logit of a vector folded into m.  v_max3_f32 on the raw values: the
// compiler's fmaxf would first canonicalise every loaded value.  A signalling NaN
// may make m NaN, which only turns the skip test built on m off.
__device__ __forceinline__ float max3_raw(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float fold_max(f32x4 o, float m) {
  return max3_raw(max3_raw(m, o.x, o.y), o.z, o.w);
}
__device__ __forceinline__ float fold_max(u32x4 o, float m) {
  const uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) m = max3_raw(m, __uint_as_float(w[q] << 16), __uint_as_float(w[q] & 0xFFFF0000u));
  return m;
}

// Largest value over the wave, by DPP moves on order-preserving integer keys (no
// index arithmetic or LDS round trips): within quads, half rows and rows, then row
// broadcasts carry the maximum to lane 63.  A NaN lane may make the result NaN,
// which makes every bound test above keep its token.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int dpp_max_step(int k) {
  return max(k, __builtin_amdgcn_update_dpp(static_cast<int>(0x80000000u), k, kCtrl, kRowMask, 0xF, false));
}
__device__ __forceinline__ float wave_max(float v) {
  int k = __float_as_int(v);
  k ^= (k >> 31) & 0x7FFFFFFF;
  k = dpp_max_step<0xB1, 0xF>(k);    // quad_perm [1,0,3,2]
  k = dpp_max_step<0x4E, 0xF>(k);    // quad_perm [2,3,0,1]
  k = dpp_max_step<0x141, 0xF>(k);   // row_half_mirror
  k = dpp_max_step<0x140, 0xF>(k);   // row_mirror
  k = dpp_max_step<0x142, 0xA>(k);   // row_bcast:15 into rows 1 and 3
  k = dpp_max_step<0x143, 0xC>(k);   // row_bcast:31 into rows 2 and 3
  k = __builtin_amdgcn_readlane(k, 63);
  return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF));
}

// The raw bits of element e of a vector (fp32 bits, or bf16 bits in the low half).
__device__ __forceinline__ uint32_t raw_elem(f32x4 o, int e) {
  const float w[4] = {o.x, o.y, o.z, o.w};
  return __float_as_uint(w[e]);
}
__device__ __forceinline__ uint32_t raw_elem(u32x4 o, int e) {
  const uint32_t w[4] = {o.x, o.y, o.z, o.w};
  return (e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu);
}
__device__ __forceinline__ float from_raw(uint32_t r, float) { return __uint_as_float(r); }
__device__ __forceinline__ uint16_t from_raw(uint32_t r, uint16_t) { return static_cast<uint16_t>(r); }

// The noise draws of vector j: 4 tokens (fp32) or 8 (bf16), one block per 4 tokens
// as CBRNG lays them out.
__device__ __forceinline__ void noise_words(uint32_t j, const RoundKeys& k, uint32_t (&x)[4]) {
  const Block n = philox_block(j, k);
  x[0] = n.w0; x[1] = n.w1; x[2] = n.w2; x[3] = n.w3;
}
__device__ __forceinline__ void noise_words(uint32_t j, const RoundKeys& k, uint32_t (&x)[8]) {
  const Block n0 = philox_block(2u * j, k);
  const Block n1 = philox_block(2u * j + 1u, k);
  x[0] = n0.w0; x[1] = n0.w1; x[2] = n0.w2; x[3] = n0.w3;
  x[4] = n1.w0; x[5] = n1.w1; x[6] = n1.w2; x[7] = n1.w3;
}

// Appends a lane's token to the wave's queue at its rank among the lanes in mask.
__device__ __forceinline__ void enqueue(uint32_t* q_v, uint32_t* q_raw, uint32_t queued, uint64_t mask,
                                        uint32_t v, uint32_t raw) {
  const uint32_t pos = queued + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                                          __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
  q_v[pos] = v;
  q_raw[pos] = raw;
}

// The exact score of one queued token: colour, bias, noise.
template <typename T, int kSeeding, int kW, bool kSample>
__device__ __forceinline__ void score_entry(LaneBest& b, uint32_t v, uint32_t raw_bits,
                                            const RowSeed<kW>& rs, uint32_t tm1, int none_green,
                                            float delta, const Score<kSample>& sc) {
  const T raw = from_raw(raw_bits, T{});
  uint32_t x;
  if constexpr (kSeeding == kContext)
    x = block_word(philox_block(v >> 2, opaque_key(key_of(rs.seed))), v & 3u);
  else
    x = draw<kSelfSalt>(rs, v);
  const bool g = !none_green && is_green(x, tm1);
  const float l = widen(bias_elem(raw, delta, g));
  if constexpr (kSample) {
    const float noise = gumbel_of(block_word(philox_block(v >> 2, opaque_key(key_of(sc.seed))), v & 3u));
    consider_any_order(b, l * sc.inv_t + noise, v);
  } else {
    consider_any_order(b, l, v);
  }
}

// Scores the queued tokens of a wave, 64 at a time, one per lane.
template <typename T, int kSeeding, int kW, bool kSample>
__device__ __forceinline__ void score_queue(LaneBest& b, const uint32_t* q_v, const uint32_t* q_raw,
                                            uint32_t queued, const RowSeed<kW>& rs, uint32_t tm1,
                                            int none_green, float delta, const Score<kSample>& sc) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (uint32_t i = threadIdx.x % 64u; i < queued; i += 64u)
    score_entry<T, kSeeding, kW, kSample>(b, q_v[i], q_raw[i], rs, tm1, none_green, delta, sc);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Fused decoding, vector path: greedy (kSample false) or Gumbel-max sampling.  A
// segment is kSub sub-batches of kThreads * kN vectors, vector n of lane t at
// offset n * kThreads + t; every lane loads a sub-batch at once.  The colour draw
// (and, sampling, the exact noise with its two logarithms) matters only for the few
// tokens that may still reach the wave's best score.  Per sub-batch:
//  1. greedy: with m the wave's largest logit, some token ends at least at
//     lb = min(m, bias(m)), and a token's value is at most max(x, bias(x));
//     sampling: lb from m with the noise's overall minimum, and a vector none of
//     whose tokens reaches lb even with the noise's overall maximum draws no noise;
//     the other vectors draw their noise, each token's score is bounded from above
//     and below by the bounds of its noise (gumbel_upper, kGumbelGap) and of its
//     logit, and lb rises to the largest lower bound of the wave;
//  2. the tokens whose upper bound reaches lb join the wave's queue in LDS; a queue
//     that would overflow is scored exactly, one token per lane, and at the end
//     the four waves' queues are scored together.
// lb only rises.  A token left out scores below lb, which some token of the wave's
// share attains, so the partial equals that of a full scan.  The sampling bounds
// follow from monotone fp32 rounding: the score is (l * 1/T) + G with both steps
// rounded and 1/T > 0.  Lanes see tokens out of index order, so their running
// argmax breaks ties by index.
template <typename T, int kSeeding, int kN, int kSub, int kW, bool kSample>
__global__ void __launch_bounds__(kThreads)
decode_vec_kernel(const T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                  const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                  int none_green, float delta, const uint64_t* __restrict__ seeds, float inv_t,
                  uint32_t segments, uint64_t* __restrict__ partials, uint32_t vbase) {
  using VecT = typename std::conditional<sizeof(T) == 4, f32x4, u32x4>::type;
  constexpr int kE = sizeof(T) == 4 ? 4 : 8;         // tokens per vector
  const uint32_t jbase = vbase / kE;                 // vector index of the first column
  __shared__ uint64_t lds_key[kThreads / 64], lds_part[kThreads / 64];
  // Per wave: token ids, then raw logits.  The queue is scored whenever it holds more
  // than 64 tokens before a vector is queued, so it never holds more than 64 plus one
  // vector's worth (kE tokens in each of 64 lanes).
  constexpr uint32_t kQueueCap = 64u + 64u * kE;
  __shared__ uint32_t lds_queue[(kThreads / 64) * 2 * kQueueCap];
  __shared__ uint32_t lds_count[kThreads / 64];
  uint32_t* q_v = lds_queue + (threadIdx.x / 64u) * 2u * kQueueCap;
  uint32_t* q_raw = q_v + kQueueCap;
  constexpr uint32_t kPer = 16u / sizeof(T);
  constexpr uint32_t kSubVecs = kThreads * kN;       // vectors per sub-batch
  const uint32_t full = V / kPer;
  const uint32_t tail = V % kPer;
  const uint32_t seg_base = blockIdx.x * (kSubVecs * kSub);
  for (int64_t row = blockIdx.y; row < B; row += gridDim.y) {
    const T* row_ptr = logits + row * row_stride;
    const VecT* vec = reinterpret_cast<const VecT*>(row_ptr);
    Score<kSample> sc{0u, inv_t};
    RoundKeys nk{};
    if constexpr (kSample) {
      sc.seed = seeds[row];
      nk = vector_round_keys(key_of(sc.seed));
    }
    const RowSeed<kW> rs = row_seed<kSeeding, kW>(key, context + row * width, width);
    const float dt = fabsf(delta) * inv_t;
    const float dplus = delta > 0.0f ? delta : 0.0f;
    LaneBest best = lane_best_init();
    float lb = -INFINITY;           // the best score is at least lb (the same in every lane)
    uint32_t queued = 0;            // tokens in the wave's queue (the same in every lane)
    // Sub-batch `sub` into registers; the next one is loaded while this one is scored.
    auto load_sub = [&](VecT (&buf)[kN], int sub) {
      // Opaque to the optimiser, so that no Philox work is hoisted out of the loops.
      uint32_t sub_first = seg_base + static_cast<uint32_t>(sub) * kSubVecs;
      asm volatile("" : "+s"(sub_first));
      if (sub_first + kSubVecs <= full) {
#pragma unroll
        for (int n = 0; n < kN; ++n) buf[n] = stream_load(vec + sub_first + n * kThreads + threadIdx.x);
      } else {
#pragma unroll
        for (int n = 0; n < kN; ++n) {
          const uint32_t j = sub_first + n * kThreads + threadIdx.x;
          buf[n] = VecT{};
          if (j < full) buf[n] = stream_load(vec + j);
        }
      }
    };
    auto process_sub = [&](const VecT (&buf)[kN], int sub) {
      uint32_t sub_first = seg_base + static_cast<uint32_t>(sub) * kSubVecs;
      asm volatile("" : "+s"(sub_first));
      // The same sub-batch counted in token-id vectors (the row's first id is vbase).
      uint32_t id_first = sub_first + jbase;
      asm volatile("" : "+s"(id_first));
      const bool whole = sub_first + kSubVecs <= full;
      float m = -INFINITY;
#pragma unroll
      for (int n = 0; n < kN; ++n)
        if (whole || sub_first + n * kThreads + threadIdx.x < full) m = fold_max(buf[n], m);
      float hi[kN][kE];
      if constexpr (!kSample) {
        // Greedy decoding: the largest logit's own value bounds the best from below,
        // and a token's larger candidate value bounds it from above.
        lb = fmaxf(lb, reach_bound(wave_max(m), delta, T{}));
#pragma unroll
        for (int n = 0; n < kN; ++n) upper_logits(buf[n], delta, dplus, hi[n]);
      } else {
      const float lb0 = fmaxf(lb, reach_bound(wave_max(m), delta, T{}) * inv_t + kGumbelLo);
      float top = -INFINITY;    // the lane's largest hi among tokens whose draw has c >= 2
#pragma unroll
      for (int n = 0; n < kN; ++n) {
        const uint32_t j = sub_first + n * kThreads + threadIdx.x;
        float phi[kE];
        upper_logits(buf[n], delta, dplus, inv_t, phi);
        float vmax = -INFINITY;   // NaN-propagating: a NaN token is always kept
#pragma unroll
        for (int e = 0; e < kE; ++e) vmax = __builtin_elementwise_maximum(vmax, phi[e]);
        const bool reach = (whole || j < full) && !(vmax + kGumbelHi < lb0);
#pragma unroll
        for (int e = 0; e < kE; ++e) hi[n][e] = -INFINITY;
        if (reach) {
          uint32_t nw[kE];
          noise_words(id_first + n * kThreads + threadIdx.x, nk, nw);
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const float c = noise_ones(nw[e]);
            hi[n][e] = phi[e] + gumbel_upper(c);
            top = fmaxf(top, c >= 2.0f ? hi[n][e] : -INFINITY);
          }
        }
      }
      // A token with c >= 2 and upper bound hi scores at least hi - gap - d: its noise
      // is at least gumbel_upper(c) - kGumbelGap, and its two candidate logits times
      // 1/T differ by at most |delta|/T plus roundings (of the bias, to 8 significant
      // bits for bf16, and of the products), which the relative term covers, as it
      // covers the rounding of this subtraction.  An infinite top gives no bound.
      {
        constexpr float kRel = sizeof(T) == 4 ? 0x1p-18f : 0x1p-7f;
        const float slack = kGumbelGap + dt + kRel * (fabsf(top) + 18.0f + dt);
        const float lb_lane = top < INFINITY ? top - slack : -INFINITY;
        lb = fmaxf(lb0, wave_max(lb_lane));
      }
      }

      // Queue the tokens whose upper bound reaches lb.  The counters are the same in
      // every lane.
#pragma unroll
      for (int n = 0; n < kN; ++n) {
        if (queued > 64u) {
          score_queue<T, kSeeding, kW, kSample>(best, q_v, q_raw, queued, rs, tm1, none_green, delta, sc);
          queued = 0;
          lb = fmaxf(lb, wave_max(best.any ? best.v : -INFINITY));
        }
        const uint32_t j = sub_first + n * kThreads + threadIdx.x;
        const uint32_t jid = id_first + n * kThreads + threadIdx.x;
        if (whole) {
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const bool reaches = !(hi[n][e] < lb);
            const uint64_t mask = __ballot(reaches);
            if (reaches) enqueue(q_v, q_raw, queued, mask, jid * kE + e, raw_elem(buf[n], e));
            queued = __builtin_amdgcn_readfirstlane(queued + static_cast<uint32_t>(__popcll(mask)));
          }
        } else {
          const bool valid = j < full;
          const uint64_t valid_mask = __ballot(valid);
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const bool reaches = !(hi[n][e] < lb);
            const uint64_t mask = __ballot(reaches) & valid_mask;
            if (valid && reaches) enqueue(q_v, q_raw, queued, mask, jid * kE + e, raw_elem(buf[n], e));
            queued = __builtin_amdgcn_readfirstlane(queued + static_cast<uint32_t>(__popcll(mask)));
          }
        }
      }
    };
    VecT buf0[kN], buf1[kN];
    load_sub(buf0, 0);
    for (int sub = 0; sub < kSub; sub += 2) {
      if (sub + 1 < kSub) load_sub(buf1, sub + 1);
      process_sub(buf0, sub);
      if (sub + 1 < kSub) {
        if (sub + 2 < kSub) load_sub(buf0, sub + 2);
        process_sub(buf1, sub + 1);
      }
    }
    // What is left in the four queues is scored together: entry i of their
    // concatenation goes to lane i % 64 of wave (i / 64) % 4, so a workgroup's few
    // candidates take one wave's pass instead of four.
    {
      const uint32_t lane = threadIdx.x % 64u, wave = threadIdx.x / 64u;
      if (lane == 0u) lds_count[wave] = queued;
      __syncthreads();
      uint32_t start[kThreads / 64 + 1];
      start[0] = 0u;
#pragma unroll
      for (int w = 0; w < kThreads / 64; ++w) start[w + 1] = start[w] + lds_count[w];
      const uint32_t total = start[kThreads / 64];
      for (uint32_t i = wave * 64u + lane; i < total; i += kThreads) {
        uint32_t w = 0;
#pragma unroll
        for (int k = 1; k < kThreads / 64; ++k) w += static_cast<uint32_t>(i >= start[k]);
        const uint32_t* wq = lds_queue + w * 2u * kQueueCap;
        const uint32_t off = i - start[w];
        score_entry<T, kSeeding, kW, kSample>(best, wq[off], wq[kQueueCap + off], rs, tm1, none_green,
                                               delta, sc);
      }
    }
    // The row's partial last vector, element by element, by lane 0 of the segment
    // that holds it.
    if (tail != 0u && threadIdx.x == 0 && full >= seg_base && full - seg_base < kSubVecs * kSub) {
      for (uint32_t e = 0; e < tail; ++e) {
        const uint32_t c = full * kPer + e;          // column; the token id is vbase + c
        const uint32_t v = vbase + c;
        const bool g = !none_green && is_green(draw<kSeeding>(rs, v), tm1);
        consider_any_order(best, sc.of(widen(bias_elem(row_ptr[c], delta, g)), v), v);
      }
    }
    block_argmax_store(best, partials + row * segments + blockIdx.x, lds_key, lds_part);
  }
}

// Rows that are not 16-byte aligned: one element per thread per step, a segment of
// kArgmaxSegElems elements per workgroup.
template <typename T, int kSeeding, int kW, bool kSample>
__global__ void __launch_bounds__(kThreads)
argmax_elem_kernel(const T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                   const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                   int none_green, float delta, const uint64_t* __restrict__ seeds, float inv_t,
                   uint32_t segments, uint64_t* __restrict__ partials, uint32_t vbase) {
  __shared__ uint64_t lds_key[kThreads / 64], lds_part[kThreads / 64];
  const uint64_t seg_first = static_cast<uint64_t>(blockIdx.x) * kArgmaxSegElems;
  for (int64_t row = blockIdx.y; row < B; row += gridDim.y) {
    const RowSeed<kW> rs = row_seed<kSeeding, kW>(key, context + row * width, width);
    const Score<kSample> sc{kSample ? seeds[row] : 0u, inv_t};
    LaneBest lb = lane_best_init();
    for (int s = 0; s < kElemSegSteps; ++s) {
      const uint64_t v64 = seg_first + static_cast<uint64_t>(s) * kThreads + threadIdx.x;
      if (v64 < V) {
        const uint32_t c = static_cast<uint32_t>(v64);   // column; the token id is vbase + c
        const uint32_t v = vbase + c;
        const bool g = !none_green && is_green(draw<kSeeding>(rs, v), tm1);
        consider(lb, sc.of(widen(bias_elem(logits[row * row_stride + c], delta, g)), v), v);
      }
    }
    block_argmax_store(lb, partials + row * segments + blockIdx.x, lds_key, lds_part);
  }
}

// Read-out: one wavefront per row loads the row's partials at once, reduces their
// keys with shuffles, and lane 0 unpacks the winner.
__global__ void __launch_bounds__(kThreads)
argmax_finish_kernel(const uint64_t* __restrict__ partials, uint32_t segments, int64_t B,
                     int32_t* __restrict__ tokens, float* __restrict__ values) {
  const int lane = threadIdx.x % 64;
  for (int64_t b = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + threadIdx.x / 64; b < B;
       b += static_cast<int64_t>(gridDim.x) * (kThreads / 64)) {
    const uint64_t* p = partials + b * segments;
    uint64_t bk = 0u, bp = 0u;
    for (uint32_t s = lane; s < segments; s += 64) {
      const uint64_t k = partial_key(p[s]);
      if (k > bk) { bk = k; bp = p[s]; }
    }
    wave_argmax(bk, bp);
    if (lane == 0) {
      tokens[b] = static_cast<int32_t>(static_cast<uint32_t>(bp));
      if (values != nullptr) values[b] = __uint_as_float(static_cast<uint32_t>(bp >> 32));
    }
  }
}

// ---------------------------------------------------------------------------
// Candidate-restricted watermark (top-k self-salt).  One workgroup per row; lane t
// takes candidates t, t + kThreads, ...  A candidate's logit load is issued as soon
// as its id arrives, and the row's window loads, the repeat test and the colour
// draw overlap it.  An id outside [0, V), or equal to an earlier id of the row, is
// skipped, so every logit is written by at most one lane.
// ---------------------------------------------------------------------------
constexpr int kMaxCandidates = 1024;

template <typename T, int kSeeding, int kW>
__global__ void __launch_bounds__(kThreads)
candidates_kernel(T* __restrict__ logits, int64_t row_stride, uint32_t V, int64_t B,
                  const int32_t* __restrict__ cand, int k, const int32_t* __restrict__ context,
                  int width, uint64_t key, uint32_t tm1, float delta) {
  __shared__ int32_t ids[kMaxCandidates];
  for (int64_t row = blockIdx.x; row < B; row += gridDim.x) {
    const int32_t* row_cand = cand + row * k;
    T* row_ptr = logits + row * row_stride;
    for (int j = threadIdx.x; j < k; j += kThreads) ids[j] = row_cand[j];
    const RowSeed<kW> rs = row_seed<kSeeding, kW>(key, context + row * width, width);
    __syncthreads();
    for (int base = 0; base < k; base += kThreads) {
      const int j = base + static_cast<int>(threadIdx.x);
      const int32_t id = j < k ? ids[j] : -1;
      const bool in_range = id >= 0 && static_cast<uint32_t>(id) < V;
      T l{};
      if (in_range) l = row_ptr[id];
      // repeat test: a loop of uniform length over broadcast LDS reads
      const int upto = min(k, base + kThreads) - 1;
      int repeat = 0;
#pragma unroll 8
      for (int i = 0; i < upto; ++i) repeat |= static_cast<int>(ids[i] == id) & static_cast<int>(i < j);
      if (in_range && !repeat && is_green(draw<kSeeding>(rs, static_cast<uint32_t>(id)), tm1))
        row_ptr[id] = bias_elem(l, delta, true);
    }
    __syncthreads();  // ids is refilled for the next row of this workgroup
  }
}

// ---------------------------------------------------------------------------
// Green mask: one lane per 32-bit word (tokens 32w .. 32w+31).
// ---------------------------------------------------------------------------
template <int kSeeding, int kW>
__global__ void __launch_bounds__(kThreads)
green_mask_kernel(uint32_t* __restrict__ bits, uint32_t V, uint32_t words_per_row,
                  const int32_t* __restrict__ context, int width, uint64_t key, uint32_t tm1,
                  int none_green, int64_t num_words) {
  for (int64_t w = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; w < num_words;
       w += static_cast<int64_t>(gridDim.x) * kThreads) {
    const int64_t row = w / words_per_row;
    const uint32_t word = static_cast<uint32_t>(w - row * words_per_row);
    uint32_t out = 0u;
    if (!none_green) {
      const RowSeed<kW> rs = row_seed<kSeeding, kW>(key, context + row * width, width);
      const uint32_t v0 = word * 32u;
      if (kSeeding == kContext) {
        const Key k = key_of(rs.seed);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const Block blk = philox_block(v0 / 4u + q, k);
          const uint32_t xs[4] = {blk.w0, blk.w1, blk.w2, blk.w3};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            out |= static_cast<uint32_t>(is_green(xs[e], tm1)) << (4 * q + e);
        }
      } else {
#pragma unroll 4
        for (int e = 0; e < 32; ++e)
          out |= static_cast<uint32_t>(is_green(draw<kSeeding>(rs, v0 + e), tm1)) << e;
      }
      const uint32_t valid = V - v0;  // >= 1 for every word of the row
      if (valid < 32u) out &= (1u << valid) - 1u;
    }
    bits[w] = out;
  }
}

// ---------------------------------------------------------------------------
// Detect: one wavefront per sequence, ballot + popcount.
// ---------------------------------------------------------------------------
constexpr int kWave = 64;
constexpr int kWavesPerBlock = kThreads / kWave;

// Lane `l`'s 64-bit value, in every lane.
__device__ __forceinline__ uint64_t readlane64(uint64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(x), l);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(x >> 32), l);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Lane t gets lane t - 1's x (wave_shr:1); lane 0 gets `first`.
__device__ __forceinline__ uint64_t wave_shift_right(uint64_t x, uint64_t first) {
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      static_cast<int>(static_cast<uint32_t>(first)), static_cast<int>(static_cast<uint32_t>(x)),
      0x138, 0xF, 0xF, false));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
      static_cast<int>(static_cast<uint32_t>(first >> 32)),
      static_cast<int>(static_cast<uint32_t>(x >> 32)), 0x138, 0xF, 0xF, false));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Membership of token v at a position whose window is w[0..width-1].
template <int kSeeding, int kW>
__device__ __forceinline__ bool window_green(uint64_t key, const uint32_t (&w)[kW], int width,
                                             uint32_t v, uint32_t tm1) {
  uint64_t r;
  if (kSeeding == kContext) {
    if constexpr (kW == 1) {
      r = lane_mul_64x32(key, w[0]);
    } else {
      uint64_t sum = 0u;
#pragma unroll
      for (int i = 0; i < kW; ++i)
        if (i < width) sum += w[i];
      r = key * sum;
    }
  } else {
    const uint32_t jv = jenkins32_lane(v);
    r = mul_64x64(key, wide_mul(jv, jv));
#pragma unroll
    for (int i = 0; i < kW; ++i) {
      if (kW == 1 || i < width) {
        const uint64_t t = lane_mul_64x32(key * static_cast<uint64_t>(jenkins32_lane(w[i])), jv);
        r = t < r ? t : r;
      }
    }
  }
  return is_green(cbrng_lane(v, r), tm1);
}

// Positions handled per lane per pass: a pass covers 64 * kChunk positions and
// issues all of its token loads before any arithmetic.  The host picks kChunk from
// the number of scored positions so that short sequences do not compute idle slots.
// Outputs of a detect launch; `lengths` (per-sequence token counts, clamped to
// [0, L]) and `scored` (T per sequence) may be null.
struct DetectIO {
  const int32_t* lengths;
  int32_t* counts;
  int32_t* scored;
  double* z;
};

__device__ __forceinline__ int64_t sequence_length(const int32_t* lengths, int64_t n, int64_t L) {
  if (lengths == nullptr) return L;
  const int64_t len = lengths[n];
  return len < 0 ? 0 : (len > L ? L : len);
}

__device__ __forceinline__ void detect_store(const DetectIO& io, int64_t n, uint32_t green,
                                             int64_t T, double gamma) {
  const double t = static_cast<double>(T);
  const double numerator = static_cast<double>(green) - t * gamma;
  const double denominator = sqrt(t * gamma * (1.0 - gamma));
  io.counts[n] = static_cast<int32_t>(green);
  if (io.scored != nullptr) io.scored[n] = static_cast<int32_t>(T);
  io.z[n] = numerator / denominator;
}

// Positions are 32-bit (L < 2^31).  Lanes past the end of the sequence load the last
// token instead (a valid address), so the loads need no branch; their positions are
// masked out of the count with a lane mask built in scalar registers.  The four waves
// of a workgroup take four sequences; their counts meet in LDS and one wave computes
// the four z-scores side by side (lanes 0-3), so the fp64 epilogue issues once per
// workgroup instead of once per wave.  Every wave of the workgroup runs the same
// number of outer iterations, so the barriers are reached by all of them.
template <int kSeeding, int kChunk, int kW>
__global__ void __launch_bounds__(kThreads)
detect_kernel(const int32_t* __restrict__ tokens, int64_t N, int64_t L, int64_t row_stride,
              int width, uint64_t key, uint32_t tm1, double gamma, DetectIO io) {
  __shared__ uint32_t lds_green[kWavesPerBlock], lds_len[kWavesPerBlock];
  const uint32_t lane = threadIdx.x % kWave;
  // the wave's index in the workgroup, in a scalar register
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
  for (int64_t n0 = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock; n0 < N;
       n0 += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
    const int64_t n = n0 + wave;
    uint32_t green = 0u;  // wave-uniform count
    uint32_t len = 0u;
    if (n < N) {
      const int32_t* seq = tokens + n * row_stride;
      len = static_cast<uint32_t>(sequence_length(io.lengths, n, L));
      for (uint32_t base = static_cast<uint32_t>(width); base < len; base += kWave * kChunk) {
        // The pass's tokens and their windows from two wave-uniform bases; each load
        // adds the lane's byte offset, clamped to the pass's last position.
        const char* pass = reinterpret_cast<const char*>(seq + base);
        const char* pass_w = pass - 4 * width;
        const uint32_t rem = len - base;              // positions left, > 0
        const uint32_t last_byte = 4u * (rem - 1u);
        uint32_t w[kChunk][kW], v[kChunk];
        constexpr bool kShared = kSeeding == kSelfSalt && kW == 1;   // terms handed over
#pragma unroll
        for (int c = 0; c < kChunk; ++c) {
          const uint32_t ob = min(4u * (static_cast<uint32_t>(c * kWave) + lane), last_byte);
          v[c] = *reinterpret_cast<const uint32_t*>(pass + ob);
#pragma unroll
          for (int k = 0; k < kW; ++k)
            w[c][k] = ((kW == 1 || k < width) && !kShared)
                          ? *reinterpret_cast<const uint32_t*>(pass_w + ob + 4u * static_cast<uint32_t>(k))
                          : 0u;
        }
        // Independent membership chains first (instruction-level parallelism), then
        // one ballot per chunk.
        bool g[kChunk];
        if constexpr (kShared) {
          // Self-salt, width 1: the seed of position i is min(K J(p) J(v), K J(v) J(v))
          // with p the token at i - 1.  Each lane computes K J(v) of its own token once;
          // position i's K J(p) is position i - 1's K J(v), held by the lane before (lane
          // 63 of the chunk before, for lane 0), and a wave shift hands it over.  The
          // pass's first window token is the same for the whole wave: one scalar load,
          // hashed in scalar registers.
          uint32_t jv[kChunk];
          uint64_t kj[kChunk];
#pragma unroll
          for (int c = 0; c < kChunk; ++c) {
            jv[c] = jenkins32_lane(v[c]);
            kj[c] = lane_mul_64x32(key, jv[c]);
          }
          const uint32_t p0 = *reinterpret_cast<const uint32_t*>(pass_w);
          uint64_t carry = key * static_cast<uint64_t>(jenkins32(p0));
#pragma unroll
          for (int c = 0; c < kChunk; ++c) {
            if (c > 0) carry = readlane64(kj[c - 1], kWave - 1);
            const uint64_t kjp = wave_shift_right(kj[c], carry);
            const uint64_t self = lane_mul_64x32(kj[c], jv[c]);
            const uint64_t t = lane_mul_64x32(kjp, jv[c]);
            g[c] = is_green(cbrng_lane(v[c], t < self ? t : self), tm1);
          }
        } else {
#pragma unroll
          for (int c = 0; c < kChunk; ++c) g[c] = window_green<kSeeding, kW>(key, w[c], width, v[c], tm1);
        }
        // Chunks before rem / 64 lie inside the sequence, the next one holds its last
        // rem % 64 positions, the others none (masks in scalar registers).
        const uint32_t full_chunks = rem / static_cast<uint32_t>(kWave);
        const uint64_t part_mask = (uint64_t{1} << (rem % static_cast<uint32_t>(kWave))) - 1u;
#pragma unroll
        for (int c = 0; c < kChunk; ++c) {
          const uint32_t cu = static_cast<uint32_t>(c);
          const uint64_t valid = cu < full_chunks ? ~uint64_t{0} : (cu == full_chunks ? part_mask : 0u);
          green += static_cast<uint32_t>(__popcll(__ballot(g[c]) & valid));
        }
      }
    }
    if (lane == 0u) {
      lds_green[wave] = green;
      lds_len[wave] = len;
    }
    __syncthreads();
    if (wave == 0 && lane < static_cast<uint32_t>(kWavesPerBlock) && n0 + lane < N) {
      const uint32_t ln = lds_len[lane];
      detect_store(io, n0 + lane, lds_green[lane], ln > static_cast<uint32_t>(width) ? ln - width : 0, gamma);
    }
    __syncthreads();  // the LDS slots are rewritten by the next iteration
  }
}

// Detection with each distinct (width+1)-gram scored once.  One workgroup per
// sequence: the sequence is staged in LDS, next to an insert-only hash set of
// positions (linear probing; a quarter full, half for the longest texts).  A slot
// holds the position in its low 13 bits and 19 bits of the n-gram's hash above them.
// A lane claims an empty slot with a compare-and-swap, or meets a slot holding an
// equal n-gram and stops there, so exactly one position of every distinct n-gram is
// claimed and scored, whatever the interleaving; the tokens are compared only when
// the hash bits agree.
constexpr uint32_t kMaxUniqueSlots = 8192;   // 32 KB of LDS (+ up to 16 KB of tokens): 4096 positions
constexpr uint32_t kSlotPosBits = 13;        // positions < 8192 (L <= 4096 + kMaxWidth)
constexpr int32_t kEmptySlot = -1;           // never a slot value: no position is 8191
static_assert(kMaxUniqueSlots / 2 + kMaxWidth < (1u << kSlotPosBits) - 1u,
              "every position fits the slot's position bits and differs from 8191");

__device__ __forceinline__ uint32_t ngram_hash(const int32_t* seq, int64_t i, int width) {
  uint32_t h = 0x9E3779B9u;
  for (int k = 0; k <= width; ++k) {
    h = (h ^ static_cast<uint32_t>(seq[i - width + k])) * 0x85EBCA6Bu;
    h ^= h >> 13;
  }
  return h ^ (h >> 16);
}

__device__ __forceinline__ bool same_ngram(const int32_t* seq, int64_t a, int64_t b, int width) {
  bool same = true;
  for (int k = 0; k <= width; ++k) same = same && seq[a - width + k] == seq[b - width + k];
  return same;
}

#ifndef SBW_UNIQUE_BLOCK
#define SBW_UNIQUE_BLOCK 256  // threads per sequence of the repeat-rule detect
#endif
constexpr int kUniqueBlock = SBW_UNIQUE_BLOCK;

template <int kSeeding, int kW>
__global__ void __launch_bounds__(kUniqueBlock)
detect_unique_kernel(const int32_t* __restrict__ tokens, int64_t N, int64_t L, int64_t row_stride,
                     int width, uint64_t key, uint32_t tm1, double gamma, uint32_t slots,
                     DetectIO io) {
  extern __shared__ int32_t smem[];
  int32_t* table = smem;           // `slots` entries, a power of two
  int32_t* seq = smem + slots;     // the sequence's tokens (up to L)
  __shared__ uint32_t sums[2];
  for (int64_t n = blockIdx.x; n < N; n += gridDim.x) {
    const int32_t* src = tokens + n * row_stride;
    const int64_t len = sequence_length(io.lengths, n, L);
    for (int64_t t = threadIdx.x; t < len; t += kUniqueBlock) seq[t] = src[t];
    for (uint32_t sl = threadIdx.x; sl < slots; sl += kUniqueBlock) table[sl] = kEmptySlot;
    if (kUniqueBlock > kWave && threadIdx.x < 2) sums[threadIdx.x] = 0u;
    __syncthreads();
    uint32_t trials = 0u, green = 0u;
    for (int64_t i = width + threadIdx.x; i < len; i += kUniqueBlock) {
      const uint32_t h = ngram_hash(seq, i, width);
      const uint32_t fp = h >> kSlotPosBits;
      const int32_t mine = static_cast<int32_t>((fp << kSlotPosBits) | static_cast<uint32_t>(i));
      uint32_t slot = h & (slots - 1u);
      bool claimed = false;
      // at most `slots` probes; the set never fills, so a lane stops long before
      for (uint32_t probe = 0; probe < slots; ++probe) {
        const int32_t held = atomicCAS(&table[slot], kEmptySlot, mine);
        if (held == kEmptySlot) { claimed = true; break; }
        if ((static_cast<uint32_t>(held) >> kSlotPosBits) == fp &&
            same_ngram(seq, static_cast<int64_t>(static_cast<uint32_t>(held) & ((1u << kSlotPosBits) - 1u)), i, width))
          break;
        slot = (slot + 1u) & (slots - 1u);
      }
      if (claimed) {
        uint32_t w[kW];
#pragma unroll
        for (int k = 0; k < kW; ++k)
          w[k] = (kW == 1 || k < width) ? static_cast<uint32_t>(seq[i - width + k]) : 0u;
        ++trials;
        green += window_green<kSeeding, kW>(key, w, width, static_cast<uint32_t>(seq[i]), tm1)
                     ? 1u : 0u;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      trials += __shfl_xor(trials, off, 64);
      green += __shfl_xor(green, off, 64);
    }
    if constexpr (kUniqueBlock == kWave) {
      if (threadIdx.x == 0) detect_store(io, n, green, trials, gamma);
    } else {
      if (threadIdx.x % 64 == 0) {
        atomicAdd(&sums[0], trials);
        atomicAdd(&sums[1], green);
      }
      __syncthreads();
      if (threadIdx.x == 0) detect_store(io, n, sums[1], sums[0], gamma);
    }
    __syncthreads();  // the table (and sums) are reset for the next sequence
  }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
thread_local hipError_t g_last_hip_error = hipSuccess;

// ceil(gamma * 2^32) clamped to [0, 2^32] (the scaling by 2^32 is exact).
uint64_t threshold_of(double gamma) {
  const double scaled = ceil(gamma * 4294967296.0);
  if (!(scaled > 0.0)) return 0u;
  if (scaled >= 4294967296.0) return 4294967296ull;
  return static_cast<uint64_t>(scaled);
}

sbw_status_t check_device() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    g_last_hip_error = e;
    (void)hipGetLastError();
    return SBW_ERR_NO_DEVICE;
  }
  return SBW_OK;
}

sbw_status_t after_launch() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_last_hip_error = e;
    return SBW_ERR_HIP;
  }
  return SBW_OK;
}

int64_t grid_for(int64_t work_groups) { return work_groups < kMaxGrid ? work_groups : kMaxGrid; }

bool valid_seeding(int s) { return s == SBW_SEED_CONTEXT || s == SBW_SEED_SELF_SALT; }

sbw_status_t check_width(int64_t width) {
  if (width < 1) return SBW_ERR_INVALID_ARG;
  if (width > kMaxWidth) return SBW_ERR_UNSUPPORTED;
  return SBW_OK;
}

// Vectors per lane.  Two in flight per lane measured best for the context pass (~80 %
// of HBM peak; one per lane: ~75 %) and for fp32 self-salt (two independent sets of
// Philox chains per lane); bf16 self-salt does best with one (8 tokens) per lane and
// row groups that load their successor while drawing.
template <int kSeeding, typename T>
constexpr int unroll_for() {
  return kSeeding == kContext
             ? (sizeof(T) == 4 ? SBW_CONTEXT_UNROLL : SBW_CONTEXT_UNROLL_BF16)
             : (sizeof(T) == 4 ? SBW_SELF_SALT_UNROLL : SBW_SELF_SALT_UNROLL_BF16);
}

template <typename T, int kSeeding, int kW>
void launch_watermark(void* logits, int64_t B, uint32_t V, int64_t row_stride,
                      const int32_t* context, int width, uint64_t key, uint32_t tm1, float delta,
                      uint32_t vbase, bool aligned, hipStream_t stream) {
  T* p = static_cast<T*>(logits);
  const uint32_t rows = static_cast<uint32_t>(B < kMaxGridY ? B : kMaxGridY);
  if (aligned) {
    constexpr int kU = unroll_for<kSeeding, T>();
    constexpr uint32_t kPer = 16u / sizeof(T);
    const uint64_t vectors = (static_cast<uint64_t>(V) + kPer - 1) / kPer;
    const uint32_t tiles = static_cast<uint32_t>((vectors + kThreads * kU - 1) / (kThreads * kU));
    if constexpr (kSeeding == kSelfSalt) {
      if constexpr (SBW_SELF_SALT_SLAB && kW == 1) {
        const uint32_t tiles1 = static_cast<uint32_t>((vectors + kThreads - 1) / kThreads);
        const int64_t slabs12 = (B + 11) / 12, slabs8 = (B + 7) / 8, slabs6 = (B + 5) / 6;
        if (static_cast<int64_t>(tiles1) * slabs12 >= int64_t{SBW_SLAB12_MIN_GROUPS}) {
          const dim3 grid(tiles1, static_cast<uint32_t>(slabs12 < kMaxGridY ? slabs12 : kMaxGridY));
          hipLaunchKernelGGL((watermark_ss_slab_kernel<T, 12>), grid, dim3(kThreads), 0, stream, p,
                             row_stride, V, B, context, key, tm1, delta, vbase);
          return;
        }
        if (static_cast<int64_t>(tiles1) * slabs8 >= int64_t{SBW_SLAB_MIN_GROUPS}) {
          const dim3 grid(tiles1, static_cast<uint32_t>(slabs8 < kMaxGridY ? slabs8 : kMaxGridY));
          hipLaunchKernelGGL((watermark_ss_slab_kernel<T, 8>), grid, dim3(kThreads), 0, stream, p,
                             row_stride, V, B, context, key, tm1, delta, vbase);
          return;
        }
        if (static_cast<int64_t>(tiles1) * slabs6 >= int64_t{SBW_SLAB_MIN_GROUPS}) {
          const dim3 grid(tiles1, static_cast<uint32_t>(slabs6 < kMaxGridY ? slabs6 : kMaxGridY));
          hipLaunchKernelGGL((watermark_ss_slab_kernel<T, 6>), grid, dim3(kThreads), 0, stream, p,
                             row_stride, V, B, context, key, tm1, delta, vbase);
          return;
        }
      }
      constexpr int kMaxRows = kW > 1 ? 1 : (sizeof(T) == 4 ? 4 : 2);
      const int64_t work = static_cast<int64_t>(tiles) * B;
      if constexpr (kMaxRows == 4) {
        // fp32, width 1: 4-row groups take one vector per lane, whenever that makes
        // SBW_SELF_SALT_MIN_GROUPS workgroups (the narrower tiles keep more of them
        // resident at once than two vectors per lane do)
        const uint32_t tiles1 = static_cast<uint32_t>((vectors + kThreads - 1) / kThreads);
        if (static_cast<int64_t>(tiles1) * B >= 4 * int64_t{SBW_SELF_SALT_MIN_GROUPS}) {
          const int64_t groups = (B + 3) / 4;
          const dim3 grid(tiles1, static_cast<uint32_t>(groups < kMaxGridY ? groups : kMaxGridY));
          hipLaunchKernelGGL((watermark_ss_rows_kernel<T, 1, kW, 4, false>), grid, dim3(kThreads),
                             0, stream, p, row_stride, V, B, context, width, key, tm1, delta,
                             vbase);
          return;
        }
      }
      const int rows_per_group =
          (kMaxRows >= 2 && work >= 2 * int64_t{SBW_SELF_SALT_MIN_GROUPS}) ? 2 : 1;
      const int64_t groups = (B + rows_per_group - 1) / rows_per_group;
      // Each workgroup takes up to kIters groups while that still leaves
      // SBW_SELF_SALT_MIN_GROUPS workgroups.
      int64_t slots = groups;
      constexpr int kIters = sizeof(T) == 4 ? SBW_SELF_SALT_GROUP_ITERS : SBW_SELF_SALT_GROUP_ITERS_BF16;
      for (int it = kIters; it > 1; --it) {
        const int64_t s2 = (groups + it - 1) / it;
        if (s2 * tiles >= int64_t{SBW_SELF_SALT_MIN_GROUPS}) { slots = s2; break; }
      }
      const dim3 grid(tiles, static_cast<uint32_t>(slots < kMaxGridY ? slots : kMaxGridY));
      constexpr bool kPf = (sizeof(T) == 4 ? SBW_SELF_SALT_PREFETCH : SBW_SELF_SALT_PREFETCH_BF16) != 0;
      if (kMaxRows >= 2 && rows_per_group == 2)
        hipLaunchKernelGGL((watermark_ss_rows_kernel<T, kU, kW, (kMaxRows >= 2 ? 2 : 1), kPf>), grid,
                           dim3(kThreads), 0, stream, p, row_stride, V, B, context, width, key, tm1,
                           delta, vbase);
      else
        hipLaunchKernelGGL((watermark_ss_rows_kernel<T, kU, kW, 1, kPf>), grid, dim3(kThreads), 0,
                           stream, p, row_stride, V, B, context, width, key, tm1, delta, vbase);
    } else {
      // whole rows per XCD for large launches (one launch row per grid row, workgroup
      // numbers below 2^32)
      const uint32_t xcd_rows =
          B >= SBW_XCD_ROWS_MIN && B % 8 == 0 && B <= kMaxGridY &&
                  B * static_cast<int64_t>(V) * static_cast<int64_t>(sizeof(T)) >= SBW_XCD_ROWS_MIN_BYTES &&
                  static_cast<uint64_t>(tiles) * static_cast<uint64_t>(B) < (uint64_t{1} << 32)
              ? 1u
              : 0u;
      hipLaunchKernelGGL((watermark_vec_kernel<T, kU, kW>), dim3(tiles, rows),
                         dim3(kThreads), 0, stream, p, row_stride, V, B, context, width, key, tm1,
                         delta, vbase, xcd_rows);
    }
  } else {
    const uint32_t tiles = static_cast<uint32_t>((static_cast<uint64_t>(V) + kThreads - 1) / kThreads);
    hipLaunchKernelGGL((watermark_elem_kernel<T, kSeeding, kW>), dim3(tiles, rows), dim3(kThreads),
                       0, stream, p, row_stride, V, B, context, width, key, tm1, delta, vbase);
  }
}

template <typename T>
void dispatch_watermark(void* logits, int64_t B, uint32_t V, int64_t row_stride,
                        const int32_t* context, int width, uint64_t key, uint32_t tm1, float delta,
                        sbw_seeding_t seeding, uint32_t vbase, bool aligned, hipStream_t st) {
  // Context seeding folds any window into one row seed; self-salt needs the window
  // per candidate, so wider windows take the kMaxWidth instantiation.
  if (seeding == SBW_SEED_CONTEXT)
    launch_watermark<T, kContext, kMaxWidth>(logits, B, V, row_stride, context, width, key, tm1,
                                             delta, vbase, aligned, st);
  else if (width == 1)
    launch_watermark<T, kSelfSalt, 1>(logits, B, V, row_stride, context, width, key, tm1, delta,
                                      vbase, aligned, st);
  else if (width <= kMidWidth)
    launch_watermark<T, kSelfSalt, kMidWidth>(logits, B, V, row_stride, context, width, key, tm1,
                                              delta, vbase, aligned, st);
  else
    launch_watermark<T, kSelfSalt, kMaxWidth>(logits, B, V, row_stride, context, width, key, tm1,
                                              delta, vbase, aligned, st);
}

template <typename T>
void dispatch_candidates(void* logits, int64_t B, uint32_t V, int64_t row_stride,
                         const int32_t* cand, int k, const int32_t* context, int width,
                         uint64_t key, uint32_t tm1, float delta, sbw_seeding_t seeding,
                         hipStream_t st) {
  T* p = static_cast<T*>(logits);
  const dim3 grid(static_cast<uint32_t>(grid_for(B)));
  if (seeding == SBW_SEED_CONTEXT)
    hipLaunchKernelGGL((candidates_kernel<T, kContext, kMaxWidth>), grid, dim3(kThreads), 0, st, p,
                       row_stride, V, B, cand, k, context, width, key, tm1, delta);
  else if (width == 1)
    hipLaunchKernelGGL((candidates_kernel<T, kSelfSalt, 1>), grid, dim3(kThreads), 0, st, p,
                       row_stride, V, B, cand, k, context, width, key, tm1, delta);
  else if (width <= kMidWidth)
    hipLaunchKernelGGL((candidates_kernel<T, kSelfSalt, kMidWidth>), grid, dim3(kThreads), 0, st,
                       p, row_stride, V, B, cand, k, context, width, key, tm1, delta);
  else
    hipLaunchKernelGGL((candidates_kernel<T, kSelfSalt, kMaxWidth>), grid, dim3(kThreads), 0, st,
                       p, row_stride, V, B, cand, k, context, width, key, tm1, delta);
}

// Segments per row of the fused decoding: vector path and element path.
template <typename T>
constexpr int decode_vecs_for(bool sample) {
  return sizeof(T) == 4 ? (sample ? SBW_DECODE_VECS_F32 : SBW_DECODE_VECS_F32_GREEDY)
                        : (sample ? SBW_DECODE_VECS_BF16_SAMPLE : SBW_DECODE_VECS_BF16);
}
template <typename T>
constexpr uint64_t vec_segment_elems(int kN) { return (16u / sizeof(T)) * kThreads * kN; }
// Small grids: a launch of fewer workgroups than this takes half the vectors per lane
// (twice the segments), which hides more of the load latency when the chip is not
// full: a vocabulary shard of 19008 fp32 or bf16 logits at B = 256 gets 1280
// workgroups instead of 768 (about 8 % faster); B = 64 rows of 152064 (960-1600
// workgroups) stay.
constexpr int64_t kSmallDecodeGrid = 900;
// The workspace is sized for the element path; vector segments must be at least as long.
static_assert(vec_segment_elems<float>(SBW_DECODE_VECS_F32 / 2) >= kArgmaxSegElems &&
                  vec_segment_elems<float>(SBW_DECODE_VECS_F32_GREEDY / 2) >= kArgmaxSegElems &&
                  vec_segment_elems<uint16_t>(SBW_DECODE_VECS_BF16 / 2) >= kArgmaxSegElems &&
                  vec_segment_elems<uint16_t>(SBW_DECODE_VECS_BF16_SAMPLE / 2) >= kArgmaxSegElems,
              "vector segments must not outnumber element segments");

// The per-row noise seeds and 1/T of a sampling pass (unused by greedy decoding).
struct SampleArgs {
  const uint64_t* seeds;
  float inv_t;
};

template <typename T, int kSeeding, int kW, bool kSample>
void launch_argmax(const void* logits, int64_t B, uint32_t V, int64_t row_stride,
                   const int32_t* context, int width, uint64_t key, uint32_t tm1, int none,
                   float delta, const SampleArgs& sa, uint32_t vbase, bool aligned, int32_t* tokens,
                   float* values, uint64_t* partials, hipStream_t stream) {
  const T* p = static_cast<const T*>(logits);
  const uint32_t rows = static_cast<uint32_t>(B < kMaxGridY ? B : kMaxGridY);
  uint32_t segments;
  if (aligned) {
    constexpr int kN = decode_vecs_for<T>(kSample);
    constexpr int kNs = kN / 2;
    const uint64_t seg = vec_segment_elems<T>(kN) * SBW_DECODE_SUBS;
    segments = static_cast<uint32_t>((static_cast<uint64_t>(V) + seg - 1) / seg);
    if (int64_t{segments} * rows >= kSmallDecodeGrid) {
      hipLaunchKernelGGL((decode_vec_kernel<T, kSeeding, kN, SBW_DECODE_SUBS, kW, kSample>),
                         dim3(segments, rows), dim3(kThreads), 0, stream, p, row_stride, V, B,
                         context, width, key, tm1, none, delta, sa.seeds, sa.inv_t, segments,
                         partials, vbase);
    } else {
      const uint64_t seg_s = vec_segment_elems<T>(kNs) * SBW_DECODE_SUBS;
      segments = static_cast<uint32_t>((static_cast<uint64_t>(V) + seg_s - 1) / seg_s);
      hipLaunchKernelGGL((decode_vec_kernel<T, kSeeding, kNs, SBW_DECODE_SUBS, kW, kSample>),
                         dim3(segments, rows), dim3(kThreads), 0, stream, p, row_stride, V, B,
                         context, width, key, tm1, none, delta, sa.seeds, sa.inv_t, segments,
                         partials, vbase);
    }
  } else {
    segments = static_cast<uint32_t>((static_cast<uint64_t>(V) + kArgmaxSegElems - 1) /
                                     kArgmaxSegElems);
    hipLaunchKernelGGL((argmax_elem_kernel<T, kSeeding, kW, kSample>), dim3(segments, rows),
                       dim3(kThreads), 0, stream, p, row_stride, V, B, context, width, key, tm1,
                       none, delta, sa.seeds, sa.inv_t, segments, partials, vbase);
  }
  const int64_t row_blocks = grid_for((B + kThreads / 64 - 1) / (kThreads / 64));
  hipLaunchKernelGGL(argmax_finish_kernel, dim3(row_blocks), dim3(kThreads), 0, stream, partials,
                     segments, B, tokens, values);
}

template <typename T, bool kSample>
void dispatch_argmax(const void* logits, int64_t B, uint32_t V, int64_t row_stride,
                     const int32_t* context, int width, uint64_t key, uint32_t tm1, int none,
                     float delta, const SampleArgs& sa, sbw_seeding_t seeding, uint32_t vbase,
                     bool aligned, int32_t* tokens, float* values, uint64_t* partials,
                     hipStream_t st) {
  if (seeding == SBW_SEED_CONTEXT)
    launch_argmax<T, kContext, kMaxWidth, kSample>(logits, B, V, row_stride, context, width, key,
                                                   tm1, none, delta, sa, vbase, aligned, tokens,
                                                   values, partials, st);
  else if (width == 1)
    launch_argmax<T, kSelfSalt, 1, kSample>(logits, B, V, row_stride, context, width, key, tm1,
                                            none, delta, sa, vbase, aligned, tokens, values,
                                            partials, st);
  else if (width <= kMidWidth)
    launch_argmax<T, kSelfSalt, kMidWidth, kSample>(logits, B, V, row_stride, context, width, key,
                                                    tm1, none, delta, sa, vbase, aligned, tokens,
                                                    values, partials, st);
  else
    launch_argmax<T, kSelfSalt, kMaxWidth, kSample>(logits, B, V, row_stride, context, width, key,
                                                    tm1, none, delta, sa, vbase, aligned, tokens,
                                                    values, partials, st);
}

template <int kSeeding, int kW>
void launch_detect(int64_t positions, hipStream_t st, const int32_t* tokens, int64_t N, int64_t L,
                   int64_t row_stride, int width, uint64_t key, uint32_t tm1, double gamma,
                   const DetectIO& io) {
  const int64_t blocks = grid_for((N + kWavesPerBlock - 1) / kWavesPerBlock);
  if (positions <= kWave)
    hipLaunchKernelGGL((detect_kernel<kSeeding, 1, kW>), dim3(blocks), dim3(kThreads), 0, st,
                       tokens, N, L, row_stride, width, key, tm1, gamma, io);
  else if (positions <= 2 * kWave)
    hipLaunchKernelGGL((detect_kernel<kSeeding, 2, kW>), dim3(blocks), dim3(kThreads), 0, st,
                       tokens, N, L, row_stride, width, key, tm1, gamma, io);
  else if (positions <= 4 * kWave || kW > kMidWidth)   // windows of 5-8: 4 chunks (registers)
    hipLaunchKernelGGL((detect_kernel<kSeeding, 4, kW>), dim3(blocks), dim3(kThreads), 0, st,
                       tokens, N, L, row_stride, width, key, tm1, gamma, io);
  else
    hipLaunchKernelGGL((detect_kernel<kSeeding, 8, kW>), dim3(blocks), dim3(kThreads), 0, st,
                       tokens, N, L, row_stride, width, key, tm1, gamma, io);
}

template <int kSeeding, int kW>
void launch_detect_unique(int64_t N, hipStream_t st, const int32_t* tokens, int64_t L,
                          int64_t row_stride, int width, uint64_t key, uint32_t tm1, double gamma,
                          uint32_t slots, const DetectIO& io) {
  const size_t lds = (static_cast<size_t>(slots) + static_cast<size_t>(L)) * sizeof(int32_t);
  hipLaunchKernelGGL((detect_unique_kernel<kSeeding, kW>), dim3(static_cast<uint32_t>(grid_for(N))),
                     dim3(kUniqueBlock), lds, st, tokens, N, L, row_stride, width, key, tm1, gamma,
                     slots, io);
}

// Every detect entry point: validation, then one launch.
sbw_status_t detect_impl(const int32_t* tokens, int64_t N, int64_t L, int64_t row_stride,
                         const int32_t* lengths, int64_t width, uint64_t key, double gamma,
                         sbw_seeding_t seeding, uint32_t flags, int32_t* green_counts,
                         int32_t* scored, double* z, hipStream_t st) {
  if (N < 0 || L < 0 || row_stride < L) return SBW_ERR_INVALID_ARG;
  sbw_status_t s = check_width(width);
  if (s != SBW_OK) return s;
  if (!valid_seeding(seeding)) return SBW_ERR_UNSUPPORTED;
  if ((flags & ~static_cast<uint32_t>(SBW_DETECT_IGNORE_REPEATED)) != 0u) return SBW_ERR_UNSUPPORTED;
  if (!(gamma > 0.0 && gamma < 1.0)) return SBW_ERR_GAMMA;
  if (L > INT32_MAX) return SBW_ERR_UNSUPPORTED;
  const bool unique = (flags & SBW_DETECT_IGNORE_REPEATED) != 0u;
  const int64_t positions = L > width ? L - width : 0;
  if (unique && 2 * positions > static_cast<int64_t>(kMaxUniqueSlots)) return SBW_ERR_UNSUPPORTED;
  if (N == 0) return SBW_OK;
  if (green_counts == nullptr || z == nullptr || (L > 0 && tokens == nullptr))
    return SBW_ERR_INVALID_ARG;
  if (row_stride > 0 && N > INT64_MAX / 4 / row_stride) return SBW_ERR_UNSUPPORTED;
  s = check_device();
  if (s != SBW_OK) return s;

  const uint64_t T = threshold_of(gamma);  // in [1, 2^32 - 1] for 0 < gamma < 1
  const uint32_t tm1 = static_cast<uint32_t>(T - 1);
  const int w = static_cast<int>(width);
  const DetectIO io{lengths, green_counts, scored, z};
  const bool ctx = seeding == SBW_SEED_CONTEXT;
  if (unique) {
    // a power of two, four times the scored positions where it fits, at least twice
    uint32_t slots = 64u;
    while (slots < 4 * positions && slots < kMaxUniqueSlots) slots *= 2u;
    if (w == 1) {
      if (ctx) launch_detect_unique<kContext, 1>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
      else launch_detect_unique<kSelfSalt, 1>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
    } else if (w <= kMidWidth) {
      if (ctx) launch_detect_unique<kContext, kMidWidth>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
      else launch_detect_unique<kSelfSalt, kMidWidth>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
    } else {
      if (ctx) launch_detect_unique<kContext, kMaxWidth>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
      else launch_detect_unique<kSelfSalt, kMaxWidth>(N, st, tokens, L, row_stride, w, key, tm1, gamma, slots, io);
    }
    return after_launch();
  }
  if (w == 1) {
    if (ctx) launch_detect<kContext, 1>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
    else launch_detect<kSelfSalt, 1>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
  } else if (w <= kMidWidth) {
    if (ctx) launch_detect<kContext, kMidWidth>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
    else launch_detect<kSelfSalt, kMidWidth>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
  } else {
    if (ctx) launch_detect<kContext, kMaxWidth>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
    else launch_detect<kSelfSalt, kMaxWidth>(positions, st, tokens, N, L, row_stride, w, key, tm1, gamma, io);
  }
  return after_launch();
}

// Token ids are 32-bit: a row holds fewer than 2^32 columns (its length is a 32-bit
// count), and a shard's last id, v_offset + V - 1, must fit.  v_offset >= 0.
constexpr int64_t kMaxTokenIds = int64_t{1} << 32;
bool ids_fit(int64_t V, int64_t v_offset) {
  return V < kMaxTokenIds && v_offset <= kMaxTokenIds - V;
}

// The vector kernels load 16 bytes per lane and draw whole Philox blocks: rows must
// start on 16 bytes, and the shard's first token id must sit at the start of a vector
// (a multiple of 4 for fp32, of 8 for bf16).  Anything else takes the element path.
bool vector_path_ok(const void* logits, int64_t row_stride, sbw_dtype_t dtype, uint32_t vbase) {
  const uint32_t esize = dtype == SBW_F32 ? 4u : 2u;
  return reinterpret_cast<uintptr_t>(logits) % 16 == 0 &&
         (static_cast<uint64_t>(row_stride) * esize) % 16 == 0 && vbase % (16u / esize) == 0;
}

// ---------------------------------------------------------------------------
// Scratch of sbw_watermark_argmax_noalloc: the per-segment partials that the other
// decoding calls keep in the caller's workspace, in an array of the code object, one
// copy per device, shared by every call on that device.  In host code the name is
// only a handle: the array's device address comes from hipGetSymbolAddress, resolved
// once per device with that device current, and only that address reaches a kernel.
// ---------------------------------------------------------------------------
constexpr int64_t kScratchElems = int64_t{1} << 18;  // uint64 partials: 2 MiB
static_assert(kScratchElems == SBW_NOALLOC_SCRATCH_ELEMS, "the header states the limit");
constexpr int kMaxDevices = 64;
std::atomic<uint64_t*> g_scratch_of_device[kMaxDevices];

}  // namespace
}  // namespace sbw

static __device__ __align__(256) uint64_t scratch[sbw::kScratchElems];

namespace sbw {
namespace {

// The device address of `scratch` on the current device (resolved on the first call
// made on that device).
sbw_status_t scratch_address(uint64_t** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    g_last_hip_error = e;
    (void)hipGetLastError();
    return SBW_ERR_NO_DEVICE;
  }
  if (dev < 0 || dev >= kMaxDevices) return SBW_ERR_UNSUPPORTED;
  uint64_t* p = g_scratch_of_device[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    void* addr = nullptr;
    e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || addr == nullptr) {
      g_last_hip_error = e != hipSuccess ? e : hipErrorInvalidSymbol;
      (void)hipGetLastError();
      return SBW_ERR_HIP;
    }
    p = static_cast<uint64_t*>(addr);
    // every thread that resolves it gets the same address, so a race only repeats work
    g_scratch_of_device[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return SBW_OK;
}

// Greedy decoding and sampling: validation, then the segment pass and the read-out.
// With use_scratch the partials go to the device's `scratch` array instead of
// `workspace` (which may then be null).
template <bool kSample>
sbw_status_t decode_impl(const void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                         int64_t row_stride, const int32_t* context, int64_t width,
                         int64_t v_offset, uint64_t key, double gamma, float delta,
                         sbw_seeding_t seeding, const SampleArgs& sa, int32_t* tokens,
                         float* values, uint64_t* workspace, void* stream,
                         bool use_scratch = false) {
  if (B < 0 || V < 0 || row_stride < V || v_offset < 0) return SBW_ERR_INVALID_ARG;
  sbw_status_t s = check_width(width);
  if (s != SBW_OK) return s;
  if (dtype != SBW_F32 && dtype != SBW_BF16) return SBW_ERR_UNSUPPORTED;
  if (!valid_seeding(seeding)) return SBW_ERR_UNSUPPORTED;
  if (!(gamma >= 0.0 && gamma <= 1.0)) return SBW_ERR_GAMMA;
  if (!isfinite(delta)) return SBW_ERR_DELTA;
  if (!ids_fit(V, v_offset)) return SBW_ERR_UNSUPPORTED;
  if (B == 0) return SBW_OK;
  if (V == 0) return SBW_ERR_INVALID_ARG;  // no token to choose
  if (logits == nullptr || context == nullptr || tokens == nullptr ||
      (workspace == nullptr && !use_scratch))
    return SBW_ERR_INVALID_ARG;
  if (B > INT64_MAX / 4 / row_stride) return SBW_ERR_UNSUPPORTED;
  s = check_device();
  if (s != SBW_OK) return s;
  if (use_scratch) {
    s = scratch_address(&workspace);
    if (s != SBW_OK) return s;
  }

  // gamma == 0: nothing is green, every logit (and the value returned) is unchanged.
  const uint64_t T = threshold_of(gamma);
  const int none = T == 0 ? 1 : 0;
  const uint32_t tm1 = none ? 0u : static_cast<uint32_t>(T - 1);
  const float d = delta;
  const uint32_t vbase = static_cast<uint32_t>(v_offset);
  const bool aligned = vector_path_ok(logits, row_stride, dtype, vbase);
  const uint32_t v32 = static_cast<uint32_t>(V);
  const int w = static_cast<int>(width);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == SBW_F32)
    dispatch_argmax<float, kSample>(logits, B, v32, row_stride, context, w, key, tm1, none, d, sa,
                                    seeding, vbase, aligned, tokens, values, workspace, st);
  else
    dispatch_argmax<uint16_t, kSample>(logits, B, v32, row_stride, context, w, key, tm1, none, d,
                                       sa, seeding, vbase, aligned, tokens, values, workspace, st);
  return after_launch();
}

}  // namespace
}  // namespace sbw

using namespace sbw;

extern "C" {

sbw_status_t sbw_watermark_shard(void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                 int64_t row_stride, const int32_t* context, int64_t width,
                                 int64_t v_offset, uint64_t key, double gamma, float delta,
                                 sbw_seeding_t seeding, void* stream) {
  if (B < 0 || V < 0 || row_stride < V || v_offset < 0) return SBW_ERR_INVALID_ARG;
  sbw_status_t s = check_width(width);
  if (s != SBW_OK) return s;
  if (dtype != SBW_F32 && dtype != SBW_BF16) return SBW_ERR_UNSUPPORTED;
  if (!valid_seeding(seeding)) return SBW_ERR_UNSUPPORTED;
  if (!(gamma >= 0.0 && gamma <= 1.0)) return SBW_ERR_GAMMA;
  if (!isfinite(delta)) return SBW_ERR_DELTA;
  if (!ids_fit(V, v_offset)) return SBW_ERR_UNSUPPORTED;  // token ids are 32-bit
  if (B == 0 || V == 0) return SBW_OK;
  if (logits == nullptr || context == nullptr) return SBW_ERR_INVALID_ARG;
  if (B > INT64_MAX / 4 / row_stride) return SBW_ERR_UNSUPPORTED;
  const uint64_t T = threshold_of(gamma);
  if (T == 0) return SBW_OK;  // nothing is green: the logits stay as they are
  s = check_device();
  if (s != SBW_OK) return s;

  const uint32_t vbase = static_cast<uint32_t>(v_offset);
  const bool aligned = vector_path_ok(logits, row_stride, dtype, vbase);
  const uint32_t tm1 = static_cast<uint32_t>(T - 1);
  const uint32_t v32 = static_cast<uint32_t>(V);
  const int w = static_cast<int>(width);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == SBW_F32)
    dispatch_watermark<float>(logits, B, v32, row_stride, context, w, key, tm1, delta, seeding,
                              vbase, aligned, st);
  else
    dispatch_watermark<uint16_t>(logits, B, v32, row_stride, context, w, key, tm1, delta, seeding,
                                 vbase, aligned, st);
  return after_launch();
}

sbw_status_t sbw_watermark_window(void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t* context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  void* stream) {
  return sbw_watermark_shard(logits, dtype, B, V, row_stride, context, width, 0, key, gamma, delta,
                             seeding, stream);
}

sbw_status_t sbw_watermark(void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                           int64_t row_stride, const int32_t* prev_tokens, uint64_t key,
                           double gamma, float delta, sbw_seeding_t seeding, void* stream) {
  return sbw_watermark_window(logits, dtype, B, V, row_stride, prev_tokens, 1, key, gamma, delta,
                              seeding, stream);
}

sbw_status_t sbw_watermark_candidates(void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                      int64_t row_stride, const int32_t* candidates, int64_t k,
                                      const int32_t* context, int64_t width, uint64_t key,
                                      double gamma, float delta, sbw_seeding_t seeding,
                                      void* stream) {
  if (B < 0 || V < 0 || row_stride < V || k < 0) return SBW_ERR_INVALID_ARG;
  sbw_status_t s = check_width(width);
  if (s != SBW_OK) return s;
  if (dtype != SBW_F32 && dtype != SBW_BF16) return SBW_ERR_UNSUPPORTED;
  if (!valid_seeding(seeding)) return SBW_ERR_UNSUPPORTED;
  if (!(gamma >= 0.0 && gamma <= 1.0)) return SBW_ERR_GAMMA;
  if (!isfinite(delta)) return SBW_ERR_DELTA;
  if (V >= (int64_t{1} << 32) || k > kMaxCandidates) return SBW_ERR_UNSUPPORTED;
  if (B == 0 || V == 0 || k == 0) return SBW_OK;
  if (logits == nullptr || candidates == nullptr || context == nullptr) return SBW_ERR_INVALID_ARG;
  if (B > INT64_MAX / 4 / row_stride) return SBW_ERR_UNSUPPORTED;
  const uint64_t T = threshold_of(gamma);
  if (T == 0) return SBW_OK;  // nothing is green
  s = check_device();
  if (s != SBW_OK) return s;

  const uint32_t tm1 = static_cast<uint32_t>(T - 1);
  const uint32_t v32 = static_cast<uint32_t>(V);
  const int w = static_cast<int>(width);
  const int kk = static_cast<int>(k);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == SBW_F32)
    dispatch_candidates<float>(logits, B, v32, row_stride, candidates, kk, context, w, key, tm1,
                               delta, seeding, st);
  else
    dispatch_candidates<uint16_t>(logits, B, v32, row_stride, candidates, kk, context, w, key,
                                  tm1, delta, seeding, st);
  return after_launch();
}

sbw_status_t sbw_watermark_argmax(const void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t* context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  int32_t* tokens, float* values, uint64_t* workspace,
                                  void* stream) {
  return decode_impl<false>(logits, dtype, B, V, row_stride, context, width, 0, key, gamma, delta,
                            seeding, SampleArgs{nullptr, 1.0f}, tokens, values, workspace, stream);
}

sbw_status_t sbw_watermark_argmax_shard(const void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                        int64_t row_stride, const int32_t* context, int64_t width,
                                        int64_t v_offset, uint64_t key, double gamma, float delta,
                                        sbw_seeding_t seeding, int32_t* tokens, float* values,
                                        uint64_t* workspace, void* stream) {
  return decode_impl<false>(logits, dtype, B, V, row_stride, context, width, v_offset, key, gamma,
                            delta, seeding, SampleArgs{nullptr, 1.0f}, tokens, values, workspace,
                            stream);
}

sbw_status_t sbw_watermark_sample(const void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                  int64_t row_stride, const int32_t* context, int64_t width,
                                  uint64_t key, double gamma, float delta, sbw_seeding_t seeding,
                                  const uint64_t* seeds, float inv_temperature, int32_t* tokens,
                                  float* scores, uint64_t* workspace, void* stream) {
  return sbw_watermark_sample_shard(logits, dtype, B, V, row_stride, context, width, 0, key, gamma,
                                    delta, seeding, seeds, inv_temperature, tokens, scores,
                                    workspace, stream);
}

sbw_status_t sbw_watermark_sample_shard(const void* logits, sbw_dtype_t dtype, int64_t B, int64_t V,
                                        int64_t row_stride, const int32_t* context, int64_t width,
                                        int64_t v_offset, uint64_t key, double gamma, float delta,
                                        sbw_seeding_t seeding, const uint64_t* seeds,
                                        float inv_temperature, int32_t* tokens, float* scores,
                                        uint64_t* workspace, void* stream) {
  if (!(isfinite(inv_temperature) && inv_temperature > 0.0f)) return SBW_ERR_INVALID_ARG;
  if (B > 0 && V > 0 && seeds == nullptr) return SBW_ERR_INVALID_ARG;
  return decode_impl<true>(logits, dtype, B, V, row_stride, context, width, v_offset, key, gamma,
                           delta, seeding, SampleArgs{seeds, inv_temperature}, tokens, scores,
                           workspace, stream);
}

sbw_status_t sbw_watermark_argmax_noalloc(const void* logits, sbw_dtype_t dtype, int64_t B,
                                          int64_t V, int64_t row_stride, const int32_t* context,
                                          int64_t width, uint64_t key, double gamma, float delta,
                                          sbw_seeding_t seeding, int32_t* tokens, float* values,
                                          void* stream) {
  // The partials must fit the static array: B * ceil(V / kArgmaxSegElems) elements,
  // compared by division so that no product overflows.
  if (B > 0 && V > 0 && B > kScratchElems / ((V + kArgmaxSegElems - 1) / kArgmaxSegElems))
    return SBW_ERR_UNSUPPORTED;
  return decode_impl<false>(logits, dtype, B, V, row_stride, context, width, 0, key, gamma, delta,
                            seeding, SampleArgs{nullptr, 1.0f}, tokens, values, nullptr, stream,
                            /*use_scratch=*/true);
}

int64_t sbw_watermark_argmax_workspace(int64_t B, int64_t V) {
  if (B <= 0 || V <= 0) return 0;
  // the element path has the most segments per row (the vector paths fewer)
  return B * ((V + kArgmaxSegElems - 1) / kArgmaxSegElems);
}

sbw_status_t sbw_green_mask_window(uint32_t* bits, int64_t B, int64_t V, const int32_t* context,
                                   int64_t width, uint64_t key, double gamma,
                                   sbw_seeding_t seeding, void* stream) {
  if (B < 0 || V < 0) return SBW_ERR_INVALID_ARG;
  sbw_status_t s = check_width(width);
  if (s != SBW_OK) return s;
  if (!valid_seeding(seeding)) return SBW_ERR_UNSUPPORTED;
  if (!(gamma >= 0.0 && gamma <= 1.0)) return SBW_ERR_GAMMA;
  if (V >= (int64_t{1} << 32)) return SBW_ERR_UNSUPPORTED;
  if (B == 0 || V == 0) return SBW_OK;
  if (bits == nullptr || context == nullptr) return SBW_ERR_INVALID_ARG;
  const int64_t words = (V + 31) / 32;
  if (B > INT64_MAX / 4 / words) return SBW_ERR_UNSUPPORTED;
  s = check_device();
  if (s != SBW_OK) return s;

  const uint64_t T = threshold_of(gamma);
  const uint32_t tm1 = T == 0 ? 0u : static_cast<uint32_t>(T - 1);
  const int64_t num_words = B * words;
  const int64_t blocks = grid_for((num_words + kThreads - 1) / kThreads);
  const int w = static_cast<int>(width);
  const int none = T == 0 ? 1 : 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint32_t v32 = static_cast<uint32_t>(V), wpr = static_cast<uint32_t>(words);
  if (seeding == SBW_SEED_CONTEXT)
    hipLaunchKernelGGL((green_mask_kernel<kContext, kMaxWidth>), dim3(blocks), dim3(kThreads), 0,
                       st, bits, v32, wpr, context, w, key, tm1, none, num_words);
  else if (w == 1)
    hipLaunchKernelGGL((green_mask_kernel<kSelfSalt, 1>), dim3(blocks), dim3(kThreads), 0, st,
                       bits, v32, wpr, context, w, key, tm1, none, num_words);
  else
    hipLaunchKernelGGL((green_mask_kernel<kSelfSalt, kMaxWidth>), dim3(blocks), dim3(kThreads), 0,
                       st, bits, v32, wpr, context, w, key, tm1, none, num_words);
  return after_launch();
}

sbw_status_t sbw_green_mask(uint32_t* bits, int64_t B, int64_t V, const int32_t* prev_tokens,
                            uint64_t key, double gamma, sbw_seeding_t seeding, void* stream) {
  return sbw_green_mask_window(bits, B, V, prev_tokens, 1, key, gamma, seeding, stream);
}

sbw_status_t sbw_detect_window(const int32_t* tokens, int64_t N, int64_t L, int64_t row_stride,
                               int64_t width, uint64_t key, double gamma, sbw_seeding_t seeding,
                               int32_t* green_counts, double* z, void* stream) {
  return detect_impl(tokens, N, L, row_stride, nullptr, width, key, gamma, seeding, 0u,
                     green_counts, nullptr, z, static_cast<hipStream_t>(stream));
}

sbw_status_t sbw_detect_ex(const int32_t* tokens, int64_t N, int64_t L, int64_t row_stride,
                           const int32_t* lengths, int64_t width, uint64_t key, double gamma,
                           sbw_seeding_t seeding, uint32_t flags, int32_t* green_counts,
                           int32_t* scored, double* z, void* stream) {
  return detect_impl(tokens, N, L, row_stride, lengths, width, key, gamma, seeding, flags,
                     green_counts, scored, z, static_cast<hipStream_t>(stream));
}

sbw_status_t sbw_detect(const int32_t* tokens, int64_t N, int64_t L, int64_t row_stride,
                        uint64_t key, double gamma, sbw_seeding_t seeding,
                        int32_t* green_counts, double* z, void* stream) {
  return sbw_detect_window(tokens, N, L, row_stride, 1, key, gamma, seeding, green_counts, z,
                           stream);
}

const char* sbw_strerror(sbw_status_t status) {
  switch (status) {
    case SBW_OK: return "success";
    case SBW_ERR_INVALID_ARG: return "invalid argument (null pointer, negative size or stride too small)";
    case SBW_ERR_GAMMA: return "gamma out of range";
    case SBW_ERR_DELTA: return "delta is not finite";
    case SBW_ERR_UNSUPPORTED: return "unsupported dtype, seeding, width or size";
    case SBW_ERR_NO_DEVICE: return "no HIP device available";
    case SBW_ERR_HIP: return "HIP runtime or launch error";
  }
  return "unknown status";
}

const char* sbw_last_hip_error(void) { return hipGetErrorName(g_last_hip_error); }

const char* sbw_version(void) { return "0.5.0"; }

}  // extern "C"
