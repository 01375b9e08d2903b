// Throughput probe of the Philox4x32-10 CBRNG on gfx950, for the benchmark's ALU
// roof.  Not part of libsbw's ABI: it is built into its own library (libsbw_rate.so)
// and only bench.py loads it.
//
// Every lane draws `iters` blocks in kChains independent chains.  Each block has a
// fresh per-lane key and the counter (c, 0, 0, 0): the shape of a full-vocabulary
// self-salt draw (Sec. 2.2), where the key changes from token to token, so the ten
// round keys are derived again for every block (18 key adds) and nothing can be
// hoisted out of the loop.  The four output words are folded into the chain's next
// key (w0 ^ w1, w2 ^ w3), which keeps every round live.  No memory is touched inside
// the loop.  Per block: 19 products (round 0 has one, the counter's other words being
// zero), 19 xors, 18 key adds and the 2 xors of the fold.
//
// Lane 0 of every workgroup also reads the shader-clock counter (s_memtime) and the
// constant-rate real-time counter (s_memrealtime) at its start and end, so the host
// can tell the core clock the probe ran at.
//
// A second kernel draws the same blocks through the library's per-lane-key block
// (sbw::philox_block_lane: rounds 1-8 in the fixed issue order products, key adds,
// xors), so the benchmark can report the better of the two orders.
//
// The same launch shape also times single instruction kinds (kChains independent
// dependency chains per lane, one instruction per link), so that the issue cost of
// each of the block's three instruction kinds, and of their mix, can be measured in
// lane-ops per compute-unit clock: 32x32->64-bit products (v_mad_u64_u32), three-input
// xors (v_bitop3_b32) and 32-bit adds, with vector operands, and the xor and the add
// with one scalar operand.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sbw_device.hpp"

namespace {

constexpr uint32_t kMulA = 0xD2511F53u;
constexpr uint32_t kMulB = 0xCD9E8D57u;
constexpr uint32_t kWeyl0 = 0x9E3779B9u;
constexpr uint32_t kWeyl1 = 0xBB67AE85u;
constexpr int kThreads = 256;
constexpr int kChains = 8;

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// One Philox4x32-10 block at counter (c, 0, 0, 0) under key (k0, k1); the key is
// replaced by (w0 ^ w1, w2 ^ w3) of the block.
__device__ __forceinline__ void block_fold(uint32_t c, uint32_t& key0, uint32_t& key1) {
  uint32_t k0 = key0, k1 = key1;
  uint32_t x0 = c, x1 = 0u, x2 = 0u, x3 = 0u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t pa = static_cast<uint64_t>(kMulA) * x0;
    const uint64_t pb = static_cast<uint64_t>(kMulB) * x2;
    const uint32_t y0 = xor3(static_cast<uint32_t>(pb >> 32), x1, k0);
    const uint32_t y1 = static_cast<uint32_t>(pb);
    const uint32_t y2 = xor3(static_cast<uint32_t>(pa >> 32), x3, k1);
    const uint32_t y3 = static_cast<uint32_t>(pa);
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    k0 += kWeyl0;
    k1 += kWeyl1;
  }
  key0 = x0 ^ x1;
  key1 = x2 ^ x3;
}

__global__ void __launch_bounds__(kThreads)
philox_rate_kernel(uint32_t* __restrict__ out, uint64_t* __restrict__ clocks, int iters,
                   uint32_t salt) {
  uint64_t t0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    r0 = __builtin_amdgcn_s_memrealtime();
    t0 = __builtin_amdgcn_s_memtime();
  }
  const uint32_t lane = blockIdx.x * kThreads + threadIdx.x;
  uint32_t k0[kChains], k1[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) {
    k0[c] = lane ^ (static_cast<uint32_t>(c) << 24) ^ salt;
    k1[c] = lane * 0x9E3779B1u + static_cast<uint32_t>(c);
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) block_fold(static_cast<uint32_t>(i), k0[c], k1[c]);
  }
  uint32_t acc = 0u;
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc ^= k0[c] ^ k1[c];
  out[lane] = acc;
  if (threadIdx.x == 0) {
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clocks[4 * blockIdx.x + 0] = t0;
    clocks[4 * blockIdx.x + 1] = t1;
    clocks[4 * blockIdx.x + 2] = r0;
    clocks[4 * blockIdx.x + 3] = r1;
  }
}

// The same blocks as philox_rate_kernel through sbw::philox_block_lane.
__global__ void __launch_bounds__(kThreads)
philox_sched_kernel(uint32_t* __restrict__ out, uint64_t* __restrict__ clocks, int iters,
                    uint32_t salt) {
  uint64_t t0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    r0 = __builtin_amdgcn_s_memrealtime();
    t0 = __builtin_amdgcn_s_memtime();
  }
  const uint32_t lane = blockIdx.x * kThreads + threadIdx.x;
  uint32_t k0[kChains], k1[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) {
    k0[c] = lane ^ (static_cast<uint32_t>(c) << 24) ^ salt;
    k1[c] = lane * 0x9E3779B1u + static_cast<uint32_t>(c);
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) {
      const sbw::Block b = sbw::philox_block_lane(static_cast<uint32_t>(i), sbw::Key{k0[c], k1[c]});
      k0[c] = b.w0 ^ b.w1;
      k1[c] = b.w2 ^ b.w3;
    }
  }
  uint32_t acc = 0u;
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc ^= k0[c] ^ k1[c];
  out[lane] = acc;
  if (threadIdx.x == 0) {
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clocks[4 * blockIdx.x + 0] = t0;
    clocks[4 * blockIdx.x + 1] = t1;
    clocks[4 * blockIdx.x + 2] = r0;
    clocks[4 * blockIdx.x + 3] = r1;
  }
}

enum OpKind : int {
  kOpMad64 = 1, kOpBitop3 = 2, kOpAdd = 3, kOpPhiloxMix = 4, kOpBitop3Scalar = 5, kOpAddScalar = 6,
  kOpMulLo = 7
};

// kChains chains of `iters` x 16 links of one instruction kind per lane.  kOpPhiloxMix
// interleaves them in the block's proportions: per link one product, one xor and one
// add.  Every operand is a vector register except in the two scalar kinds, whose xor
// or add takes one wave-uniform operand.
template <int kKind>
__global__ void __launch_bounds__(kThreads)
op_rate_kernel(uint32_t* __restrict__ out, uint64_t* __restrict__ clocks, int iters,
               uint32_t salt) {
  uint64_t t0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    r0 = __builtin_amdgcn_s_memrealtime();
    t0 = __builtin_amdgcn_s_memtime();
  }
  const uint32_t lane = blockIdx.x * kThreads + threadIdx.x;
  uint32_t a[kChains], b[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) {
    a[c] = lane ^ (static_cast<uint32_t>(c) << 24) ^ salt;
    b[c] = lane * 0x9E3779B1u + static_cast<uint32_t>(c);
  }
  const uint32_t m = salt | 1u;                  // wave-uniform: a scalar register
  uint32_t mv = m ^ (lane & 1u);                 // per lane: a vector register
  asm volatile("" : "+v"(mv));
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int l = 0; l < 16; ++l) {
#pragma unroll
      for (int c = 0; c < kChains; ++c) {
        if constexpr (kKind == kOpMad64) {
          // the 64-bit chain value (b:a) <- kMulA * a + (b:a), one v_mad_u64_u32
          const uint64_t ab = (static_cast<uint64_t>(b[c]) << 32) | a[c];
          const uint64_t p = static_cast<uint64_t>(kMulA) * a[c] + ab;
          a[c] = static_cast<uint32_t>(p);
          b[c] = static_cast<uint32_t>(p >> 32);
        } else if constexpr (kKind == kOpBitop3) {
          a[c] = xor3(a[c], b[c], mv);
        } else if constexpr (kKind == kOpAdd) {
          // alternating a += b, b += a: no two links fold into one
          if (l & 1) b[c] = b[c] + a[c];
          else a[c] = a[c] + b[c];
        } else if constexpr (kKind == kOpPhiloxMix) {
          const uint64_t p = static_cast<uint64_t>(kMulA) * a[c];
          a[c] = xor3(static_cast<uint32_t>(p >> 32), b[c], mv);
          b[c] = b[c] + static_cast<uint32_t>(p);
        } else if constexpr (kKind == kOpBitop3Scalar) {
          a[c] = xor3(a[c], b[c], m);
        } else if constexpr (kKind == kOpMulLo) {
          // low half of a 32x32 product, alternating as the adds do
          if (l & 1) b[c] = b[c] * a[c];
          else a[c] = a[c] * b[c];
        } else {
          // a scalar operand (written out: the compiler would fold a chain of adds of
          // one uniform value into one product)
          asm volatile("v_add_u32 %0, %1, %0" : "+v"(a[c]) : "s"(m));
        }
      }
    }
  }
  uint32_t acc = 0u;
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc ^= a[c] ^ b[c];
  out[lane] = acc;
  if (threadIdx.x == 0) {
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clocks[4 * blockIdx.x + 0] = t0;
    clocks[4 * blockIdx.x + 1] = t1;
    clocks[4 * blockIdx.x + 2] = r0;
    clocks[4 * blockIdx.x + 3] = r1;
  }
}

}  // namespace

extern "C" {

// The same with the library's per-lane-key block (fixed round issue order).
int sbw_rate_philox_sched(uint32_t* out, uint64_t* clocks, int workgroups, int iters,
                          uint32_t salt, void* stream) {
  if (out == nullptr || clocks == nullptr || workgroups <= 0 || iters <= 0)
    return static_cast<int>(hipErrorInvalidValue);
  hipLaunchKernelGGL(philox_sched_kernel, dim3(workgroups), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), out, clocks, iters, salt);
  return static_cast<int>(hipGetLastError());
}

// Blocks drawn per lane and launch: iters * chains.
int sbw_rate_chains(void) { return kChains; }
int sbw_rate_threads(void) { return kThreads; }

// Launches the probe on `stream`: `workgroups` workgroups of sbw_rate_threads() lanes,
// each lane drawing iters * sbw_rate_chains() blocks.  out: device uint32 [workgroups *
// threads]; clocks: device uint64 [4 * workgroups] (start and end of the shader-clock
// counter, then of the real-time counter, per workgroup).  Returns a hipError_t.
int sbw_rate_philox(uint32_t* out, uint64_t* clocks, int workgroups, int iters, uint32_t salt,
                    void* stream) {
  if (out == nullptr || clocks == nullptr || workgroups <= 0 || iters <= 0)
    return static_cast<int>(hipErrorInvalidValue);
  hipLaunchKernelGGL(philox_rate_kernel, dim3(workgroups), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), out, clocks, iters, salt);
  return static_cast<int>(hipGetLastError());
}

// The single-kind chains: kind 1 products, 2 three-input xors, 3 adds, 4 the mix of
// one of each per link, 5 three-input xors and 6 adds with one scalar operand, 7 the
// low halves of 32x32 products.  Each
// lane runs iters * 16 * sbw_rate_chains() links (the mix: three instructions per
// link).  Same buffers as sbw_rate_philox.
int sbw_rate_op(int kind, uint32_t* out, uint64_t* clocks, int workgroups, int iters,
                uint32_t salt, void* stream) {
  if (out == nullptr || clocks == nullptr || workgroups <= 0 || iters <= 0)
    return static_cast<int>(hipErrorInvalidValue);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid(workgroups), block(kThreads);
  switch (kind) {
    case kOpMad64:
      hipLaunchKernelGGL(op_rate_kernel<kOpMad64>, grid, block, 0, st, out, clocks, iters, salt);
      break;
    case kOpBitop3:
      hipLaunchKernelGGL(op_rate_kernel<kOpBitop3>, grid, block, 0, st, out, clocks, iters, salt);
      break;
    case kOpAdd:
      hipLaunchKernelGGL(op_rate_kernel<kOpAdd>, grid, block, 0, st, out, clocks, iters, salt);
      break;
    case kOpPhiloxMix:
      hipLaunchKernelGGL(op_rate_kernel<kOpPhiloxMix>, grid, block, 0, st, out, clocks, iters,
                         salt);
      break;
    case kOpBitop3Scalar:
      hipLaunchKernelGGL(op_rate_kernel<kOpBitop3Scalar>, grid, block, 0, st, out, clocks, iters,
                         salt);
      break;
    case kOpAddScalar:
      hipLaunchKernelGGL(op_rate_kernel<kOpAddScalar>, grid, block, 0, st, out, clocks, iters,
                         salt);
      break;
    case kOpMulLo:
      hipLaunchKernelGGL(op_rate_kernel<kOpMulLo>, grid, block, 0, st, out, clocks, iters, salt);
      break;
    default:
      return static_cast<int>(hipErrorInvalidValue);
  }
  return static_cast<int>(hipGetLastError());
}

// Frequency of the real-time counter, in kHz (hipDeviceAttributeWallClockRate).
int sbw_rate_wall_clock_khz(void) {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
  return khz;
}

}  // extern "C"
