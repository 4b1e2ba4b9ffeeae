// Internal helpers shared by the gfx950 kernels of libsirius.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <stddef.h>
#include <stdint.h>

namespace sirius {

constexpr int kWave = 64;

// bf16 -> fp32 is exact: a bf16 is the high half of an fp32.
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// Round-to-nearest-even fp32 -> bf16 bits (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Sum over the 64 lanes of a wave; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

// Exclusive prefix sum over a 256-thread block. s_tmp holds 4 ints of LDS.
__device__ __forceinline__ int block_exclusive_scan_256(int v, int* s_tmp, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += t;
  }
  if (lane == kWave - 1) s_tmp[wave] = incl;
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wave; ++w) off += s_tmp[w];
  *total = s_tmp[0] + s_tmp[1] + s_tmp[2] + s_tmp[3];
  __syncthreads();
  return off + incl - v;
}

// Last-arrival detection without waiting: an epoch-tagged arrival counter in the caller's
// workspace. The 64-bit word holds (epoch << 16) | count. A workgroup arriving with a
// word of another epoch (stale contents from an earlier call, or never written) restarts
// the count at 1, so the workspace needs no initialisation; the epoch is unique per
// launch. Returns this workgroup's arrival index (0-based). Nobody spins: only the last
// arrival (index n-1) does extra work, after an acquire fence.
__device__ __forceinline__ int arrive_count(unsigned long long* ctr, unsigned long long tag) {
  unsigned long long old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    const bool same = (old & ~0xFFFFull) == tag;
    const unsigned long long want = same ? old + 1ull : tag + 1ull;
    if (__hip_atomic_compare_exchange_strong(ctr, &old, want, __ATOMIC_ACQ_REL, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return same ? (int)(old & 0xFFFFull) : 0;
  }
}

// Byte offsets inside a caller workspace: every region starts 256-byte aligned.
struct Carve {
  size_t off = 0;
  size_t take(size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~size_t(255);
    return o;
  }
};

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

}  // namespace sirius
