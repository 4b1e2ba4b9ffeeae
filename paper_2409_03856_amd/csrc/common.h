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

// 16-byte loads for data that is read exactly once (weight rows, logits): non-temporal, so
// the stream does not displace reused lines in the caches. Measured on MI355X: the batch-1
// decode pass over a Llama-3-8B FFN layer goes from 5.0 to 5.4 TB/s.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld_stream(const float4* p) {
  const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

// Dot product of 8 bf16 weights (one 16-byte load) with 8 fp32 activations (16-byte aligned).
__device__ __forceinline__ float dot8(uint4 w, const float* xp, float acc) {
  const float4 a = *reinterpret_cast<const float4*>(xp);
  const float4 b = *reinterpret_cast<const float4*>(xp + 4);
  acc = fmaf(bf16_lo(w.x), a.x, acc);
  acc = fmaf(bf16_hi(w.x), a.y, acc);
  acc = fmaf(bf16_lo(w.y), a.z, acc);
  acc = fmaf(bf16_hi(w.y), a.w, acc);
  acc = fmaf(bf16_lo(w.z), b.x, acc);
  acc = fmaf(bf16_hi(w.z), b.y, acc);
  acc = fmaf(bf16_lo(w.w), b.z, acc);
  acc = fmaf(bf16_hi(w.w), b.w, acc);
  return acc;
}

// acc[0..7] += h * (8 bf16 weights of one 16-byte load)
__device__ __forceinline__ void axpy8(float h, uint4 w, float* acc) {
  acc[0] = fmaf(h, bf16_lo(w.x), acc[0]);
  acc[1] = fmaf(h, bf16_hi(w.x), acc[1]);
  acc[2] = fmaf(h, bf16_lo(w.y), acc[2]);
  acc[3] = fmaf(h, bf16_hi(w.y), acc[3]);
  acc[4] = fmaf(h, bf16_lo(w.z), acc[4]);
  acc[5] = fmaf(h, bf16_hi(w.z), acc[5]);
  acc[6] = fmaf(h, bf16_lo(w.w), acc[6]);
  acc[7] = fmaf(h, bf16_hi(w.w), acc[7]);
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
