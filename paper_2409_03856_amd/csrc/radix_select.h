// Most-significant-digit radix select over 32-bit patterns held by a 1024-thread workgroup
// (PER values per thread), shared by the per-token top-k cut and the prompt top-k of Griffin.
// The patterns are those of non-negative floats (|a|, scores), whose bit order is their value
// order. radix_common_bits settles the bits every candidate shares (a block minimum and
// maximum), so that digits of at most 11 bits can start right below them: values that crowd
// into a narrow range (prompt scores share their exponent and leading mantissa bits) then still
// spread over the first digit's bins. Values spread over many exponents (gate activations) skip
// it and start their digits at bit 30.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"

namespace sirius {

constexpr int kSelThreads1024 = 1024;
constexpr int kSelWaves = kSelThreads1024 / kWave;  // 16
constexpr int kDigitBitsMax = 11;
constexpr int kBinsMax = 1 << kDigitBitsMax;
constexpr int kHistCopies = 8;  // first-pass histogram copies: (lane / 16) + 4 (wave % 2)

// Inclusive scan of one int per thread over the 1024-thread workgroup; *total is the sum.
__device__ __forceinline__ int block_inclusive_scan_1024(int v, int* s_w, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += t;
  }
  if (lane == kWave - 1) s_w[wave] = incl;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int c = s_w[w];
    off += (w < wave) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return off + incl;
}

// The bits shared by every pattern with ok[j]: returns the highest bit in which two of them
// differ (-1 when all are equal or there are none) and sets prefix and pmask to the bits above
// it. s_w: 2 * kSelWaves words.
template <int PER>
__device__ __forceinline__ int radix_common_bits(const uint32_t (&v)[PER], const bool (&ok)[PER],
                                                 uint32_t& prefix, uint32_t& pmask, int* s_w) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (ok[j]) {
      lo = min(lo, v[j]);
      hi = max(hi, v[j]);
    }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, m, kWave));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, m, kWave));
  }
  if (lane == 0) {
    s_w[wave] = (int)lo;
    s_w[kSelWaves + wave] = (int)hi;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    lo = min(lo, (uint32_t)s_w[w]);
    hi = max(hi, (uint32_t)s_w[kSelWaves + w]);
  }
  __syncthreads();
  if (lo >= hi) {  // one value (or none): every bit settled
    prefix = lo;
    pmask = 0xffffffffu;
    return -1;
  }
  const int top = 31 - __clz(lo ^ hi);
  pmask = top == 31 ? 0u : ~((2u << top) - 1u);
  prefix = lo & pmask;
  return top;
}

// One digit pass: among the thread's patterns v[j] with ok[j] whose bits under pmask equal
// prefix, histogram the digit (v >> shift) & (2^bits - 1) (LDS atomics in ncopy copies, so that
// equal digits of one wave instruction collide less), then a block scan over the bins (thread t
// holds the two digits 2^bits - 1 - 2t and the next one down, so the scan counts the values at or
// above them) finds the digit holding the kr-th largest. On return (every thread): prefix and
// pmask include that digit, kr is the rank inside it and *count its number of members.
// s_hist: kHistCopies * kBinsMax words; s_w: kSelWaves; s_sel: 3.
template <int PER>
__device__ __forceinline__ void radix_digit_pass(const uint32_t (&v)[PER], const bool (&ok)[PER],
                                                 int shift, int bits, int ncopy, uint32_t& prefix,
                                                 uint32_t& pmask, int& kr, int* count,
                                                 uint32_t* s_hist, int* s_w, int* s_sel) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int nb = 1 << bits;
  const uint32_t dmask = (uint32_t)nb - 1u;
  const int copy = ((lane >> 4) + 4 * (wave & 1)) % ncopy;
  for (int i = tid; i < ncopy * nb; i += kSelThreads1024) s_hist[i] = 0u;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (ok[j] && (v[j] & pmask) == prefix) atomicAdd(&s_hist[copy * nb + ((v[j] >> shift) & dmask)], 1u);
  __syncthreads();
  const int d1 = nb - 1 - 2 * tid, d2 = d1 - 1;
  int c1 = 0, c2 = 0;
  if (d2 >= 0) {
    for (int q = 0; q < ncopy; ++q) {
      c1 += (int)s_hist[q * nb + d1];
      c2 += (int)s_hist[q * nb + d2];
    }
  }
  int tot;
  const int incl = block_inclusive_scan_1024(c1 + c2, s_w, &tot);
  const int before = incl - c1 - c2;
  if (before < kr && kr <= before + c1) {
    s_sel[0] = d1;
    s_sel[1] = kr - before;
    s_sel[2] = c1;
  } else if (before + c1 < kr && kr <= incl) {
    s_sel[0] = d2;
    s_sel[1] = kr - before - c1;
    s_sel[2] = c2;
  }
  __syncthreads();
  prefix |= (uint32_t)s_sel[0] << shift;
  pmask |= dmask << shift;
  kr = s_sel[1];
  *count = s_sel[2];
  __syncthreads();  // s_sel and s_hist are rewritten by the caller's next step
}

}  // namespace sirius
