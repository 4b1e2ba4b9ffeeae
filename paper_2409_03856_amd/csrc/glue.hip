// Layer-stack glue on gfx950: unit-weight RMSNorm and a seeded bf16 normal fill.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

// out[b] = h[b] / sqrt(mean(h[b]^2) + eps); one workgroup per row, fixed-order sums.
// One workgroup per row; every thread requests all of its (at most eight) 16-byte pieces of
// the row before using any of them, and writes the result from registers. d % 4 == 0,
// d <= 8192, 16-byte aligned rows.
__global__ __launch_bounds__(256) void rmsnorm_vec_kernel(const float* h, int d, float eps, float* out) {
  constexpr int kPer = 8;  // d_model <= 8192
  __shared__ float s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int nv4 = d >> 2;
  const float4* hr = reinterpret_cast<const float4*>(h + (size_t)blockIdx.x * d);
  float4* orow = reinterpret_cast<float4*>(out + (size_t)blockIdx.x * d);
  float4 v[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    v[u] = (i < nv4) ? hr[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    ss = fmaf(v[u].x, v[u].x, ss);
    ss = fmaf(v[u].y, v[u].y, ss);
    ss = fmaf(v[u].z, v[u].z, ss);
    ss = fmaf(v[u].w, v[u].w, ss);
  }
  ss = wave_sum(ss);
  if (lane == 0) s_w[wave] = ss;
  __syncthreads();
  const float tot = ((s_w[0] + s_w[1]) + s_w[2]) + s_w[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    if (i < nv4) orow[i] = make_float4(v[u].x * inv, v[u].y * inv, v[u].z * inv, v[u].w * inv);
  }
}

// Any d_model and alignment: the same per-row reduction with scalar accesses, eight loads in
// flight per thread.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* h, int d, float eps, float* out) {
  __shared__ float s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const float* hr = h + (size_t)blockIdx.x * d;
  float* orow = out + (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int i0 = tid; i0 < d; i0 += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (i0 + 256 * u < d) ? hr[i0 + 256 * u] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) ss = fmaf(v[u], v[u], ss);
  }
  ss = wave_sum(ss);
  if (lane == 0) s_w[wave] = ss;
  __syncthreads();
  const float tot = ((s_w[0] + s_w[1]) + s_w[2]) + s_w[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int i = tid; i < d; i += 256) orow[i] = hr[i] * inv;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as easy
// as 1, 2, 3", SC 2011): ten rounds of two 32x32->64 multiplies on a 4-word
// counter, the 2-word key bumped by the Weyl constants between rounds.
struct U4 {
  uint32_t v[4];
};
__device__ __forceinline__ U4 philox4x32_10(U4 ctr, uint32_t k0, uint32_t k1) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = (uint64_t)kM0 * ctr.v[0];
    const uint64_t p1 = (uint64_t)kM1 * ctr.v[2];
    U4 n;
    n.v[0] = (uint32_t)(p1 >> 32) ^ ctr.v[1] ^ k0;
    n.v[1] = (uint32_t)p1;
    n.v[2] = (uint32_t)(p0 >> 32) ^ ctr.v[3] ^ k1;
    n.v[3] = (uint32_t)p0;
    ctr = n;
    k0 += kW0;
    k1 += kW1;
  }
  return ctr;
}

// Element e gets the (e % 4)-th normal of counter block e / 4 (Box-Muller on word pairs).
__global__ __launch_bounds__(256) void fill_normal_bf16_kernel(uint16_t* out, size_t n,
                                                               uint32_t k0, uint32_t k1,
                                                               float mean, float std) {
  const size_t nblk = (n + 3) / 4;
  for (size_t blk = (size_t)blockIdx.x * blockDim.x + threadIdx.x; blk < nblk;
       blk += (size_t)gridDim.x * blockDim.x) {
    U4 ctr;
    ctr.v[0] = (uint32_t)blk;
    ctr.v[1] = (uint32_t)(blk >> 32);
    ctr.v[2] = 0u;
    ctr.v[3] = 0u;
    const U4 r = philox4x32_10(ctr, k0, k1);
    float z[4];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      // u1 in (0, 1], u2 in [0, 1)
      const float u1 = ((float)r.v[2 * p] + 1.0f) * 2.3283064365386963e-10f;
      const float u2 = (float)r.v[2 * p + 1] * 2.3283064365386963e-10f;
      const float rad = sqrtf(-2.0f * logf(fminf(u1, 1.0f)));
      const float ang = 6.283185307179586f * u2;
      z[2 * p] = rad * cosf(ang);
      z[2 * p + 1] = rad * sinf(ang);
    }
    const size_t e0 = blk * 4;
    if (e0 + 4 <= n && ((reinterpret_cast<uintptr_t>(out + e0) & 7u) == 0)) {
      uint2 pk;
      pk.x = f32_to_bf16(fmaf(std, z[0], mean)) | (f32_to_bf16(fmaf(std, z[1], mean)) << 16);
      pk.y = f32_to_bf16(fmaf(std, z[2], mean)) | (f32_to_bf16(fmaf(std, z[3], mean)) << 16);
      *reinterpret_cast<uint2*>(out + e0) = pk;
    } else {
      for (int q = 0; q < 4 && e0 + q < n; ++q) out[e0 + q] = (uint16_t)f32_to_bf16(fmaf(std, z[q], mean));
    }
  }
}

}  // namespace

hipError_t launch_rmsnorm(const float* h, int B, int d, float eps, float* out, hipStream_t stream) {
  ProfScope prof("rmsnorm", stream);
  const bool vec = (d & 3) == 0 && d <= 8192 && (reinterpret_cast<uintptr_t>(h) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  if (vec) klaunch(rmsnorm_vec_kernel, B, 256, 0, stream, h, d, eps, out);
  else klaunch(rmsnorm_kernel, B, 256, 0, stream, h, d, eps, out);
  return hipGetLastError();
}

hipError_t launch_fill_normal_bf16(uint16_t* out, size_t n, uint64_t seed, float mean, float std,
                                   hipStream_t stream) {
  const size_t nblk = (n + 3) / 4;
  const size_t want = (nblk + 255) / 256;
  const int grid = (int)std::min<size_t>(want, 65536);
  ProfScope prof("fill_normal", stream);
  klaunch(fill_normal_bf16_kernel, grid, 256, 0, stream, out, n, (uint32_t)seed, (uint32_t)(seed >> 32),
                                                    mean, std);
  return hipGetLastError();
}

}  // namespace sirius
