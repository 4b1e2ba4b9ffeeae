// A small Llama-style decoder built from the library's kernels, and the Sirius generation
// loop (Algorithm 1) over it with every decision kept on the device.
//
//  embed_kernel        h[i] = E[token_i] (bf16 rows widened; an id outside [0, V) gives 0)
//  linear_kernel<NB>   y[i][j] = x[i] . W[j] (+ resid[i][j]) for up to NB rows of x staged in
//                      LDS; one wave per output row (W row-major [N][K] bf16), fp32 or bf16
//                      output (round to nearest even)
//  norm_qkv_kernel<NB> RMSNorm of the rows as they are staged (the same sums, in the same order,
//                      as rmsnorm_vec_kernel, so bit for bit its result), then the products of
//                      up to three matrices in one launch: q = xn Wq^T (fp32), k = xn Wk^T and
//                      v = xn Wv^T (bf16) -- a layer's attention inputs, or the final norm and
//                      the LM head (q only)
//  draft_tail_kernel   the sparse model's greedy draft: argmax of one logit row (lowest index
//                      on ties) into the chunk buffer, and the cache position advanced by one
//                      (wound back by n - 1 after the last draft, so the full model's pass
//                      starts at the period's first position)
//  period_tail_kernel  after the check: the rollback to P + min(j + 1, n), the accepted
//                      drafts and the corrected token appended to the output, and the next
//                      period's first input (the corrected token, or the last draft)
//
// One period is a fixed sequence of launches on one stream -- n sparse passes, one full pass
// over the n-token chunk, the check, the tail -- with the positions, drafts, acceptance and
// output count living in device memory, so periods run back to back without a host round
// trip.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

constexpr int kLinThreads = 256;
constexpr int kLinWaves = kLinThreads / kWave;
constexpr int kLinLds = 16384;  // floats of x staged per launch (64 KiB)
constexpr int kTailThreads = 1024;

__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ tokens, int n,
                                                    const uint4* __restrict__ E, int d8, int V,
                                                    float* __restrict__ out) {
  const int i = blockIdx.x;
  if (i >= n) return;
  const int tok = tokens[i];
  const bool ok = tok >= 0 && tok < V;
  float4* o = reinterpret_cast<float4*>(out + (size_t)i * d8 * 8);
  for (int c = threadIdx.x; c < d8; c += blockDim.x) {
    const uint4 w = ok ? E[(size_t)tok * d8 + c] : make_uint4(0u, 0u, 0u, 0u);
    o[2 * c] = make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
    o[2 * c + 1] = make_float4(bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w));
  }
}

// Rows j = blockIdx.x * 4 + wave, + gridDim.x * 4, ...; x rows 0 .. n - 1 (n <= NB) in LDS.
template <int NB, bool OUT_BF16>
__global__ __launch_bounds__(kLinThreads) void linear_kernel(const float* __restrict__ x, int n,
                                                             const uint4* __restrict__ W, int K,
                                                             int N, const float* resid, float* y,
                                                             uint16_t* __restrict__ yb) {
  __shared__ float4 s_x4[kLinLds / 4];
  const float* xs = reinterpret_cast<const float*>(s_x4);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int k4 = K >> 2, k8 = K >> 3;
  const float4* x4 = reinterpret_cast<const float4*>(x);
  for (int e = tid; e < n * k4; e += kLinThreads) s_x4[e] = x4[e];
  __syncthreads();
  for (int j = blockIdx.x * kLinWaves + wave; j < N; j += gridDim.x * kLinWaves) {
    float acc[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[i] = 0.f;
    const uint4* wr = W + (size_t)j * k8;
    for (int c = lane; c < k8; c += kWave) {
      const uint4 w = wr[c];
#pragma unroll
      for (int i = 0; i < NB; ++i)
        if (i < n) acc[i] = dot8(w, xs + (size_t)i * K + 8 * c, acc[i]);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i < n) {  // n is uniform over the wave
        const float s = wave_sum(acc[i]);
        if (lane == i) {
          const size_t o = (size_t)i * N + j;
          if (OUT_BF16) {
            yb[o] = (uint16_t)f32_to_bf16(s);
          } else {
            y[o] = (resid != nullptr) ? resid[o] + s : s;
          }
        }
      }
    }
  }
}

// Output rows j of the three products in one range: [0, Nq) of Wq into yq (fp32), then
// [Nq, Nq + Nkv) of Wk and [Nq + Nkv, Nq + 2 Nkv) of Wv into yk, yv (bf16). The rows of x are
// staged in LDS (every load in flight at once), then normalised there: each thread sums the
// squares of its float4s tid + 256 u of a row as rmsnorm_vec_kernel does, the wave sums go through
// LDS, and after one barrier each thread scales its float4s.
template <int NB>
__global__ __launch_bounds__(kLinThreads) void norm_qkv_kernel(
    const float* __restrict__ x, int n, int K, float eps, const uint4* __restrict__ Wq, int Nq,
    const uint4* __restrict__ Wk, const uint4* __restrict__ Wv, int Nkv, float* __restrict__ yq,
    uint16_t* __restrict__ yk, uint16_t* __restrict__ yv) {
  static_assert(kLinThreads == 256, "the norm's sums follow rmsnorm_vec_kernel's 256-thread layout");
  constexpr int kPer = 8;  // K <= 8192
  __shared__ float4 s_x4[kLinLds / 4];
  __shared__ float s_w[NB][kLinWaves];
  const float* xs = reinterpret_cast<const float*>(s_x4);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int k4 = K >> 2, k8 = K >> 3;
  const float4* x4 = reinterpret_cast<const float4*>(x);
  for (int e = tid; e < n * k4; e += kLinThreads) s_x4[e] = x4[e];  // every row's loads in flight
  __syncthreads();
  for (int i = 0; i < n; ++i) {
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + kLinThreads * u;
      const float4 v = (e < k4) ? s_x4[i * k4 + e] : make_float4(0.f, 0.f, 0.f, 0.f);
      ss = fmaf(v.x, v.x, ss);
      ss = fmaf(v.y, v.y, ss);
      ss = fmaf(v.z, v.z, ss);
      ss = fmaf(v.w, v.w, ss);
    }
    ss = wave_sum(ss);
    if (lane == 0) s_w[i][wave] = ss;
  }
  __syncthreads();
  for (int i = 0; i < n; ++i) {
    const float tot = ((s_w[i][0] + s_w[i][1]) + s_w[i][2]) + s_w[i][3];
    const float inv = 1.0f / sqrtf(tot / (float)K + eps);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + kLinThreads * u;
      if (e < k4) {
        const float4 t = s_x4[i * k4 + e];
        s_x4[i * k4 + e] = make_float4(t.x * inv, t.y * inv, t.z * inv, t.w * inv);
      }
    }
  }
  __syncthreads();
  const int N = Nq + 2 * Nkv;
  for (int j = blockIdx.x * kLinWaves + wave; j < N; j += gridDim.x * kLinWaves) {
    const int part = j < Nq ? 0 : (j < Nq + Nkv ? 1 : 2);  // uniform over the wave
    const int jr = part == 0 ? j : (part == 1 ? j - Nq : j - Nq - Nkv);
    const uint4* wr = (part == 0 ? Wq : (part == 1 ? Wk : Wv)) + (size_t)jr * k8;
    float acc[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[i] = 0.f;
    for (int c = lane; c < k8; c += kWave) {
      const uint4 w = wr[c];
#pragma unroll
      for (int i = 0; i < NB; ++i)
        if (i < n) acc[i] = dot8(w, xs + (size_t)i * K + 8 * c, acc[i]);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i < n) {  // n is uniform over the wave
        const float s = wave_sum(acc[i]);
        if (lane == i) {
          if (part == 0) yq[(size_t)i * Nq + jr] = s;
          else (part == 1 ? yk : yv)[(size_t)i * Nkv + jr] = (uint16_t)f32_to_bf16(s);
        }
      }
    }
  }
}

// Argmax over one row of V logits, lowest index on ties: (value, index) pairs reduced so
// that the larger value wins and, on equal values, the smaller index.
__device__ __forceinline__ void better(float& v, int& i, float ov, int oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

__device__ int block_argmax(const float* __restrict__ row, int V) {
  __shared__ float s_v[kTailThreads / kWave];
  __shared__ int s_i[kTailThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  float bv = -INFINITY;
  int bi = INT32_MAX;
  for (int v = tid; v < V; v += kTailThreads) better(bv, bi, row[v], v);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(bv, m, kWave);
    const int oi = __shfl_xor(bi, m, kWave);
    better(bv, bi, ov, oi);
  }
  if (lane == 0) {
    s_v[wave] = bv;
    s_i[wave] = bi;
  }
  __syncthreads();
  bv = s_v[0];
  bi = s_i[0];
  for (int w = 1; w < kTailThreads / kWave; ++w) better(bv, bi, s_v[w], s_i[w]);
  return bi == INT32_MAX ? 0 : bi;  // a row of NaNs only
}

__global__ __launch_bounds__(kTailThreads) void draft_tail_kernel(
    const float* __restrict__ logits, int V, int32_t* __restrict__ seq, int slot,
    int32_t* __restrict__ cache_pos, int pos_delta, int32_t* __restrict__ trace_drafted) {
  const int tok = block_argmax(logits, V);
  if (threadIdx.x == 0) {
    seq[slot] = tok;
    cache_pos[0] += pos_delta;
    if (trace_drafted != nullptr) trace_drafted[slot - 1] = tok;
  }
}

__global__ void period_tail_kernel(int32_t* __restrict__ seq, int n,
                                   const int32_t* __restrict__ accept_len,
                                   const int32_t* __restrict__ next_token,
                                   int32_t* __restrict__ cache_pos, int32_t* __restrict__ out,
                                   int32_t* __restrict__ out_count, int out_cap,
                                   int32_t* __restrict__ tr_accept, int32_t* __restrict__ tr_next) {
  if (threadIdx.x != 0) return;
  int j = accept_len[0];
  j = j < 0 ? 0 : (j > n ? n : j);
  const int nxt = next_token[0];
  cache_pos[0] += (j + 1 < n) ? j + 1 : n;
  int c = out_count[0];
  for (int i = 1; i <= j; ++i)
    if (c >= 0 && c < out_cap) out[c++] = seq[i];
  if (j < n) {
    if (c >= 0 && c < out_cap) out[c++] = nxt;
    seq[0] = nxt;
  } else {
    seq[0] = seq[n];
  }
  out_count[0] = c;
  if (tr_accept != nullptr) tr_accept[0] = j;
  if (tr_next != nullptr) tr_next[0] = (j < n) ? nxt : -1;
}

template <bool OUT_BF16>
hipError_t launch_linear_t(const float* x, int n, const uint16_t* W, int K, int N,
                           const float* resid, float* y, uint16_t* yb, hipStream_t s) {
  const int nb = std::min(16, kLinLds / K);
  for (int i0 = 0; i0 < n; i0 += nb) {
    const int m = std::min(nb, n - i0);
    const int grid = std::min(ceil_div(N, kLinWaves), 2048);
    const float* xi = x + (size_t)i0 * K;
    const float* ri = resid ? resid + (size_t)i0 * N : nullptr;
    float* yi = y ? y + (size_t)i0 * N : nullptr;
    uint16_t* ybi = yb ? yb + (size_t)i0 * N : nullptr;
    const uint4* w4 = reinterpret_cast<const uint4*>(W);
#define SIRIUS_LIN(NBV)                                                                       \
  if (m <= NBV) {                                                                             \
    klaunch(linear_kernel<NBV, OUT_BF16>, grid, kLinThreads, 0, s, xi, m, w4, K, N, ri, yi, ybi); \
    hipError_t e = hipGetLastError();                                                         \
    if (e != hipSuccess) return e;                                                            \
    continue;                                                                                 \
  }
    SIRIUS_LIN(1)
    SIRIUS_LIN(4)
    SIRIUS_LIN(16)
#undef SIRIUS_LIN
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_embed(const int32_t* tokens, int n, const uint16_t* E, int d, int V, float* out,
                        hipStream_t s) {
  ProfScope prof("embed", s);
  klaunch(embed_kernel, n, 256, 0, s, tokens, n, reinterpret_cast<const uint4*>(E), d / 8, V, out);
  return hipGetLastError();
}

hipError_t launch_norm_qkv(const float* x, int n, int K, float eps, const uint16_t* Wq, int Nq,
                           const uint16_t* Wk, const uint16_t* Wv, int Nkv, float* yq,
                           uint16_t* yk, uint16_t* yv, hipStream_t s) {
  if ((K & 7) != 0 || K > 8192 || n < 1 || Nq < 1 || Nkv < 0 ||
      (Nkv > 0 && (Wk == nullptr || Wv == nullptr || yk == nullptr || yv == nullptr)))
    return hipErrorInvalidValue;
  ProfScope prof("norm_qkv", s);
  const int nb = std::min(16, kLinLds / K);
  for (int i0 = 0; i0 < n; i0 += nb) {
    const int m = std::min(nb, n - i0);
    const int grid = std::min(ceil_div(Nq + 2 * Nkv, kLinWaves), 2048);
    const float* xi = x + (size_t)i0 * K;
    float* qi = yq + (size_t)i0 * Nq;
    uint16_t* ki = Nkv > 0 ? yk + (size_t)i0 * Nkv : nullptr;
    uint16_t* vi = Nkv > 0 ? yv + (size_t)i0 * Nkv : nullptr;
    const uint4* q4 = reinterpret_cast<const uint4*>(Wq);
    const uint4* k4 = reinterpret_cast<const uint4*>(Wk);
    const uint4* v4 = reinterpret_cast<const uint4*>(Wv);
#define SIRIUS_NQKV(NBV)                                                                          \
  if (m <= NBV) {                                                                                 \
    klaunch(norm_qkv_kernel<NBV>, grid, kLinThreads, 0, s, xi, m, K, eps, q4, Nq, k4, v4, Nkv, qi, ki, vi); \
    hipError_t e = hipGetLastError();                                                             \
    if (e != hipSuccess) return e;                                                                \
    continue;                                                                                     \
  }
    SIRIUS_NQKV(1)
    SIRIUS_NQKV(4)
    SIRIUS_NQKV(16)
#undef SIRIUS_NQKV
  }
  return hipSuccess;
}

hipError_t launch_linear(const float* x, int n, const uint16_t* W, int K, int N,
                         const float* resid, float* y, uint16_t* y_bf16, hipStream_t s) {
  if ((K & 7) != 0 || K > kLinLds || n < 1) return hipErrorInvalidValue;
  ProfScope prof("linear", s);
  if (y_bf16 != nullptr) return launch_linear_t<true>(x, n, W, K, N, nullptr, nullptr, y_bf16, s);
  return launch_linear_t<false>(x, n, W, K, N, resid, y, nullptr, s);
}

hipError_t launch_draft_tail(const float* logits, int V, int32_t* seq, int slot,
                             int32_t* cache_pos, int pos_delta, int32_t* trace_drafted,
                             hipStream_t s) {
  ProfScope prof("draft_tail", s);
  klaunch(draft_tail_kernel, 1, kTailThreads, 0, s, logits, V, seq, slot, cache_pos, pos_delta,
          trace_drafted);
  return hipGetLastError();
}

hipError_t launch_period_tail(int32_t* seq, int n, const int32_t* accept_len,
                              const int32_t* next_token, int32_t* cache_pos, int32_t* out,
                              int32_t* out_count, int out_cap, int32_t* tr_accept,
                              int32_t* tr_next, hipStream_t s) {
  ProfScope prof("period_tail", s);
  klaunch(period_tail_kernel, 1, 64, 0, s, seq, n, accept_len, next_token, cache_pos, out,
          out_count, out_cap, tr_accept, tr_next);
  return hipGetLastError();
}

}  // namespace sirius
