// Coarse-grained (prompt-fixed) neuron selection on gfx950 (Sec. 2.1; Appendix A.1).
//
//  griffin_z_kernel       Z[t, i] = SiLU(x_t . W_gate[i]) * (x_t . W_up[i]) for the
//                         T prompt tokens: both products in one MFMA pass
//                         (v_mfma_f32_16x16x32_bf16, exact bf16 products, fp32
//                         accumulation). Workgroup tile 128 tokens x 64 neurons,
//                         K staged through LDS in double-buffered 32-wide slices.
//  griffin_rownorm_kernel ||z_t||^2 per token (only for the normalised variant).
//  griffin_score_kernel   s_i = sqrt(sum_t z_ti^2 [/ ||z_t||^2]), fp64 sums in t order.
//  (radix select)         the k-th largest score.
//  griffin_pick_kernel    the k neurons of largest score (equal scores: lower
//                         index first), emitted in ascending index order with
//                         block scans.
//  condense_kernel        copies the selected rows of the three matrices.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

constexpr int kGT = 128;           // tokens per workgroup tile
constexpr int kGN = 64;            // neurons per workgroup tile
constexpr int kGK = 32;            // K slice per LDS stage
constexpr int kLdsRow = kGK + 8;   // padded LDS row (bf16 elements) against bank conflicts

// 16-byte chunk of row `r` (of `rows`), chunk `kc` of the K slice starting at k0; zero outside.
__device__ __forceinline__ uint4 load_chunk(const uint16_t* base, int rows, int d, int r, int k) {
  if (r < rows && k < d) return *reinterpret_cast<const uint4*>(base + (size_t)r * d + k);
  return make_uint4(0u, 0u, 0u, 0u);
}

__global__ __launch_bounds__(256) void griffin_z_kernel(const uint16_t* __restrict__ X, int T,
                                                        const uint16_t* __restrict__ Wg,
                                                        const uint16_t* __restrict__ Wu, int d,
                                                        int F, float* __restrict__ Z) {
  __shared__ __attribute__((aligned(16))) uint16_t sX[2][kGT * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sG[2][kGN * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sU[2][kGN * kLdsRow];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int t0 = blockIdx.y * kGT, n0 = blockIdx.x * kGN;
  const int wm = wave >> 1, wn = wave & 1;  // wave tile: 64 tokens x 32 neurons

  // Global -> LDS assignment: 4 chunks of 16 B per thread per stage.
  // X: 128 rows x 4 chunks = 512 chunks (2 per thread); W: 64 rows x 4 chunks x 2 mats.
  uint4 rx[2], rg, ru;
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = tid + 256 * j;
      rx[j] = load_chunk(X, T, d, t0 + (c >> 2), k0 + 8 * (c & 3));
    }
    rg = load_chunk(Wg, F, d, n0 + (tid >> 2), k0 + 8 * (tid & 3));
    ru = load_chunk(Wu, F, d, n0 + (tid >> 2), k0 + 8 * (tid & 3));
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = tid + 256 * j;
      *reinterpret_cast<uint4*>(&sX[buf][(c >> 2) * kLdsRow + 8 * (c & 3)]) = rx[j];
    }
    *reinterpret_cast<uint4*>(&sG[buf][(tid >> 2) * kLdsRow + 8 * (tid & 3)]) = rg;
    *reinterpret_cast<uint4*>(&sU[buf][(tid >> 2) * kLdsRow + 8 * (tid & 3)]) = ru;
  };

  floatx4_t accg[4][2], accu[4][2];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      accg[mt][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
      accu[mt][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    }

  const int nk = (d + kGK - 1) / kGK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int fr = lane & 15, fk = 8 * (lane >> 4);  // fragment row and k offset
  for (int ks = 0; ks < nk; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < nk) gload((ks + 1) * kGK);
    bf16x8_t a[4], bg[2], bu[2];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
      a[mt] = *reinterpret_cast<const bf16x8_t*>(&sX[buf][(wm * 64 + mt * 16 + fr) * kLdsRow + fk]);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      bg[nt] = *reinterpret_cast<const bf16x8_t*>(&sG[buf][(wn * 32 + nt * 16 + fr) * kLdsRow + fk]);
      bu[nt] = *reinterpret_cast<const bf16x8_t*>(&sU[buf][(wn * 32 + nt * 16 + fr) * kLdsRow + fk]);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        accg[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bg[nt], accg[mt][nt], 0, 0, 0);
        accu[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bu[nt], accu[mt][nt], 0, 0, 0);
      }
    if (ks + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // C layout: lane holds column (neuron) lane % 16 and rows (tokens) 4*(lane/16) + i.
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int n = n0 + wn * 32 + nt * 16 + (lane & 15);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + wm * 64 + mt * 16 + 4 * (lane >> 4) + i;
        if (t < T && n < F) Z[(size_t)t * F + n] = silu(accg[mt][nt][i]) * accu[mt][nt][i];
      }
    }
}

__global__ __launch_bounds__(256) void griffin_rownorm_kernel(const float* __restrict__ Z, int F,
                                                              float* __restrict__ rn2) {
  __shared__ double s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const float* zr = Z + (size_t)blockIdx.x * F;
  double s = 0.0;
  for (int i = tid; i < F; i += 256) s += (double)zr[i] * (double)zr[i];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, kWave);
  if (lane == 0) s_w[wave] = s;
  __syncthreads();
  if (tid == 0) rn2[blockIdx.x] = (float)(((s_w[0] + s_w[1]) + s_w[2]) + s_w[3]);
}

__global__ __launch_bounds__(256) void griffin_score_kernel(const float* __restrict__ Z, int T,
                                                            int F, const float* __restrict__ rn2,
                                                            float* __restrict__ scores) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= F) return;
  double s = 0.0;
  for (int t = 0; t < T; ++t) {
    const double z = (double)Z[(size_t)t * F + i];
    if (rn2 == nullptr) {
      s += z * z;
    } else {
      const double n2 = (double)rn2[t];
      if (n2 > 0.0) s += z * z / n2;
    }
  }
  scores[i] = (float)sqrt(s);
}

// Block-wide exclusive scan for 1024 threads (16 waves).
__device__ __forceinline__ int scan1024(int v, int* s_tmp, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += t;
  }
  if (lane == kWave - 1) s_tmp[wave] = incl;
  __syncthreads();
  int off = 0, tot = 0;
  for (int w = 0; w < 16; ++w) {
    if (w < wave) off += s_tmp[w];
    tot += s_tmp[w];
  }
  *total = tot;
  __syncthreads();
  return off + incl - v;
}

__global__ __launch_bounds__(1024) void griffin_pick_kernel(const float* __restrict__ s, int F,
                                                            int k, const float* __restrict__ kth,
                                                            int32_t* __restrict__ sel) {
  __shared__ int s_tmp[16];
  const float thr = kth[0];
  // number of scores strictly above the k-th largest
  int gt = 0;
  for (int i = threadIdx.x; i < F; i += 1024) gt += (s[i] > thr) ? 1 : 0;
  int n_gt;
  (void)scan1024(gt, s_tmp, &n_gt);
  const int need_eq = k - n_gt;  // equal scores taken, lowest index first
  int eq_run = 0, out_run = 0;
  for (int base = 0; base < F; base += 1024) {
    const int i = base + threadIdx.x;
    const float v = (i < F) ? s[i] : -1.0f;
    const int is_eq = (i < F && v == thr) ? 1 : 0;
    int eq_tot;
    const int eq_rank = eq_run + scan1024(is_eq, s_tmp, &eq_tot);
    const int take = (i < F && (v > thr || (is_eq && eq_rank < need_eq))) ? 1 : 0;
    int take_tot;
    const int pos = out_run + scan1024(take, s_tmp, &take_tot);
    if (take && pos < k) sel[pos] = i;
    eq_run += eq_tot;
    out_run += take_tot;
  }
}

__global__ __launch_bounds__(256) void condense_kernel(const uint4* __restrict__ wg,
                                                       const uint4* __restrict__ wu,
                                                       const uint4* __restrict__ wd, int nch, int F,
                                                       const int32_t* __restrict__ sel,
                                                       uint4* __restrict__ wgc, uint4* __restrict__ wuc,
                                                       uint4* __restrict__ wdc) {
  const int j = blockIdx.x;
  const uint4* src = blockIdx.y == 0 ? wg : (blockIdx.y == 1 ? wu : wd);
  uint4* dst = blockIdx.y == 0 ? wgc : (blockIdx.y == 1 ? wuc : wdc);
  const int r = sel[j];
  if (r < 0 || r >= F) return;  // sel comes from device memory; never gather outside the matrix
  const size_t row = (size_t)r;
  for (int c = threadIdx.x; c < nch; c += 256) dst[(size_t)j * nch + c] = src[row * nch + c];
}

}  // namespace

GriffinLayout griffin_layout(int T, int d, int F) {
  (void)d;
  GriffinLayout L{};
  Carve c;
  L.z = c.take((size_t)T * F * sizeof(float));
  L.rownorm = c.take((size_t)T * sizeof(float));
  L.select = c.take(select_ws_bytes());
  L.kth = c.take(sizeof(float));
  L.scores = c.take((size_t)F * sizeof(float));
  L.total = c.off;
  return L;
}

hipError_t launch_griffin(const uint16_t* xp, int T, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, int d, int F, int k, int normalize, int32_t* sel,
                          float* scores_out, uint16_t* wgc, uint16_t* wuc, uint16_t* wdc, char* ws,
                          const GriffinLayout& L, hipStream_t stream) {
  float* Z = reinterpret_cast<float*>(ws + L.z);
  float* rn2 = reinterpret_cast<float*>(ws + L.rownorm);
  char* sel_ws = ws + L.select;
  float* kth = reinterpret_cast<float*>(ws + L.kth);
  float* scores = scores_out != nullptr ? scores_out : reinterpret_cast<float*>(ws + L.scores);

  {
    ProfScope prof("griffin_z", stream);
    griffin_z_kernel<<<dim3(ceil_div(F, kGN), ceil_div(T, kGT)), 256, 0, stream>>>(xp, T, wg, wu, d,
                                                                                  F, Z);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (normalize) {
    ProfScope prof("griffin_rownorm", stream);
    griffin_rownorm_kernel<<<T, 256, 0, stream>>>(Z, F, rn2);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    ProfScope prof("griffin_score", stream);
    griffin_score_kernel<<<ceil_div(F, 256), 256, 0, stream>>>(Z, T, F, normalize ? rn2 : nullptr,
                                                               scores);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_select_kth_largest(scores, F, k, kth, sel_ws, stream)) != hipSuccess) return e;
  {
    ProfScope prof("griffin_pick", stream);
    griffin_pick_kernel<<<1, 1024, 0, stream>>>(scores, F, k, kth, sel);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  ProfScope prof("condense", stream);
  condense_kernel<<<dim3(k, 3), 256, 0, stream>>>(
      reinterpret_cast<const uint4*>(wg), reinterpret_cast<const uint4*>(wu),
      reinterpret_cast<const uint4*>(wd), d / 8, F, sel, reinterpret_cast<uint4*>(wgc),
      reinterpret_cast<uint4*>(wuc), reinterpret_cast<uint4*>(wdc));
  return hipGetLastError();
}

}  // namespace sirius
