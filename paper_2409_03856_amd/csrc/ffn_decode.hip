// Batch-1 SwiGLU FFN decode on gfx950 in one pass per row segment: dense, condensed,
// per-token threshold sparsity (FSparse after CATS: the gate is read whole, W_up and W_down
// only for the kept neurons) and both passes of per-token top-k sparsity (the gate phase
// alone writing the activations, then the kept up and down rows under the token's cut).
//
//  decode1_kernel  one 1024-thread workgroup (16 waves) per segment of contiguous neuron
//                  rows, one workgroup per CU. In order:
//                  * the first gate row of every wave is requested before x is staged in
//                    LDS (fp32, optionally RMS-normalised with unit weight);
//                  * gate rows: wave w takes rows w, w + 16, ...; with d_model <= 4096 two
//                    rows are in flight per wave (the next one is requested before the
//                    current one is reduced); a = SiLU(W_gate[i].x), kept iff |a| > t;
//                  * a wave ballot + popcount compacts the kept rows in ascending order;
//                  * W_up rows of the kept neurons, h_i = a_i * (W_up[i].x), into LDS
//                    (dense with d_model <= 4096: every row is kept, so each wave takes the
//                    gate and up rows of its neurons together, one pair in flight, and the
//                    compaction and the separate up phase drop out);
//                  * W_down rows of the kept neurons: thread (p, c) owns the eight output
//                    columns of 16-byte chunk c and the kept rows p, p + P, ... with eight
//                    row chunks in flight (dense: the first eight requested before the
//                    barrier that completes h); the P row groups are summed in a fixed
//                    order into the segment's partial y.
//  reduce_kernel   (ffn_gemv.hip) y = resid + the segment partials in order, and the
//                  ascending active list from the per-segment lists.
//
// Two launches per call and no cross-workgroup synchronisation: no atomics, no fences. The
// kept indices, a and h never leave the workgroup, and every weight byte is read once, with
// non-temporal loads.
#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "topk.h"

namespace sirius {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;  // 16
constexpr int kSegs = 256;                // one workgroup per CU
constexpr int kMinRows = 8;               // rows per segment at least (small d_ff)
constexpr int kMaxRows = 256;             // rows per segment at most: d_ff <= 65536
constexpr int kMaxD = 8192;               // x staged in LDS: 32 KiB
constexpr int kDownUnroll = 8;            // W_down row chunks in flight per thread

// kModeKeyed: per-token top-k; the gate activations come from a separate gate pass, and a
// neuron is kept iff its top-k key reaches the token's cut (no W_gate read here).
// kModeAct: that gate pass: the gate phase alone, writing the signed activations.
constexpr int kModeDense = 0, kModeSparse = 1, kModeKeyed = 2, kModeAct = 3;

template <int CPL>
__device__ __forceinline__ void load_row(uint4 (&w)[CPL], const uint4* row, int lane, int nch,
                                         bool ok) {
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int c = lane + kWave * q;
    w[q] = (ok && c < nch) ? ld_stream(row + c) : make_uint4(0u, 0u, 0u, 0u);
  }
}

// The same with every lane issuing all CPL loads: a lane past the row's end re-reads its last
// chunk, and a row that is not wanted (ok false) is read from `spare` (x: read by every
// workgroup, resident in L2). The number of loads in flight is then fixed where each buffer is
// used, so the wait for one row leaves the next one in flight (the predicated form above makes
// the compiler wait for all of them).
template <int CPL>
__device__ __forceinline__ void load_row_all(uint4 (&w)[CPL], const uint4* row,
                                             const uint4* spare, int lane, int nch, bool ok) {
  const uint4* p = ok ? row : spare;
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int c = lane + kWave * q;
    w[q] = ld_stream(p + (c < nch ? c : nch - 1));
  }
}

// W[i].x over the wave (every lane receives the sum); lane owns chunks lane + 64 q.
template <int CPL>
__device__ __forceinline__ float row_dot(const uint4 (&w)[CPL], const float* xs, int lane,
                                         int nch) {
  float acc = 0.f;
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int c = lane + kWave * q;
    if (c < nch) acc = dot8(w[q], xs + 8 * c, acc);
  }
  return wave_sum(acc);
}

template <int CPL, int MODE>
__global__ __launch_bounds__(kThreads) void decode1_kernel(
    const float* __restrict__ x, const uint4* __restrict__ wg, const uint4* __restrict__ wu,
    const uint4* __restrict__ wd, int d, int F, float t, float norm_eps, int rmax,
    int32_t* __restrict__ uidx, int32_t* __restrict__ ucnt, float* __restrict__ part,
    const float* __restrict__ act, const unsigned long long* __restrict__ cut,
    float* __restrict__ act_out) {
  // x (normalised) during gate and up; the down phase's row-group partials afterwards
  __shared__ float4 s_x4[kMaxD / 4];
  __shared__ float s_a[kMaxRows];
  __shared__ float s_h[kMaxRows];
  __shared__ int s_keep[kMaxRows];
  __shared__ int s_list[kMaxRows];
  __shared__ int s_wc[kWaves];
  __shared__ float s_ss[kWaves];
  float* xs = reinterpret_cast<float*>(s_x4);

  constexpr int NB = CPL <= 8 ? 2 : 1;  // rows in flight per wave in the gate and up phases
  // dense with d_model <= 4096: every row is kept, so a wave takes the gate and up rows of one
  // neuron together (two rows in flight) and the separate up phase and the compaction go away
  constexpr bool kFused = MODE == kModeDense && NB == 2;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int seg = blockIdx.x, G = gridDim.x;
  const int nch = d >> 3, nv4 = d >> 2;
  const int r0 = (int)(((long long)F * seg) / G);
  const int nr = (int)(((long long)F * (seg + 1)) / G) - r0;  // 1 <= nr <= rmax <= kMaxRows

  const uint4* spare = reinterpret_cast<const uint4*>(x);
  uint4 wa[CPL], wb[CPL];
  if (kFused) {
    load_row_all(wa, wg + (size_t)(r0 + wave) * nch, spare, lane, nch, wave < nr);
    load_row_all(wb, wu + (size_t)(r0 + wave) * nch, spare, lane, nch, wave < nr);
  } else {
    load_row(wa, wg + (size_t)(r0 + wave) * nch, lane, nch, MODE != kModeKeyed && wave < nr);
  }

  // ---- x into LDS, RMS-normalised when norm_eps >= 0
  float ss = 0.f;
  const float4* x4 = reinterpret_cast<const float4*>(x);
  for (int i = tid; i < nv4; i += kThreads) {
    const float4 v = x4[i];
    s_x4[i] = v;
    ss = fmaf(v.x, v.x, ss);
    ss = fmaf(v.y, v.y, ss);
    ss = fmaf(v.z, v.z, ss);
    ss = fmaf(v.w, v.w, ss);
  }
  if (norm_eps >= 0.f) {
    ss = wave_sum(ss);
    if (lane == 0) s_ss[wave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += s_ss[w];
    const float inv = 1.0f / sqrtf(tot / (float)d + norm_eps);
    for (int i = tid; i < nv4; i += kThreads) {
      float4 v = s_x4[i];
      v.x *= inv;
      v.y *= inv;
      v.z *= inv;
      v.w *= inv;
      s_x4[i] = v;
    }
  }
  __syncthreads();

  // ---- gate rows j = wave, wave + 16, ...; the next row is requested before this one is used
  auto gate_row = [&](const uint4(&w)[CPL], int j) {
    const float a = silu(row_dot(w, xs, lane, nch));
    if (lane == 0) {
      if (MODE == kModeAct) act_out[r0 + j] = a;
      s_a[j] = a;
      s_keep[j] = (MODE == kModeDense || fabsf(a) > t) ? 1 : 0;
    }
  };
  if (MODE == kModeKeyed) {
    const unsigned long long c0 = cut[0];
    for (int j = tid; j < nr; j += kThreads) {
      const float a = act[r0 + j];
      s_a[j] = a;
      s_keep[j] = topk_key(a, r0 + j) >= c0 ? 1 : 0;
    }
  }
  if (kFused) {
    for (int j = wave; j < nr; j += kWaves) {
      const int jn = j + kWaves;
      const float a = silu(row_dot(wa, xs, lane, nch));
      load_row_all(wa, wg + (size_t)(r0 + jn) * nch, spare, lane, nch, jn < nr);
      const float u = row_dot(wb, xs, lane, nch);
      load_row_all(wb, wu + (size_t)(r0 + jn) * nch, spare, lane, nch, jn < nr);
      if (lane == 0) s_h[j] = a * u;  // kept list = the segment's rows in order
    }
    for (int j = tid; j < nr; j += kThreads) s_list[j] = j;
  }
  for (int j = wave; MODE != kModeKeyed && !kFused && j < nr; j += NB * kWaves) {
    if (NB == 2) {
      const int j1 = j + kWaves, j2 = j + 2 * kWaves;
      load_row(wb, wg + (size_t)(r0 + j1) * nch, lane, nch, j1 < nr);
      gate_row(wa, j);
      load_row(wa, wg + (size_t)(r0 + j2) * nch, lane, nch, j2 < nr);
      if (j1 < nr) gate_row(wb, j1);
    } else {
      gate_row(wa, j);
      const int j1 = j + kWaves;
      load_row(wa, wg + (size_t)(r0 + j1) * nch, lane, nch, j1 < nr);
    }
  }
  if (MODE == kModeAct) return;  // the activations are all this mode writes
  if (!kFused) __syncthreads();

  // ---- ascending compaction of the kept rows: wave ballot + popcount, wave offsets in LDS
  int nk = nr;
  if (!kFused) {
    const int keep = (tid < nr) ? s_keep[tid] : 0;
    const unsigned long long m = __ballot(keep);
    if (lane == 0) s_wc[wave] = __popcll(m);
    __syncthreads();
    int off = 0;
    nk = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int c = s_wc[w];
      off += (w < wave) ? c : 0;
      nk += c;
    }
    if (keep) {
      const int pos = off + __popcll(m & ((1ull << lane) - 1ull));
      s_list[pos] = tid;
      uidx[(size_t)seg * rmax + pos] = r0 + tid;
    }
    if (tid == 0) ucnt[seg] = nk;
    __syncthreads();
  }

  // ---- W_up rows of the kept neurons: h = a * u
  for (int k = wave; !kFused && k < nk; k += NB * kWaves) {
    load_row(wa, wu + (size_t)(r0 + s_list[k]) * nch, lane, nch, true);
    const int k1 = k + kWaves;
    if (NB == 2) load_row(wb, wu + (size_t)(r0 + s_list[k1 < nk ? k1 : k]) * nch, lane, nch, k1 < nk);
    const float u = row_dot(wa, xs, lane, nch);
    if (lane == 0) s_h[k] = s_a[s_list[k]] * u;
    if (NB == 2 && k1 < nk) {
      const float u1 = row_dot(wb, xs, lane, nch);
      if (lane == 0) s_h[k1] = s_a[s_list[k1]] * u1;
    }
  }
  const int P = kThreads / nch;  // row groups (nch <= 1024)
  const int c = tid % nch, p = tid / nch;
  // dense: the first W_down rows are known before h, so they are requested before the barrier
  uint4 wpre[kDownUnroll];
  if (kFused && p < P) {
#pragma unroll
    for (int u = 0; u < kDownUnroll; ++u) {
      const int k = p + u * P;
      wpre[u] = (k < nk) ? ld_stream(wd + (size_t)(r0 + k) * nch + c) : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __syncthreads();  // s_h complete; x no longer needed

  // ---- W_down rows of the kept neurons: thread (p, c), rows p, p + P, ...
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (p < P) {
    for (int k0 = p; k0 < nk; k0 += P * kDownUnroll) {
      uint4 w[kDownUnroll];
      if (kFused && k0 == p) {
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) w[u] = wpre[u];
      } else {
#pragma unroll
        for (int u = 0; u < kDownUnroll; ++u) {
          const int k = k0 + u * P;
          w[u] = (k < nk) ? ld_stream(wd + (size_t)(r0 + s_list[k]) * nch + c)
                          : make_uint4(0u, 0u, 0u, 0u);
        }
      }
#pragma unroll
      for (int u = 0; u < kDownUnroll; ++u) {
        const int k = k0 + u * P;
        if (k < nk) axpy8(s_h[k], w[u], acc);
      }
    }
    s_x4[p * nv4 + 2 * c] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    s_x4[p * nv4 + 2 * c + 1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
  __syncthreads();
  float4* out = reinterpret_cast<float4*>(part + (size_t)seg * d);
  for (int i = tid; i < nv4; i += kThreads) {
    float4 s = s_x4[i];
    for (int q = 1; q < P; ++q) {
      const float4 v = s_x4[q * nv4 + i];
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
    out[i] = s;
  }
}

int pow2_cpl(int nch) {
  int p = 1;
  while (p * kWave < nch && p < 16) p <<= 1;
  return p;
}

template <int MODE>
hipError_t launch_mode(int cpl, int G, hipStream_t s, const float* x, const uint4* wg,
                       const uint4* wu, const uint4* wd, int d, int F, float t, float norm_eps,
                       int rmax, int32_t* uidx, int32_t* ucnt, float* part, const float* act,
                       const unsigned long long* cut, float* act_out = nullptr) {
#define SIRIUS_DECODE1(CPLV)                                                                    \
  case CPLV:                                                                                    \
    klaunch(decode1_kernel<CPLV, MODE>, G, kThreads, 0, s, x, wg, wu, wd, d, F, t, norm_eps, rmax,    \
                                                      uidx, ucnt, part, act, cut, act_out);     \
    break;
  switch (cpl) {
    SIRIUS_DECODE1(1)
    SIRIUS_DECODE1(2)
    SIRIUS_DECODE1(4)
    SIRIUS_DECODE1(8)
    SIRIUS_DECODE1(16)
    default:
      return hipErrorInvalidValue;
  }
#undef SIRIUS_DECODE1
  return hipGetLastError();
}

}  // namespace

Decode1Layout decode1_layout(int d, int F) {
  Decode1Layout L{};
  L.nseg = std::max(1, std::min(kSegs, ceil_div(F, kMinRows)));
  L.rmax = ceil_div(F, L.nseg);
  Carve c;
  L.uidx = c.take((size_t)L.nseg * L.rmax * 4);
  L.ucnt = c.take((size_t)L.nseg * 4);
  L.part = c.take((size_t)L.nseg * d * 4);
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_decode1(const float* x, const uint16_t* wg, const uint16_t* wu,
                              const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                              const float* resid, float* y, int32_t* active_idx,
                              int32_t* active_cnt, char* ws, const Decode1Layout& L,
                              hipStream_t stream, const float* act,
                              const unsigned long long* cut) {
  if (d > kMaxD || (d & 7) != 0 || L.rmax > kMaxRows || L.nseg > kSegs) return hipErrorInvalidValue;
  if (mode == kFfnModeTopK && (act == nullptr || cut == nullptr)) return hipErrorInvalidValue;
  int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.uidx);
  int32_t* ucnt = reinterpret_cast<int32_t*>(ws + L.ucnt);
  float* part = reinterpret_cast<float*>(ws + L.part);
  const uint4* wg4 = reinterpret_cast<const uint4*>(wg);
  const uint4* wu4 = reinterpret_cast<const uint4*>(wu);
  const uint4* wd4 = reinterpret_cast<const uint4*>(wd);
  const int cpl = pow2_cpl(d / 8);
  const bool thr = mode == kFfnModeThreshold, topk = mode == kFfnModeTopK;
  hipError_t e;
  {
    ProfScope prof(topk ? "topk_decode" : (thr ? "cats_decode" : "dense_decode"), stream);
    if (topk)
      e = launch_mode<kModeKeyed>(cpl, L.nseg, stream, x, wg4, wu4, wd4, d, F, t, norm_eps, L.rmax,
                                  uidx, ucnt, part, act, cut);
    else if (thr)
      e = launch_mode<kModeSparse>(cpl, L.nseg, stream, x, wg4, wu4, wd4, d, F, t, norm_eps,
                                   L.rmax, uidx, ucnt, part, nullptr, nullptr);
    else
      e = launch_mode<kModeDense>(cpl, L.nseg, stream, x, wg4, wu4, wd4, d, F, t, norm_eps, L.rmax,
                                  uidx, ucnt, part, nullptr, nullptr);
    if (e != hipSuccess) return e;
  }
  ProfScope prof(topk ? "topk_reduce" : (thr ? "cats_reduce" : "dense_reduce"), stream);
  if (mode != kFfnModeDense && active_idx != nullptr)
    return launch_reduce(part, L.nseg, 1, d, resid, y, stream, F, L.nseg, L.rmax, uidx, ucnt,
                         active_idx, active_cnt);
  return launch_reduce(part, L.nseg, 1, d, resid, y, stream);
}

hipError_t launch_decode1_act(const float* x, const uint16_t* wg, int d, int F, float norm_eps,
                              float* act, hipStream_t stream) {
  const Decode1Layout L = decode1_layout(d, F);
  if (d > kMaxD || (d & 7) != 0 || L.rmax > kMaxRows || L.nseg > kSegs) return hipErrorInvalidValue;
  ProfScope prof("topk_gate", stream);
  return launch_mode<kModeAct>(pow2_cpl(d / 8), L.nseg, stream, x, reinterpret_cast<const uint4*>(wg),
                               nullptr, nullptr, d, F, 0.f, norm_eps, L.rmax, nullptr, nullptr, nullptr,
                               nullptr, nullptr, act);
}

}  // namespace sirius
