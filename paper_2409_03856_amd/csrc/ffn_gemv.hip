// Small-batch SwiGLU FFN decode on gfx950: dense and per-token threshold sparsity.
//
// Three kernels per call, all HBM-bound (about one bf16 weight is read per
// two flops):
//
//  gate_kernel   one wave per neuron row. The gate row is read with 16-byte
//                loads (1 KiB per wave instruction) against fp32 x staged in
//                LDS, reduced across the wave, passed through SiLU and the
//                threshold. Only when some token keeps the neuron is its W_up
//                row read, giving h_bi = a_bi * u_bi (0 for tokens that drop
//                it). A wave ballot + popcount then compacts the kept rows of
//                each 32-row tile, in ascending order, into a per-tile list.
//  down_kernel   y += h_i * W_down[i] over the kept rows only. A grid of
//                (column slice of 512) x (row range) workgroups; the row
//                ranges split the compacted list evenly whatever its length,
//                so every workgroup reads the same number of bytes. Each
//                lane accumulates 8 output columns per token in registers.
//  reduce_kernel sums the row-range partials in a fixed order (so results are
//                bitwise reproducible), adds the residual, and builds the
//                per-token ascending active lists of the C ABI.
//
// Dense mode is the same pipeline with every neuron kept; sparse mode reads
// W_up and W_down rows only for the union of the tokens' active sets.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

constexpr int kTile = 32;                 // neuron rows per gate workgroup
constexpr int kGateWaves = 4;
constexpr int kRowsPerWave = kTile / kGateWaves;
constexpr int kDownWaves = 4;
constexpr int kListCap = 512;             // kept rows resolved per pass in down_kernel
constexpr int kMaxTiles = 65536 / kTile;  // d_ff <= 65536
constexpr int kXLdsFloats = 15360;        // fp32 x staged in LDS: 60 KiB (+ static LDS < 64 KiB)
constexpr int kDownBlocks = 512;          // target workgroups of down_kernel

constexpr int kModeDense = 0, kModeSparse = 1, kModeAbsAct = 2;

// Dot product of 8 bf16 weights (one 16-byte load) with 8 fp32 activations from LDS.
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

template <int BM, int CPL>
__global__ __launch_bounds__(256) void gate_kernel(
    const float* __restrict__ x, int B, const uint4* __restrict__ wg, const uint4* __restrict__ wu,
    int d, int F, int mode, float t, float norm_eps, int32_t* __restrict__ uidx,
    float* __restrict__ hbuf, int32_t* __restrict__ ucnt, int32_t* __restrict__ bidx,
    int32_t* __restrict__ bcnt, int ntiles, float* __restrict__ absact) {
  extern __shared__ float xs[];  // [B][d] fp32
  __shared__ float s_h[kTile * BM];
  __shared__ uint32_t s_flag[kTile];
  __shared__ float s_ss[kGateWaves][BM];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int tile = blockIdx.x;
  const int nch = d >> 3;  // 16-byte chunks per row
  const int nv4 = d >> 2;

  // ---- stage x in LDS (optionally RMS-normalised with unit weight)
  float ss[BM];
#pragma unroll
  for (int b = 0; b < BM; ++b) ss[b] = 0.f;
  const float4* x4 = reinterpret_cast<const float4*>(x);
  float4* xs4 = reinterpret_cast<float4*>(xs);
#pragma unroll
  for (int b = 0; b < BM; ++b) {
    if (b < B) {
      for (int i = tid; i < nv4; i += 256) {
        const float4 v = x4[(size_t)b * nv4 + i];
        xs4[b * nv4 + i] = v;
        ss[b] = fmaf(v.x, v.x, ss[b]);
        ss[b] = fmaf(v.y, v.y, ss[b]);
        ss[b] = fmaf(v.z, v.z, ss[b]);
        ss[b] = fmaf(v.w, v.w, ss[b]);
      }
    }
  }
  if (norm_eps >= 0.f) {
#pragma unroll
    for (int b = 0; b < BM; ++b) {
      const float s = wave_sum(ss[b]);
      if (lane == 0) s_ss[wave][b] = s;
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BM; ++b) {
      if (b < B) {
        const float tot = ((s_ss[0][b] + s_ss[1][b]) + s_ss[2][b]) + s_ss[3][b];
        const float inv = 1.0f / sqrtf(tot / (float)d + norm_eps);
        for (int i = tid; i < nv4; i += 256) {
          float4 v = xs4[b * nv4 + i];
          v.x *= inv;
          v.y *= inv;
          v.z *= inv;
          v.w *= inv;
          xs4[b * nv4 + i] = v;
        }
      }
    }
  }
  __syncthreads();

  // ---- one neuron row per wave at a time
  for (int r = 0; r < kRowsPerWave; ++r) {
    const int lr = wave * kRowsPerWave + r;
    const int row = tile * kTile + lr;
    uint32_t flags = 0u;
    float hv[BM];
#pragma unroll
    for (int b = 0; b < BM; ++b) hv[b] = 0.f;
    if (row < F) {  // wave-uniform
      uint4 w[CPL];
      const uint4* wr = wg + (size_t)row * nch;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = lane + kWave * j;
        w[j] = (c < nch) ? wr[c] : make_uint4(0u, 0u, 0u, 0u);
      }
      float acc[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) acc[b] = 0.f;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = lane + kWave * j;
        if (c < nch) {
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) acc[b] = dot8(w[j], xs + b * d + 8 * c, acc[b]);
        }
      }
      float a[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) a[b] = silu(wave_sum(acc[b]));
      if (mode == kModeAbsAct) {
        if (lane == 0) {
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) absact[(size_t)b * F + row] = fabsf(a[b]);
        }
        continue;
      }
#pragma unroll
      for (int b = 0; b < BM; ++b)
        if (b < B && (mode == kModeDense || fabsf(a[b]) > t)) flags |= 1u << b;
      if (flags != 0u) {  // wave-uniform: every lane holds the same sums
        const uint4* ur = wu + (size_t)row * nch;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          const int c = lane + kWave * j;
          w[j] = (c < nch) ? ur[c] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int b = 0; b < BM; ++b) acc[b] = 0.f;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          const int c = lane + kWave * j;
          if (c < nch) {
#pragma unroll
            for (int b = 0; b < BM; ++b)
              if (b < B) acc[b] = dot8(w[j], xs + b * d + 8 * c, acc[b]);
          }
        }
#pragma unroll
        for (int b = 0; b < BM; ++b) {
          const float u = wave_sum(acc[b]);
          hv[b] = ((flags >> b) & 1u) ? a[b] * u : 0.f;
        }
      }
    }
    if (lane == 0) {
      s_flag[lr] = flags;
#pragma unroll
      for (int b = 0; b < BM; ++b) s_h[lr * BM + b] = hv[b];
    }
  }
  if (mode == kModeAbsAct) return;  // uniform over the block
  __syncthreads();

  // ---- ballot compaction of the tile's kept rows (ascending)
  if (wave == 0) {
    const uint32_t fl = (lane < kTile) ? s_flag[lane] : 0u;
    const int row = tile * kTile + lane;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t m = __ballot(fl != 0u);
    const int slot0 = tile * kTile;
    if (fl != 0u) {
      const int pos = __popcll(m & below);
      uidx[slot0 + pos] = row;
#pragma unroll
      for (int b = 0; b < BM; ++b)
        if (b < B) hbuf[(size_t)(slot0 + pos) * B + b] = s_h[lane * BM + b];
    }
    if (lane == 0) ucnt[tile] = __popcll(m);
    if (mode == kModeSparse && bidx != nullptr) {
#pragma unroll
      for (int b = 0; b < BM; ++b) {
        if (b < B) {
          const bool on = ((fl >> b) & 1u) != 0u;
          const uint64_t mb = __ballot(on);
          if (on) bidx[(size_t)b * F + slot0 + __popcll(mb & below)] = row;
          if (lane == 0) bcnt[b * ntiles + tile] = __popcll(mb);
        }
      }
    }
  }
}

template <int BM>
__global__ __launch_bounds__(256) void down_kernel(const uint4* __restrict__ wd, int d, int B,
                                                   const int32_t* __restrict__ uidx,
                                                   const float* __restrict__ hbuf,
                                                   const int32_t* __restrict__ ucnt, int ntiles,
                                                   float* __restrict__ part) {
  __shared__ int s_pref[kMaxTiles + 1];
  __shared__ int s_row[kListCap];
  __shared__ float s_hl[kListCap * BM];
  __shared__ float s_red[kDownWaves][kWave * 8];
  __shared__ int s_tmp[4];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int nch = d >> 3;
  const int cbase = blockIdx.x * kWave;  // this workgroup's 64 chunks = 512 columns
  const int rho = blockIdx.y, gr = gridDim.y;

  // ---- exclusive prefix of the per-tile kept counts
  const int per = (ntiles + 255) / 256;
  const int beg = min(tid * per, ntiles), end = min(beg + per, ntiles);
  int local = 0;
  for (int i = beg; i < end; ++i) local += ucnt[i];
  int total;
  int run = block_exclusive_scan_256(local, s_tmp, &total);
  for (int i = beg; i < end; ++i) {
    s_pref[i] = run;
    run += ucnt[i];
  }
  if (tid == 0) s_pref[ntiles] = total;
  __syncthreads();

  // ---- this workgroup's share of the compacted list
  const int start = (int)(((long long)total * rho) / gr);
  const int stop = (int)(((long long)total * (rho + 1)) / gr);
  const int c = cbase + lane;
  const bool cv = c < nch;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);

  float acc[BM][8];
#pragma unroll
  for (int b = 0; b < BM; ++b)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[b][e] = 0.f;

  auto fma_row = [&](uint4 w, int i) {
#pragma unroll
    for (int b = 0; b < BM; ++b) {
      if (b < B) {
        const float h = s_hl[i * BM + b];
        acc[b][0] = fmaf(h, bf16_lo(w.x), acc[b][0]);
        acc[b][1] = fmaf(h, bf16_hi(w.x), acc[b][1]);
        acc[b][2] = fmaf(h, bf16_lo(w.y), acc[b][2]);
        acc[b][3] = fmaf(h, bf16_hi(w.y), acc[b][3]);
        acc[b][4] = fmaf(h, bf16_lo(w.z), acc[b][4]);
        acc[b][5] = fmaf(h, bf16_hi(w.z), acc[b][5]);
        acc[b][6] = fmaf(h, bf16_lo(w.w), acc[b][6]);
        acc[b][7] = fmaf(h, bf16_hi(w.w), acc[b][7]);
      }
    }
  };

  for (int base = start; base < stop; base += kListCap) {
    const int n = min(kListCap, stop - base);
    __syncthreads();  // previous pass finished reading s_row / s_hl
    for (int i = tid; i < n; i += 256) {
      const int p = base + i;
      int lo = 0, hi = ntiles;  // s_pref[lo] <= p < s_pref[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_pref[mid] <= p) lo = mid;
        else hi = mid;
      }
      const int slot = lo * kTile + (p - s_pref[lo]);
      s_row[i] = uidx[slot];
#pragma unroll
      for (int b = 0; b < BM; ++b)
        if (b < B) s_hl[i * BM + b] = hbuf[(size_t)slot * B + b];
    }
    __syncthreads();

    int i = wave;
    for (; i + 3 * kDownWaves < n; i += 4 * kDownWaves) {  // four rows in flight per wave
      const int r0 = s_row[i], r1 = s_row[i + kDownWaves];
      const int r2 = s_row[i + 2 * kDownWaves], r3 = s_row[i + 3 * kDownWaves];
      const uint4 w0 = cv ? wd[(size_t)r0 * nch + c] : zero;
      const uint4 w1 = cv ? wd[(size_t)r1 * nch + c] : zero;
      const uint4 w2 = cv ? wd[(size_t)r2 * nch + c] : zero;
      const uint4 w3 = cv ? wd[(size_t)r3 * nch + c] : zero;
      fma_row(w0, i);
      fma_row(w1, i + kDownWaves);
      fma_row(w2, i + 2 * kDownWaves);
      fma_row(w3, i + 3 * kDownWaves);
    }
    for (; i < n; i += kDownWaves) {
      const uint4 w0 = cv ? wd[(size_t)s_row[i] * nch + c] : zero;
      fma_row(w0, i);
    }
  }

  // ---- fixed-order reduction over the four waves, one token at a time
#pragma unroll
  for (int b = 0; b < BM; ++b) {
    if (b < B) {
      __syncthreads();
#pragma unroll
      for (int e = 0; e < 8; ++e) s_red[wave][lane * 8 + e] = acc[b][e];
      __syncthreads();
      for (int q = tid; q < kWave * 8; q += 256) {
        const int col = cbase * 8 + q;
        if (col < d)
          part[((size_t)rho * B + b) * d + col] =
              ((s_red[0][q] + s_red[1][q]) + s_red[2][q]) + s_red[3][q];
      }
    }
  }
}

__global__ __launch_bounds__(256) void reduce_kernel(
    const float* __restrict__ part, int gr, int n, const float* resid, float* y, int nred, int B,
    int F, int ntiles, const int32_t* __restrict__ bidx, const int32_t* __restrict__ bcnt,
    int32_t* __restrict__ active_idx, int32_t* __restrict__ active_cnt) {
  __shared__ float s_red[4][kWave];
  __shared__ int s_tmp[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  if ((int)blockIdx.x < nred) {
    const int o = blockIdx.x * kWave + lane;
    float s = 0.f;
    if (o < n)
      for (int rho = wave; rho < gr; rho += 4) s += part[(size_t)rho * n + o];
    s_red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && o < n) {
      float v = ((s_red[0][lane] + s_red[1][lane]) + s_red[2][lane]) + s_red[3][lane];
      if (resid != nullptr) v = resid[o] + v;
      y[o] = v;
    }
    return;
  }
  // ---- ascending active list of token b
  const int b = blockIdx.x - nred;
  const int per = (ntiles + 255) / 256;
  const int beg = min(tid * per, ntiles), end = min(beg + per, ntiles);
  int local = 0;
  for (int i = beg; i < end; ++i) local += bcnt[b * ntiles + i];
  int total;
  int run = block_exclusive_scan_256(local, s_tmp, &total);
  for (int i = beg; i < end; ++i) {
    const int cnt = bcnt[b * ntiles + i];
    for (int j = 0; j < cnt; ++j)
      active_idx[(size_t)b * F + run + j] = bidx[(size_t)b * F + i * kTile + j];
    run += cnt;
  }
  if (tid == 0) active_cnt[b] = total;
}

int pow2_at_least(int v, int cap) {
  int p = 1;
  while (p < v && p < cap) p <<= 1;
  return p;
}

template <int BM>
hipError_t launch_gate_bm(int cpl, dim3 grid, size_t lds, hipStream_t s, const float* x, int B,
                          const uint4* wg, const uint4* wu, int d, int F, int mode, float t,
                          float norm_eps, int32_t* uidx, float* hbuf, int32_t* ucnt, int32_t* bidx,
                          int32_t* bcnt, int ntiles, float* absact) {
#define SIRIUS_GATE(CPLV)                                                                          \
  case CPLV:                                                                                       \
    gate_kernel<BM, CPLV><<<grid, 256, lds, s>>>(x, B, wg, wu, d, F, mode, t, norm_eps, uidx,      \
                                                 hbuf, ucnt, bidx, bcnt, ntiles, absact);          \
    break;
  switch (cpl) {
    SIRIUS_GATE(1)
    SIRIUS_GATE(2)
    SIRIUS_GATE(4)
    SIRIUS_GATE(8)
    SIRIUS_GATE(16)
    default:
      return hipErrorInvalidValue;
  }
#undef SIRIUS_GATE
  return hipGetLastError();
}

hipError_t launch_gate(int bm, int cpl, dim3 grid, size_t lds, hipStream_t s, const float* x,
                       int B, const uint4* wg, const uint4* wu, int d, int F, int mode, float t,
                       float norm_eps, int32_t* uidx, float* hbuf, int32_t* ucnt, int32_t* bidx,
                       int32_t* bcnt, int ntiles, float* absact) {
  switch (bm) {
    case 1: return launch_gate_bm<1>(cpl, grid, lds, s, x, B, wg, wu, d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, ntiles, absact);
    case 2: return launch_gate_bm<2>(cpl, grid, lds, s, x, B, wg, wu, d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, ntiles, absact);
    case 4: return launch_gate_bm<4>(cpl, grid, lds, s, x, B, wg, wu, d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, ntiles, absact);
    case 8: return launch_gate_bm<8>(cpl, grid, lds, s, x, B, wg, wu, d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, ntiles, absact);
    case 16: return launch_gate_bm<16>(cpl, grid, lds, s, x, B, wg, wu, d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, ntiles, absact);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

GemvLayout gemv_layout(int B, int d, int F) {
  GemvLayout L{};
  L.bc = std::max(1, std::min(std::min(B, 16), kXLdsFloats / d));
  L.ntiles = ceil_div(F, kTile);
  const int nch = d / 8;
  L.cs = ceil_div(nch, kWave);
  L.gr = std::max(1, std::min(kDownBlocks / L.cs, ceil_div(F, 8)));
  Carve c;
  L.uidx = c.take((size_t)F * 4);
  L.h = c.take((size_t)F * L.bc * 4);
  L.ucnt = c.take((size_t)L.ntiles * 4);
  L.bidx = c.take((size_t)L.bc * F * 4);
  L.bcnt = c.take((size_t)L.bc * L.ntiles * 4);
  L.part = c.take((size_t)L.gr * L.bc * d * 4);
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_gemv(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                           const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                           char* ws, const GemvLayout& L, hipStream_t stream) {
  if (B < 1 || B > L.bc) return hipErrorInvalidValue;
  const int bm = pow2_at_least(B, 16);
  const int cpl = pow2_at_least(ceil_div(d / 8, kWave), 16);
  int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.uidx);
  float* hbuf = reinterpret_cast<float*>(ws + L.h);
  int32_t* ucnt = reinterpret_cast<int32_t*>(ws + L.ucnt);
  const bool lists = (mode == kModeSparse) && active_idx != nullptr;
  int32_t* bidx = lists ? reinterpret_cast<int32_t*>(ws + L.bidx) : nullptr;
  int32_t* bcnt = lists ? reinterpret_cast<int32_t*>(ws + L.bcnt) : nullptr;
  float* part = reinterpret_cast<float*>(ws + L.part);
  const size_t lds = (size_t)B * d * sizeof(float);

  hipError_t e;
  {
    ProfScope prof("cats_gate", stream);
    e = launch_gate(bm, cpl, dim3(L.ntiles), lds, stream, x, B,
                             reinterpret_cast<const uint4*>(wg), reinterpret_cast<const uint4*>(wu),
                    d, F, mode, t, norm_eps, uidx, hbuf, ucnt, bidx, bcnt, L.ntiles, nullptr);
  }
  if (e != hipSuccess) return e;

  const dim3 dgrid(L.cs, L.gr);
  const uint4* wd4 = reinterpret_cast<const uint4*>(wd);
  {
  ProfScope prof("ffn_down", stream);
  switch (bm) {
    case 1: down_kernel<1><<<dgrid, 256, 0, stream>>>(wd4, d, B, uidx, hbuf, ucnt, L.ntiles, part); break;
    case 2: down_kernel<2><<<dgrid, 256, 0, stream>>>(wd4, d, B, uidx, hbuf, ucnt, L.ntiles, part); break;
    case 4: down_kernel<4><<<dgrid, 256, 0, stream>>>(wd4, d, B, uidx, hbuf, ucnt, L.ntiles, part); break;
    case 8: down_kernel<8><<<dgrid, 256, 0, stream>>>(wd4, d, B, uidx, hbuf, ucnt, L.ntiles, part); break;
    case 16: down_kernel<16><<<dgrid, 256, 0, stream>>>(wd4, d, B, uidx, hbuf, ucnt, L.ntiles, part); break;
    default: return hipErrorInvalidValue;
  }
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;

  const int n = B * d;
  ProfScope prof("ffn_reduce", stream);
  const int nred = ceil_div(n, kWave);
  reduce_kernel<<<nred + (lists ? B : 0), 256, 0, stream>>>(part, L.gr, n, resid, y, nred, B, F,
                                                             L.ntiles, bidx, bcnt, active_idx,
                                                             active_cnt);
  return hipGetLastError();
}

hipError_t launch_gate_absact(const float* x, int N, const uint16_t* wg, int d, int F,
                              float* absact, hipStream_t stream) {
  const int bc = std::max(1, std::min(16, kXLdsFloats / d));
  const int cpl = pow2_at_least(ceil_div(d / 8, kWave), 16);
  const int ntiles = ceil_div(F, kTile);
  for (int b0 = 0; b0 < N; b0 += bc) {
    const int nb = std::min(bc, N - b0);
    const int bm = pow2_at_least(nb, 16);
    ProfScope prof("cats_gate", stream);
    hipError_t e = launch_gate(bm, cpl, dim3(ntiles), (size_t)nb * d * sizeof(float), stream,
                               x + (size_t)b0 * d, nb, reinterpret_cast<const uint4*>(wg), nullptr,
                               d, F, kModeAbsAct, 0.f, -1.f, nullptr, nullptr, nullptr, nullptr,
                               nullptr, ntiles, absact + (size_t)b0 * F);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sirius
