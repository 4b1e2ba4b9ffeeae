// Small-batch SwiGLU FFN decode on gfx950, dense and per-token threshold sparsity (FSparse
// after CATS: the gate is read whole, up and down only for neurons some token keeps), and
// the calibration pass. Batched calls whose d_model is not a multiple of 256 run here in chunks
// of up to 8 tokens (threshold sparsity and top-k at any batch, dense and condensed with 2 to 7
// tokens); batch 1 runs the one-pass kernel of ffn_decode.hip, batches of 2..64 with d_model a
// multiple of 256 the batched MFMA kernels of ffn_batch.hip, and the remaining dense calls
// with 8 or more tokens the MFMA kernels of ffn_mfma.hip. The reduce kernel below serves all.
//
// Three kernels per call, HBM-bound (one bf16 weight per two flops per token). No grid-wide
// barrier, atomics or fences: workgroups hand results to each other only through kernel
// boundaries, and every sum has a fixed order (bitwise reproducible).
//
//  gate_kernel   a workgroup owns one contiguous segment of neuron rows (1024 segments at
//                most, four per CU). x (up to 8 tokens) is staged in LDS, optionally RMS-
//                normalised; each wave streams gate rows two at a time (16-byte loads, 1 KiB
//                per wave instruction), reduces across the wave, applies SiLU and the
//                threshold per token; a block scan compacts the rows some token keeps, in
//                ascending order; the W_up rows of those neurons are then streamed and
//                h_bi = a_bi * u_bi (0 for tokens that drop the neuron) stored with the
//                segment's kept list. Per-token lists go to a side buffer for the outputs.
//  down_kernel   partial y over the kept rows only. Grid: (512-column slice) x (row range
//                of the concatenated kept lists, split evenly by position, so every
//                workgroup reads the same number of bytes whatever the sparsity pattern).
//                A wave reads whole 1 KiB row chunks (16 rows in flight) and each lane
//                accumulates 8 output columns per token; the four waves are summed in a
//                fixed order into one partial per workgroup. (Owning columns instead, to
//                avoid partials, means 32-byte reads per row, and the per-CU limit on
//                outstanding line requests then caps useful bandwidth near a quarter.)
//  reduce_kernel y = resid + the row-range partials summed in order (one output per thread with
//                every row in flight for at most 16 rows and 256K outputs or more); extra
//                blocks build the per-token ascending active lists.



#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "topk.h"

namespace sirius {
namespace {

constexpr int kRPW = 2;                     // rows in flight per gate wave
constexpr int kGateWaves = 4;
constexpr int kGateSegs = 1024;             // gate workgroups: four per CU on a 256-CU part
constexpr int kListSegs = 2048;             // per-segment kept lists the reduce kernel can join
constexpr int kMaxSeg = 256;                // rows per gate workgroup at most (d_ff <= 65536)
constexpr int kDownWaves = 4;
constexpr int kDownUnroll = 16;             // full-row chunks in flight per down wave
// kept rows resolved per pass in down_kernel (h staged for BM tokens: <= 16 KiB of LDS)
template <int BM>
constexpr int range_cap() { return BM >= 8 ? 256 : 1024; }
constexpr int kDownBlocks = 512;            // target workgroups of down_kernel
constexpr int kListBlocks = 16;             // workgroups copying each token's active list
constexpr int kMaxSegs = 4096;              // row segments a down launch can take (d_ff / 16)
constexpr int kRedOut4 = 16;                // float4 outputs per reduce workgroup
constexpr int kRedGroups = 256 / kRedOut4;  // partial-row groups per reduce workgroup
constexpr int kRedUnroll = 16;              // partial rows in flight per reduce thread (one round
                                            // for up to 256 partial rows)
constexpr int kXLdsFloats = 32768;          // fp32 x staged in LDS: 128 KiB (LDS is 160 KiB)

// kModeAct writes the signed gate activations and stops; kModeKeyed takes them (and a per-token
// top-k key cut) from that pass instead of reading W_gate again.
constexpr int kModeDense = 0, kModeSparse = 1, kModeAbsAct = 2, kModeAct = 3, kModeKeyed = 4;
constexpr bool writes_act(int mode) { return mode == kModeAbsAct || mode == kModeAct; }

template <int BM, int CPL, int MODE>
__global__ __launch_bounds__(256) void gate_kernel(
    const float* __restrict__ x, int B, const uint4* __restrict__ wg, const uint4* __restrict__ wu,
    int d, int F, float t, float norm_eps, int rmax, int32_t* __restrict__ uidx,
    float* __restrict__ hbuf, int32_t* __restrict__ ucnt, int32_t* __restrict__ bidx,
    int32_t* __restrict__ bcnt, float* __restrict__ absact,
    const unsigned long long* __restrict__ cut) {
  extern __shared__ float xs[];  // [B][d] fp32
  __shared__ float s_a[kMaxSeg * BM];
  __shared__ uint32_t s_flag[kMaxSeg];
  __shared__ int s_list[kMaxSeg];
  __shared__ float s_ss[kGateWaves][BM];
  __shared__ int s_tmp[4];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int seg = blockIdx.x, G = gridDim.x;
  const int nch = d >> 3;  // 16-byte chunks per row
  const int nv4 = d >> 2;
  const int r0 = (int)(((long long)F * seg) / G);
  const int nr = (int)(((long long)F * (seg + 1)) / G) - r0;  // <= rmax <= kMaxSeg

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

  uint4 w[kRPW][CPL];
  if (MODE == kModeKeyed) {
    // ---- phase a from the stored activations: kept iff the top-k key reaches the cut
    for (int j = tid; j < nr; j += 256) {
      uint32_t fl = 0u;
#pragma unroll
      for (int b = 0; b < BM; ++b) {
        const float a = (b < B) ? absact[(size_t)b * F + r0 + j] : 0.f;
        if (b < B && topk_key(a, r0 + j) >= cut[b]) fl |= 1u << b;
        s_a[j * BM + b] = a;
      }
      s_flag[j] = fl;
    }
  }
  // ---- phase a: gate rows j = wave, wave + 4, ... of the segment, kRPW rows in flight
  for (int j0 = wave; MODE != kModeKeyed && j0 < nr; j0 += kRPW * kGateWaves) {
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const int j = j0 + r * kGateWaves;
      const uint4* wr = wg + (size_t)(r0 + j) * nch;
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const int c = lane + kWave * q;
        w[r][q] = (j < nr && c < nch) ? ld_stream(wr + c) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const int j = j0 + r * kGateWaves;
      float acc[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) acc[b] = 0.f;
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const int c = lane + kWave * q;
        if (c < nch) {
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) acc[b] = dot8(w[r][q], xs + b * d + 8 * c, acc[b]);
        }
      }
      uint32_t fl = 0u;
      float a[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) {
        a[b] = silu(wave_sum(acc[b]));  // every lane holds the row's sums
        if (b < B && (MODE == kModeDense || fabsf(a[b]) > t)) fl |= 1u << b;
      }
      if (lane == 0 && j < nr) {
        if (writes_act(MODE)) {
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) absact[(size_t)b * F + r0 + j] = (MODE == kModeAbsAct) ? fabsf(a[b]) : a[b];
        } else {
          s_flag[j] = fl;
#pragma unroll
          for (int b = 0; b < BM; ++b) s_a[j * BM + b] = a[b];
        }
      }
    }
  }
  if (writes_act(MODE)) return;  // uniform over the block
  __syncthreads();

  // ---- compact the segment's kept rows (some token keeps them), ascending
  const uint32_t myfl = (tid < nr) ? s_flag[tid] : 0u;
  int nkept;
  const int pos = block_exclusive_scan_256(myfl != 0u ? 1 : 0, s_tmp, &nkept);
  if (myfl != 0u) s_list[pos] = tid;
  if ((MODE == kModeSparse || MODE == kModeKeyed) && bidx != nullptr) {
#pragma unroll
    for (int b = 0; b < BM; ++b) {
      if (b < B) {
        const int on = (myfl >> b) & 1u;
        int nb;
        const int pb = block_exclusive_scan_256(on, s_tmp, &nb);
        if (on) bidx[(size_t)b * G * rmax + (size_t)seg * rmax + pb] = r0 + tid;
        if (tid == 0) bcnt[b * G + seg] = nb;
      }
    }
  }
  __syncthreads();

  // ---- phase b: W_up rows of the kept rows, shared evenly by the waves, kRPW in flight
  for (int k0 = wave; k0 < nkept; k0 += kRPW * kGateWaves) {
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const int k = k0 + r * kGateWaves;
      const uint4* ur = wu + (size_t)(r0 + (k < nkept ? s_list[k] : 0)) * nch;
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const int c = lane + kWave * q;
        w[r][q] = (k < nkept && c < nch) ? ld_stream(ur + c) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int r = 0; r < kRPW; ++r) {
      const int k = k0 + r * kGateWaves;
      float acc[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) acc[b] = 0.f;
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const int c = lane + kWave * q;
        if (c < nch) {
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) acc[b] = dot8(w[r][q], xs + b * d + 8 * c, acc[b]);
        }
      }
      float u[BM];
#pragma unroll
      for (int b = 0; b < BM; ++b) u[b] = wave_sum(acc[b]);
      if (lane == 0 && k < nkept) {
        const int j = s_list[k];
        const uint32_t fl = s_flag[j];
        const size_t slot = (size_t)seg * rmax + k;
        uidx[slot] = r0 + j;
#pragma unroll
        for (int b = 0; b < BM; ++b)
          if (b < B) hbuf[slot * B + b] = ((fl >> b) & 1u) ? s_a[j * BM + b] * u[b] : 0.f;
      }
    }
  }
  if (tid == 0) ucnt[seg] = nkept;
}

template <int BM>
__global__ __launch_bounds__(256) void down_kernel(
    const uint4* __restrict__ wd, int d, int B, const int32_t* __restrict__ uidx,
    const float* __restrict__ hbuf, int hstride, const int32_t* __restrict__ ucnt, int ntiles,
    int rmax, int gr, float* __restrict__ part) {
  __shared__ int s_pref[kMaxSegs + 1];
  constexpr int kRangeCap = range_cap<BM>();
  __shared__ int s_row[kRangeCap];
  __shared__ float s_h[kRangeCap * BM];
  __shared__ float4 s_red[kDownWaves][kWave * 2];
  __shared__ int s_tmp[4];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int nch = d >> 3;
  const int kap = blockIdx.x;  // column slice: chunks [64*kap, 64*kap + 64) = 512 columns
  const int rho = blockIdx.y;  // row range of the compacted list

  // ---- exclusive prefix of the per-segment kept counts
  {
    const int per = (ntiles + 255) / 256;
    const int beg = min(tid * per, ntiles), end = min(beg + per, ntiles);
    int local = 0;
    for (int i = beg; i < end; ++i) local += ucnt[i];
    int tot;
    int run = block_exclusive_scan_256(local, s_tmp, &tot);
    for (int i = beg; i < end; ++i) {
      s_pref[i] = run;
      run += ucnt[i];
    }
    if (tid == 0) s_pref[ntiles] = tot;
    __syncthreads();
  }
  const int total = s_pref[ntiles];
  const int start = (int)(((long long)total * rho) / gr);
  const int stop = (int)(((long long)total * (rho + 1)) / gr);
  const int c = kap * kWave + lane;
  const bool cv = c < nch;

  float acc[BM][8];
#pragma unroll
  for (int b = 0; b < BM; ++b)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[b][e] = 0.f;

  for (int base = start; base < stop; base += kRangeCap) {
    const int n = min(kRangeCap, stop - base);
    __syncthreads();  // previous pass done with s_row / s_h
    // segments holding positions base and base + n - 1 (same search in every thread)
    auto seg_of = [&](int p) {
      int lo = 0, hi = ntiles;  // s_pref[lo] <= p < s_pref[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_pref[mid] <= p) lo = mid;
        else hi = mid;
      }
      return lo;
    };
    const int seg_lo = seg_of(base), seg_hi = seg_of(base + n - 1);
    const int nslot = (seg_hi - seg_lo + 1) * rmax;
    // flattened (segment, entry) slots of those segments; 4 independent loads per thread
    for (int q0 = tid; q0 < nslot; q0 += 4 * 256) {
      int rv[4], pv[4];
      float hv[4][BM];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int q = q0 + 256 * u, i = seg_lo + q / rmax, j = q % rmax;
        const int p = (q < nslot) ? s_pref[i] + j : -1;
        const bool ok = q < nslot && p < s_pref[i + 1] && p >= base && p < base + n;
        const size_t slot = (size_t)i * rmax + j;
        pv[u] = ok ? p - base : -1;
        rv[u] = ok ? uidx[slot] : 0;
#pragma unroll
        for (int b = 0; b < BM; ++b) hv[u][b] = (ok && b < B) ? hbuf[slot * hstride + b] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (pv[u] >= 0) {
          s_row[pv[u]] = rv[u];
#pragma unroll
          for (int b = 0; b < BM; ++b)
            if (b < B) s_h[pv[u] * BM + b] = hv[u][b];
        }
      }
    }
    __syncthreads();
    // wave v takes rows v, v + 4, ...; kDownUnroll full-row chunks (1 KiB each) in flight
    for (int i0 = wave; i0 < n; i0 += kDownUnroll * kDownWaves) {
      uint4 w[kDownUnroll];
#pragma unroll
      for (int u = 0; u < kDownUnroll; ++u) {
        const int i = i0 + u * kDownWaves;
        w[u] = (i < n && cv) ? ld_stream(wd + (size_t)s_row[i] * nch + c) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < kDownUnroll; ++u) {
        const int i = i0 + u * kDownWaves;
        if (i < n) {
#pragma unroll
          for (int b = 0; b < BM; ++b) {
            if (b < B) {
              const float h = s_h[i * BM + b];
              acc[b][0] = fmaf(h, bf16_lo(w[u].x), acc[b][0]);
              acc[b][1] = fmaf(h, bf16_hi(w[u].x), acc[b][1]);
              acc[b][2] = fmaf(h, bf16_lo(w[u].y), acc[b][2]);
              acc[b][3] = fmaf(h, bf16_hi(w[u].y), acc[b][3]);
              acc[b][4] = fmaf(h, bf16_lo(w[u].z), acc[b][4]);
              acc[b][5] = fmaf(h, bf16_hi(w[u].z), acc[b][5]);
              acc[b][6] = fmaf(h, bf16_lo(w[u].w), acc[b][6]);
              acc[b][7] = fmaf(h, bf16_hi(w[u].w), acc[b][7]);
            }
          }
        }
      }
    }
  }

  // ---- fixed-order sum of the four waves, one partial slice per token
  const int col0 = kap * kWave * 8;
#pragma unroll
  for (int b = 0; b < BM; ++b) {
    if (b < B) {
      __syncthreads();
      s_red[wave][2 * lane] = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
      s_red[wave][2 * lane + 1] = make_float4(acc[b][4], acc[b][5], acc[b][6], acc[b][7]);
      __syncthreads();
      if (tid < 2 * kWave) {  // 128 float4 = 512 columns
        const int col = col0 + 4 * tid;
        if (col < d) {
          const float4 p0 = s_red[0][tid], p1 = s_red[1][tid], p2 = s_red[2][tid], p3 = s_red[3][tid];
          float4 s;
          s.x = ((p0.x + p1.x) + p2.x) + p3.x;
          s.y = ((p0.y + p1.y) + p2.y) + p3.y;
          s.z = ((p0.z + p1.z) + p2.z) + p3.z;
          s.w = ((p0.w + p1.w) + p2.w) + p3.w;
          *reinterpret_cast<float4*>(part + ((size_t)rho * B + b) * d + col) = s;
        }
      }
    }
  }
}

// The one-output-per-thread form of the sums (below) when there are at most 16 partial rows and
// enough outputs for 256 workgroups; with fewer outputs the grouped form keeps more workgroups
// busy. Both give the same bits.
__host__ __device__ constexpr bool red_wide(int gr, int n) {
  return gr <= kRedGroups && n >= 4 * 256 * 256;
}

// y = resid + sum over the gr row-range partials in order (bitwise reproducible); the blocks
// past the reduction build the per-token ascending active lists.
__global__ __launch_bounds__(256) void reduce_kernel(
    const float* __restrict__ part, int gr, int n, const float* resid, float* y, int nred, int B,
    int F, int ntiles, int rmax, const int32_t* __restrict__ bidx, const int32_t* __restrict__ bcnt,
    int32_t* __restrict__ active_idx, int32_t* __restrict__ active_cnt) {
  __shared__ float4 s_red[kRedGroups][kRedOut4];
  __shared__ int s_tmp[4];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x < nred && red_wide(gr, n)) {
    // at most 16 partial rows: one float4 output per thread with every row's load in flight
    // (each row read 4 KiB contiguous per block), added in the order of the grouped sum below,
    // whose group g then holds 0 + row g: the same bits
    const int o4 = blockIdx.x * 256 + tid;
    if (4 * o4 >= n) return;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    const size_t stride4 = (size_t)(n >> 2);
    float4 v[kRedGroups];
#pragma unroll
    for (int r = 0; r < kRedGroups; ++r)
      v[r] = r < gr ? p4[(size_t)r * stride4 + o4] : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 s = make_float4(0.f + v[0].x, 0.f + v[0].y, 0.f + v[0].z, 0.f + v[0].w);
#pragma unroll
    for (int r = 1; r < kRedGroups; ++r) {
      s.x += 0.f + v[r].x;
      s.y += 0.f + v[r].y;
      s.z += 0.f + v[r].z;
      s.w += 0.f + v[r].w;
    }
    if (resid != nullptr) {
      const float4 rv = reinterpret_cast<const float4*>(resid)[o4];
      s.x = rv.x + s.x;
      s.y = rv.y + s.y;
      s.z = rv.z + s.z;
      s.w = rv.w + s.w;
    }
    reinterpret_cast<float4*>(y)[o4] = s;
    return;
  }
  if ((int)blockIdx.x < nred) {
    // kRedOut4 float4 outputs per block; thread (o, g) sums partial rows g, g + 16, ... of
    // output o with kRedUnroll loads in flight; the 16 groups are then added in order
    const int o = tid % kRedOut4, g = tid / kRedOut4;
    const int o4 = blockIdx.x * kRedOut4 + o;
    const bool ov = 4 * o4 < n;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4* p4 = reinterpret_cast<const float4*>(part);
    const size_t stride4 = (size_t)(n >> 2);
    for (int r0 = g; r0 < gr; r0 += kRedUnroll * kRedGroups) {
      float4 v[kRedUnroll];
#pragma unroll
      for (int u = 0; u < kRedUnroll; ++u) {
        const int r = r0 + kRedGroups * u;
        v[u] = (ov && r < gr) ? p4[(size_t)r * stride4 + o4] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < kRedUnroll; ++u) {
        s.x += v[u].x;
        s.y += v[u].y;
        s.z += v[u].z;
        s.w += v[u].w;
      }
    }
    s_red[g][o] = s;
    __syncthreads();
    if (tid < kRedOut4 && ov) {
      float4 v = s_red[0][tid];
      for (int q = 1; q < kRedGroups; ++q) {
        const float4 a = s_red[q][tid];
        v.x += a.x;
        v.y += a.y;
        v.z += a.z;
        v.w += a.w;
      }
      if (resid != nullptr) {
        const float4 rv = reinterpret_cast<const float4*>(resid)[o4];
        v.x = rv.x + v.x;
        v.y = rv.y + v.y;
        v.z = rv.z + v.z;
        v.w = rv.w + v.w;
      }
      reinterpret_cast<float4*>(y)[o4] = v;
    }
    return;
  }
  // ---- ascending active list of token b: prefix over the segment counts, then every thread
  // copies list slots tid, tid + 256, ..., 8 in flight. The first slots are requested together
  // with the counts: every slot lies inside the [ntiles, rmax] list buffer, so reading one that
  // its segment did not fill is harmless, and whether it is kept is decided after the prefix.
  __shared__ int s_pref[kListSegs + 1];
  const int b = (blockIdx.x - nred) / kListBlocks, part_k = (blockIdx.x - nred) % kListBlocks;
  const int32_t* src = bidx + (size_t)b * ntiles * rmax;
  const int nslot = ntiles * rmax;
  const int q_lo = (int)(((long long)nslot * part_k) / kListBlocks);
  const int q_hi = (int)(((long long)nslot * (part_k + 1)) / kListBlocks);
  int v[8];
  auto load_slots = [&](int q0) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int q = q0 + 256 * u;
      v[u] = q < q_hi ? src[q] : -1;
    }
  };
  load_slots(q_lo + tid);
  const int per = (ntiles + 255) / 256;
  const int beg = min(tid * per, ntiles), end = min(beg + per, ntiles);
  int local = 0;
  for (int i = beg; i < end; ++i) local += bcnt[b * ntiles + i];
  int total;
  int run = block_exclusive_scan_256(local, s_tmp, &total);
  for (int i = beg; i < end; ++i) {
    s_pref[i] = run;
    run += bcnt[b * ntiles + i];
  }
  if (tid == 0) s_pref[ntiles] = total;
  __syncthreads();
  // flattened (segment, slot) pairs: slot q = i * rmax + j holds entry j of segment i; this
  // block copies the filled slots among [q_lo, q_hi) of token b
  for (int q0 = q_lo + tid; q0 < q_hi; q0 += 8 * 256) {
    if (q0 != q_lo + tid) load_slots(q0);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int q = q0 + 256 * u, i = q / rmax, j = q - i * rmax;
      if (q < q_hi && j < s_pref[i + 1] - s_pref[i]) active_idx[(size_t)b * F + s_pref[i] + j] = v[u];
    }
  }
  if (tid == 0 && part_k == 0) active_cnt[b] = total;
}

int pow2_at_least(int v, int cap) {
  int p = 1;
  while (p < v && p < cap) p <<= 1;
  return p;
}

template <int BM, int MODE>
hipError_t launch_gate_bm(int cpl, dim3 grid, size_t lds, hipStream_t s, const float* x, int B,
                          const uint4* wg, const uint4* wu, int d, int F, float t, float norm_eps,
                          int rmax, int32_t* uidx, float* hbuf, int32_t* ucnt, int32_t* bidx,
                          int32_t* bcnt, float* absact, const unsigned long long* cut) {
#define SIRIUS_GATE(CPLV)                                                                        \
  case CPLV:                                                                                     \
    klaunch(gate_kernel<BM, CPLV, MODE>, grid, 256, lds, s, x, B, wg, wu, d, F, t, norm_eps, rmax,    \
                                                       uidx, hbuf, ucnt, bidx, bcnt, absact,     \
                                                       cut);                                     \
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

template <int MODE>
hipError_t launch_gate_mode(int bm, int cpl, dim3 grid, size_t lds, hipStream_t s, const float* x,
                            int B, const uint4* wg, const uint4* wu, int d, int F, float t,
                            float norm_eps, int rmax, int32_t* uidx, float* hbuf, int32_t* ucnt,
                            int32_t* bidx, int32_t* bcnt, float* absact,
                            const unsigned long long* cut = nullptr) {
  switch (bm) {
    case 1: return launch_gate_bm<1, MODE>(cpl, grid, lds, s, x, B, wg, wu, d, F, t, norm_eps, rmax, uidx, hbuf, ucnt, bidx, bcnt, absact, cut);
    case 2: return launch_gate_bm<2, MODE>(cpl, grid, lds, s, x, B, wg, wu, d, F, t, norm_eps, rmax, uidx, hbuf, ucnt, bidx, bcnt, absact, cut);
    case 4: return launch_gate_bm<4, MODE>(cpl, grid, lds, s, x, B, wg, wu, d, F, t, norm_eps, rmax, uidx, hbuf, ucnt, bidx, bcnt, absact, cut);
    case 8: return launch_gate_bm<8, MODE>(cpl, grid, lds, s, x, B, wg, wu, d, F, t, norm_eps, rmax, uidx, hbuf, ucnt, bidx, bcnt, absact, cut);
    default: return hipErrorInvalidValue;
  }
}

// Gate segments: kGateSegs workgroups (two per CU) when d_ff is large enough, else ~4 rows each.
int gate_segments(int F) { return std::max(1, std::min(kGateSegs, ceil_div(F, 4))); }

}  // namespace

GemvLayout gemv_layout(int B, int d, int F) {
  GemvLayout L{};
  L.bc = std::max(1, std::min(std::min(B, 8), kXLdsFloats / d));
  L.ntiles = gate_segments(F);
  L.rmax = ceil_div(F, L.ntiles);
  L.cs = ceil_div(d / 8, kWave);  // 512-column slices
  L.gr = std::max(1, std::min(kDownBlocks / L.cs, ceil_div(F, 32)));
  const size_t segcap = (size_t)L.ntiles * L.rmax;  // >= F
  Carve c;
  L.uidx = c.take(segcap * 4);
  L.h = c.take(segcap * L.bc * 4);
  L.ucnt = c.take((size_t)L.ntiles * 4);
  L.bidx = c.take((size_t)L.bc * segcap * 4);
  L.bcnt = c.take((size_t)L.bc * L.ntiles * 4);
  L.part = c.take((size_t)L.gr * L.bc * d * 4);
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_gemv(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                           const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                           char* ws, const GemvLayout& L, hipStream_t stream, const float* act,
                           const unsigned long long* cut) {
  if (B < 1 || B > L.bc || L.rmax > kMaxSeg || L.ntiles > kGateSegs) return hipErrorInvalidValue;
  if (mode == kFfnModeTopK && (act == nullptr || cut == nullptr)) return hipErrorInvalidValue;
  const bool topk = mode == kFfnModeTopK;
  const int bm = pow2_at_least(B, 8);
  const int cpl = pow2_at_least(ceil_div(d / 8, kWave), 16);
  int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.uidx);
  float* hbuf = reinterpret_cast<float*>(ws + L.h);
  int32_t* ucnt = reinterpret_cast<int32_t*>(ws + L.ucnt);
  const bool lists = (mode != kFfnModeDense) && active_idx != nullptr;
  int32_t* bidx = lists ? reinterpret_cast<int32_t*>(ws + L.bidx) : nullptr;
  int32_t* bcnt = lists ? reinterpret_cast<int32_t*>(ws + L.bcnt) : nullptr;
  const size_t lds = (size_t)B * d * sizeof(float);
  const uint4* wg4 = reinterpret_cast<const uint4*>(wg);
  const uint4* wu4 = reinterpret_cast<const uint4*>(wu);

  const bool thr = mode == kFfnModeThreshold;
  hipError_t e;
  {
    ProfScope prof(topk ? "topk_up" : (thr ? "cats_gate" : "dense_gate"), stream);
    if (topk)
      e = launch_gate_mode<kModeKeyed>(bm, cpl, dim3(L.ntiles), lds, stream, x, B, wg4, wu4, d, F,
                                       t, norm_eps, L.rmax, uidx, hbuf, ucnt, bidx, bcnt,
                                       const_cast<float*>(act), cut);
    else if (thr)
      e = launch_gate_mode<kModeSparse>(bm, cpl, dim3(L.ntiles), lds, stream, x, B, wg4, wu4, d, F,
                                        t, norm_eps, L.rmax, uidx, hbuf, ucnt, bidx, bcnt, nullptr);
    else
      e = launch_gate_mode<kModeDense>(bm, cpl, dim3(L.ntiles), lds, stream, x, B, wg4, wu4, d, F,
                                       t, norm_eps, L.rmax, uidx, hbuf, ucnt, bidx, bcnt, nullptr);
  }
  if (e != hipSuccess) return e;

  float* part = reinterpret_cast<float*>(ws + L.part);
  {
    ProfScope prof(topk ? "topk_down" : (thr ? "cats_down" : "dense_down"), stream);
    if ((e = launch_down(B, d, L.ntiles, L.rmax, L.gr, wd, uidx, hbuf, B, ucnt, part, stream)) !=
        hipSuccess)
      return e;
  }
  const int n = B * d;
  const int nred = ceil_div(n, 4 * (red_wide(L.gr, n) ? 256 : kRedOut4));  // blocks of the sums
  ProfScope prof(topk ? "topk_reduce" : (thr ? "cats_reduce" : "dense_reduce"), stream);
  klaunch(reduce_kernel, nred + (lists ? B * kListBlocks : 0), 256, 0, stream, 
      part, L.gr, n, resid, y, nred, B, F, L.ntiles, L.rmax, bidx, bcnt, active_idx, active_cnt);
  return hipGetLastError();
}

hipError_t launch_down(int B, int d, int nseg, int rmax, int gr, const uint16_t* wd,
                       const int32_t* uidx, const float* hbuf, int hstride, const int32_t* ucnt,
                       float* part, hipStream_t stream) {
  if (B < 1 || B > 16 || nseg > kMaxSegs) return hipErrorInvalidValue;
  const dim3 dgrid(ceil_div(d / 8, kWave), gr);
  const uint4* wd4 = reinterpret_cast<const uint4*>(wd);
#define SIRIUS_DOWN(BMV)                                                                     \
  case BMV:                                                                                  \
    klaunch(down_kernel<BMV>, dgrid, 256, 0, stream, wd4, d, B, uidx, hbuf, hstride, ucnt, nseg, \
                                                rmax, gr, part);                             \
    break;
  switch (pow2_at_least(B, 16)) {
    SIRIUS_DOWN(1)
    SIRIUS_DOWN(2)
    SIRIUS_DOWN(4)
    SIRIUS_DOWN(8)
    SIRIUS_DOWN(16)
    default:
      return hipErrorInvalidValue;
  }
#undef SIRIUS_DOWN
  return hipGetLastError();
}

hipError_t launch_reduce(const float* part, int gr, int B, int d, const float* resid, float* y,
                         hipStream_t stream, int F, int nseg, int rmax, const int32_t* bidx,
                         const int32_t* bcnt, int32_t* active_idx, int32_t* active_cnt) {
  const int n = B * d;
  const int nred = ceil_div(n, 4 * (red_wide(gr, n) ? 256 : kRedOut4));  // blocks of the sums
  const bool lists = active_idx != nullptr;
  if (lists && nseg > kListSegs) return hipErrorInvalidValue;
  klaunch(reduce_kernel, nred + (lists ? B * kListBlocks : 0), 256, 0, stream, 
      part, gr, n, resid, y, nred, B, F, nseg, rmax, bidx, bcnt, active_idx, active_cnt);
  return hipGetLastError();
}

hipError_t launch_gate_act(const float* x, int N, const uint16_t* wg, int d, int F,
                           float norm_eps, float* act, hipStream_t stream) {
  const int bc = std::max(1, std::min(8, kXLdsFloats / d));
  const int cpl = pow2_at_least(ceil_div(d / 8, kWave), 16);
  const int nseg = gate_segments(F);
  const int rmax = ceil_div(F, nseg);
  if (rmax > kMaxSeg) return hipErrorInvalidValue;
  for (int b0 = 0; b0 < N; b0 += bc) {
    const int nb = std::min(bc, N - b0);
    const int bm = pow2_at_least(nb, 8);
    ProfScope prof("topk_gate", stream);
    hipError_t e = launch_gate_mode<kModeAct>(
        bm, cpl, dim3(nseg), (size_t)nb * d * sizeof(float), stream, x + (size_t)b0 * d, nb,
        reinterpret_cast<const uint4*>(wg), nullptr, d, F, 0.f, norm_eps, rmax, nullptr, nullptr,
        nullptr, nullptr, nullptr, act + (size_t)b0 * F);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gate_absact(const float* x, int N, const uint16_t* wg, int d, int F,
                              float* absact, hipStream_t stream) {
  const int bc = std::max(1, std::min(8, kXLdsFloats / d));
  const int cpl = pow2_at_least(ceil_div(d / 8, kWave), 16);
  const int nseg = gate_segments(F);
  const int rmax = ceil_div(F, nseg);
  if (rmax > kMaxSeg) return hipErrorInvalidValue;
  for (int b0 = 0; b0 < N; b0 += bc) {
    const int nb = std::min(bc, N - b0);
    const int bm = pow2_at_least(nb, 8);
    ProfScope prof("calib_gate", stream);
    hipError_t e = launch_gate_mode<kModeAbsAct>(
        bm, cpl, dim3(nseg), (size_t)nb * d * sizeof(float), stream, x + (size_t)b0 * d, nb,
        reinterpret_cast<const uint4*>(wg), nullptr, d, F, 0.f, -1.f, rmax, nullptr, nullptr,
        nullptr, nullptr, nullptr, absact + (size_t)b0 * F);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sirius
