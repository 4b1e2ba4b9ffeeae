// Attention over the KV cache shared by the sparse and the full model, with the full model's
// direct rewrite (Algorithm 1; Sec. 4, how to correct), on gfx950.
//
// A call carries n tokens per batch entry at positions p .. p + n - 1 (p = cache_pos[b]): their
// keys and values (k_new, v_new) replace the cache rows there, and token i attends causally to
// rows 0 .. p + i. n = 1 is the sparse model's decode step, n = kernel size the full model's
// verification pass over the drafted chunk. Query head h reads key/value head h / G
// (G = H / Hkv); the G x n query rows that share a key/value head are processed together, so
// every key and value row is read once per call.
//
//  attn_partial_kernel  grid (position chunk, key/value head x row group, batch), 256 threads.
//                       The chunk's keys and values are staged 64 rows at a time in LDS as
//                       fp32 (cache rows below p, the new rows from p on; the row-group-0
//                       workgroup also writes the new rows into the cache: each is written by
//                       exactly one workgroup and never read back from the cache in the
//                       call). Scores in fp32 from register blocks (4 rows x 4 positions, or
//                       4 rows x 1 position for up to 16 rows), causal mask, online softmax
//                       (running max and sum per row), P.V into 4 x 4 register blocks; the
//                       chunk's (max, sum, unnormalised output) per row go to the workspace.
//  attn_combine_kernel  one workgroup per query row merges the chunks in order.
//  kv_rollback_kernel   cache_pos[b] += min(accept_len[b] + 1, n).
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

constexpr int kAttnThreads = 256;
constexpr int kTile = 64;                 // positions staged per step
constexpr int kMaxHd = 128;
constexpr int kMaxRowsWg = 64;            // query rows per workgroup
constexpr int kPitch = kMaxHd + 4;        // LDS row pitch (floats): 16-byte rows off the banks
constexpr int kPPitch = kMaxRowsWg + 4;   // score tile pitch: a position's rows off the banks
constexpr int kMaxOB = 2;                 // 4 x 4 output blocks per thread: 64 rows x 128 / 256 / 16

__device__ __forceinline__ void widen8(uint4 w, float* dst) {
  dst[0] = bf16_lo(w.x);
  dst[1] = bf16_hi(w.x);
  dst[2] = bf16_lo(w.y);
  dst[3] = bf16_hi(w.y);
  dst[4] = bf16_lo(w.z);
  dst[5] = bf16_hi(w.z);
  dst[6] = bf16_lo(w.w);
  dst[7] = bf16_hi(w.w);
}

// BIG: up to 64 rows, scores in 4 x 4 blocks; else up to 16 rows, 4 x 1 blocks.
template <bool BIG>
__global__ __launch_bounds__(kAttnThreads) void attn_partial_kernel(
    const float* __restrict__ q, const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    uint4* __restrict__ k_cache, uint4* __restrict__ v_cache, const int32_t* __restrict__ cache_pos,
    int n, int H, int Hkv, int hd, int Lmax, int chunk, int rgroups, int R, float scale,
    float* __restrict__ pm, float* __restrict__ pl, float* __restrict__ po) {
  __shared__ float s_q[kMaxRowsWg * kPitch];
  __shared__ float s_k[kTile * kPitch];
  __shared__ float s_v[kTile * kPitch];
  __shared__ float s_p[kTile * kPPitch];  // scores, then probabilities, [position][row]
  __shared__ float s_m[kMaxRowsWg], s_l[kMaxRowsWg], s_alpha[kMaxRowsWg];
  const int tid = threadIdx.x;
  const int split = blockIdx.x, nsplit = gridDim.x;
  const int kvh = blockIdx.y / rgroups, rg = blockIdx.y % rgroups, b = blockIdx.z;
  const int G = H / Hkv;
  const int p = cache_pos[b];
  const bool valid = p >= 0 && p + n <= Lmax;
  const int L = p + n;
  const int c0 = split * chunk, c1 = min(c0 + chunk, L);
  const int r0 = rg * kMaxRowsWg, nr = min(kMaxRowsWg, R - r0);
  const int nr4 = (nr + 3) & ~3;
  const int hd4 = hd >> 2, hd8 = hd >> 3;
  const size_t rowbase = ((size_t)b * Hkv + kvh) * R + r0;  // partial row index of row r0

  if (!valid || c0 >= L) {  // nothing visible in this chunk (or a position outside the cache)
    if (tid < nr) {
      pm[(rowbase + tid) * nsplit + split] = -INFINITY;
      pl[(rowbase + tid) * nsplit + split] = 0.f;
    }
    return;
  }
  // the direct rewrite: the new rows of this chunk go into the cache
  if (rg == 0) {
    const int w0 = max(c0, p);
    for (int e = tid; e < (c1 - w0) * hd8; e += kAttnThreads) {
      const int j = e / hd8, c = e - j * hd8, pos = w0 + j;
      const size_t src = (((size_t)b * n + (pos - p)) * Hkv + kvh) * hd8 + c;
      const size_t dst = (((size_t)b * Lmax + pos) * Hkv + kvh) * hd8 + c;
      k_cache[dst] = k_new[src];
      v_cache[dst] = v_new[src];
    }
  }
  // query rows (row r = token i * G + head g), scaled; padding rows are zero
  for (int e = tid; e < nr4 * hd4; e += kAttnThreads) {
    const int r = e / hd4, d4 = e - r * hd4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < nr) {
      const int rr = r0 + r, i = rr / G, h = kvh * G + (rr - i * G);
      v = reinterpret_cast<const float4*>(q + (((size_t)b * n + i) * H + h) * hd)[d4];
      v.x *= scale;
      v.y *= scale;
      v.z *= scale;
      v.w *= scale;
    }
    *reinterpret_cast<float4*>(&s_q[r * kPitch + 4 * d4]) = v;
  }
  if (tid < nr) {
    s_m[tid] = -INFINITY;
    s_l[tid] = 0.f;
  }
  // output blocks: block ob = rows 4 (ob / hd4) .. + 4, columns 4 (ob % hd4) .. + 4
  const int nob = (nr4 >> 2) * hd4;
  float4 acc[kMaxOB][4];
#pragma unroll
  for (int u = 0; u < kMaxOB; ++u)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) acc[u][rr] = make_float4(0.f, 0.f, 0.f, 0.f);

  for (int t0 = c0; t0 < c1; t0 += kTile) {
    const int tn = min(kTile, c1 - t0);
    __syncthreads();  // the previous step's readers are done with s_k, s_v, s_p
    // ---- stage keys and values (fp32): cache rows below p, new rows from p on; zero past tn
    for (int e = tid; e < kTile * hd8; e += kAttnThreads) {
      const int j = e / hd8, c = e - j * hd8, pos = t0 + j;
      uint4 kw = make_uint4(0u, 0u, 0u, 0u), vw = make_uint4(0u, 0u, 0u, 0u);
      if (j < tn) {
        if (pos < p) {
          const size_t i = (((size_t)b * Lmax + pos) * Hkv + kvh) * hd8 + c;
          kw = k_cache[i];
          vw = v_cache[i];
        } else {
          const size_t i = (((size_t)b * n + (pos - p)) * Hkv + kvh) * hd8 + c;
          kw = k_new[i];
          vw = v_new[i];
        }
      }
      widen8(kw, &s_k[j * kPitch + 8 * c]);
      widen8(vw, &s_v[j * kPitch + 8 * c]);
    }
    __syncthreads();
    // ---- scores with the causal mask, into s_p[position][row]
    {
      constexpr int CB = BIG ? 4 : 1;
      const int ncb = kTile / CB;  // positions cb, cb + ncb, ... (neighbouring lanes, rows)
      const int rb = tid / ncb, cb = tid - rb * ncb;
      if (4 * rb < nr4) {
        float s[4][CB];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
#pragma unroll
          for (int cc = 0; cc < CB; ++cc) s[rr][cc] = 0.f;
        for (int d4 = 0; d4 < hd4; ++d4) {
          float4 qv[4], kv[CB];
#pragma unroll
          for (int rr = 0; rr < 4; ++rr)
            qv[rr] = *reinterpret_cast<const float4*>(&s_q[(4 * rb + rr) * kPitch + 4 * d4]);
#pragma unroll
          for (int cc = 0; cc < CB; ++cc)
            kv[cc] = *reinterpret_cast<const float4*>(&s_k[(cb + ncb * cc) * kPitch + 4 * d4]);
#pragma unroll
          for (int rr = 0; rr < 4; ++rr)
#pragma unroll
            for (int cc = 0; cc < CB; ++cc) {
              s[rr][cc] = fmaf(qv[rr].x, kv[cc].x, s[rr][cc]);
              s[rr][cc] = fmaf(qv[rr].y, kv[cc].y, s[rr][cc]);
              s[rr][cc] = fmaf(qv[rr].z, kv[cc].z, s[rr][cc]);
              s[rr][cc] = fmaf(qv[rr].w, kv[cc].w, s[rr][cc]);
            }
        }
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int r = 4 * rb + rr;
          const int lim = p + (r0 + r) / G;  // last visible position of row r
#pragma unroll
          for (int cc = 0; cc < CB; ++cc) {
            const int j = cb + ncb * cc;
            // padding rows get 0 (they never enter the softmax); hidden positions -inf
            s_p[j * kPPitch + r] = (r >= nr) ? 0.f : ((j < tn && t0 + j <= lim) ? s[rr][cc] : -INFINITY);
          }
        }
      }
    }
    __syncthreads();
    // ---- online softmax: four lanes per row, 16 positions each
    {
      const int r = tid >> 2, part = tid & 3;
      float mx = -INFINITY;
      if (r < nr) {
#pragma unroll
        for (int jj = 0; jj < kTile / 4; ++jj) mx = fmaxf(mx, s_p[(part * (kTile / 4) + jj) * kPPitch + r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 1, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 2, kWave));
      float m_old = -INFINITY, m_new = -INFINITY;
      if (r < nr) {
        m_old = s_m[r];
        m_new = fmaxf(m_old, mx);
      }
      float sum = 0.f;
      if (r < nr) {
#pragma unroll
        for (int jj = 0; jj < kTile / 4; ++jj) {
          float* sp = &s_p[(part * (kTile / 4) + jj) * kPPitch + r];
          const float e = (*sp > -INFINITY) ? expf(*sp - m_new) : 0.f;
          *sp = e;
          sum += e;
        }
      }
      sum += __shfl_xor(sum, 1, kWave);
      sum += __shfl_xor(sum, 2, kWave);
      if (r < nr && part == 0) {
        const float alpha = (m_old > -INFINITY) ? expf(m_old - m_new) : 0.f;
        s_alpha[r] = alpha;
        s_m[r] = m_new;
        s_l[r] = s_l[r] * alpha + sum;
      }
    }
    __syncthreads();
    // ---- O = alpha O + P V over 4 x 4 output blocks
#pragma unroll
    for (int u = 0; u < kMaxOB; ++u) {
      const int ob = tid + u * kAttnThreads;
      if (ob < nob) {
        const int rb = ob / hd4, d4 = ob - rb * hd4;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int r = 4 * rb + rr;
          const float al = (r < nr) ? s_alpha[r] : 0.f;
          acc[u][rr].x *= al;
          acc[u][rr].y *= al;
          acc[u][rr].z *= al;
          acc[u][rr].w *= al;
        }
        for (int j = 0; j < tn; ++j) {
          const float4 pv = *reinterpret_cast<const float4*>(&s_p[j * kPPitch + 4 * rb]);
          const float4 vv = *reinterpret_cast<const float4*>(&s_v[j * kPitch + 4 * d4]);
          const float pr[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            acc[u][rr].x = fmaf(pr[rr], vv.x, acc[u][rr].x);
            acc[u][rr].y = fmaf(pr[rr], vv.y, acc[u][rr].y);
            acc[u][rr].z = fmaf(pr[rr], vv.z, acc[u][rr].z);
            acc[u][rr].w = fmaf(pr[rr], vv.w, acc[u][rr].w);
          }
        }
      }
    }
  }
  // ---- this chunk's partial: max, sum and the unnormalised output per row
  if (tid < nr) {
    pm[(rowbase + tid) * nsplit + split] = s_m[tid];
    pl[(rowbase + tid) * nsplit + split] = s_l[tid];
  }
#pragma unroll
  for (int u = 0; u < kMaxOB; ++u) {
    const int ob = tid + u * kAttnThreads;
    if (ob < nob) {
      const int rb = ob / hd4, d4 = ob - rb * hd4;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int r = 4 * rb + rr;
        if (r < nr)
          reinterpret_cast<float4*>(po + ((rowbase + r) * nsplit + split) * hd)[d4] = acc[u][rr];
      }
    }
  }
}

// One workgroup (hd threads) per query row: the chunks merged in order.
__global__ __launch_bounds__(kMaxHd) void attn_combine_kernel(
    int n, int H, int Hkv, int hd, int R, int nsplit, const float* __restrict__ pm,
    const float* __restrict__ pl, const float* __restrict__ po, float* __restrict__ out) {
  const int row = blockIdx.x;  // (b, kvh, r)
  const int r = row % R, bk = row / R, kvh = bk % Hkv, b = bk / Hkv;
  const int G = H / Hkv, i = r / G, h = kvh * G + (r - i * G);
  const int d = threadIdx.x;
  const float* m = pm + (size_t)row * nsplit;
  const float* l = pl + (size_t)row * nsplit;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, m[s]);
  float den = 0.f, num = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    if (m[s] > -INFINITY) {
      const float w = expf(m[s] - M);
      den = fmaf(l[s], w, den);
      if (d < hd) num = fmaf(po[((size_t)row * nsplit + s) * hd + d], w, num);
    }
  }
  if (d < hd) out[(((size_t)b * n + i) * H + h) * hd + d] = num / den;
}

__global__ void kv_rollback_kernel(int32_t* __restrict__ cache_pos,
                                   const int32_t* __restrict__ accept_len, int B, int n) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    const int a = accept_len[b];
    cache_pos[b] += min(max(a, 0) + 1, n);
  }
}

}  // namespace

AttnLayout attn_layout(int B, int n, int H, int Hkv, int hd, int Lmax) {
  AttnLayout L{};
  const int R = (H / Hkv) * n;
  L.rgroups = ceil_div(R, kMaxRowsWg);
  L.chunk = kTile * std::max(1, ceil_div(ceil_div(Lmax, kTile), 256));  // 256 chunks at most
  L.nsplit = ceil_div(Lmax, L.chunk);
  const size_t rows = (size_t)B * Hkv * R;
  Carve c;
  L.pm = c.take(rows * L.nsplit * sizeof(float));
  L.pl = c.take(rows * L.nsplit * sizeof(float));
  L.po = c.take(rows * L.nsplit * hd * sizeof(float));
  L.total = c.off;
  return L;
}

hipError_t launch_attn_kv(const float* q, const uint16_t* k_new, const uint16_t* v_new,
                          uint16_t* k_cache, uint16_t* v_cache, const int32_t* cache_pos, int B,
                          int n, int H, int Hkv, int hd, int Lmax, float* out, char* ws,
                          const AttnLayout& L, hipStream_t stream) {
  if (hd > kMaxHd || (hd & 7) != 0 || H % Hkv != 0) return hipErrorInvalidValue;
  const int R = (H / Hkv) * n;
  float* pm = reinterpret_cast<float*>(ws + L.pm);
  float* pl = reinterpret_cast<float*>(ws + L.pl);
  float* po = reinterpret_cast<float*>(ws + L.po);
  const float scale = (float)(1.0 / sqrt((double)hd));
  const dim3 grid(L.nsplit, Hkv * L.rgroups, B);
  {
    ProfScope prof("attn_partial", stream);
    if (std::min(R, kMaxRowsWg) > 16)
      attn_partial_kernel<true><<<grid, kAttnThreads, 0, stream>>>(
          q, reinterpret_cast<const uint4*>(k_new), reinterpret_cast<const uint4*>(v_new),
          reinterpret_cast<uint4*>(k_cache), reinterpret_cast<uint4*>(v_cache), cache_pos, n, H,
          Hkv, hd, Lmax, L.chunk, L.rgroups, R, scale, pm, pl, po);
    else
      attn_partial_kernel<false><<<grid, kAttnThreads, 0, stream>>>(
          q, reinterpret_cast<const uint4*>(k_new), reinterpret_cast<const uint4*>(v_new),
          reinterpret_cast<uint4*>(k_cache), reinterpret_cast<uint4*>(v_cache), cache_pos, n, H,
          Hkv, hd, Lmax, L.chunk, L.rgroups, R, scale, pm, pl, po);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ProfScope prof("attn_combine", stream);
  attn_combine_kernel<<<B * Hkv * R, kMaxHd, 0, stream>>>(n, H, Hkv, hd, R, L.nsplit, pm, pl, po,
                                                          out);
  return hipGetLastError();
}

hipError_t launch_kv_rollback(int32_t* cache_pos, const int32_t* accept_len, int B, int n,
                              hipStream_t stream) {
  ProfScope prof("kv_rollback", stream);
  kv_rollback_kernel<<<ceil_div(B, 256), 256, 0, stream>>>(cache_pos, accept_len, B, n);
  return hipGetLastError();
}

}  // namespace sirius
