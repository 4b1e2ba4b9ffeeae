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
//                       bf16, every load of a tile issued before the first is stored (cache
//                       rows below p, the new rows from p on; the row-group-0 workgroup also
//                       writes the new rows into the cache: each is written by exactly one
//                       workgroup and never read back from the cache in the call). Scores in
//                       fp32: with more than 16 query rows from 4 rows x 4 positions register
//                       blocks, else each score's dot product split over four lanes; causal
//                       mask, online softmax (running max and sum per row), P.V into 4 x 4
//                       register blocks (with few rows, the tile's positions split over groups
//                       of threads whose shares are summed in a fixed order); the chunk's
//                       (max, sum, unnormalised output) per row go to the workspace. The score
//                       tile reuses the key buffer once the scores are formed. A cache of at
//                       most 256 rows is one chunk per workgroup (its tiles in turn), and the
//                       kernel writes the normalised output itself: no merge launch.
//  attn_combine_kernel  one workgroup per query row: the chunks' (max, sum) and their first
//                       outputs (all of them, up to 64 chunks) requested together, the
//                       weights exp(m_c - M) (one chunk per thread), then each thread sums
//                       its output column over the chunks in order.
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
constexpr int kKVPitch8 = kMaxHd / 8 + 1; // bf16 key/value rows in 16-byte units (+1 off the banks)
constexpr int kMaxOB = 2;                 // 4 x 4 output blocks per thread: 64 rows x 128 / 256 / 16
constexpr int kStagePer = kTile * kMaxHd / 8 / kAttnThreads;  // 16-byte loads per thread and tile
constexpr int kMaxSplits = 256;           // position chunks per call at most
constexpr int kDirectMax = 256;           // caches up to this many rows: one chunk, no combine
constexpr int kOneBatchMax = 64;          // merges of at most this many chunks: one load batch

// BIG: up to 64 rows, scores in 4 x 4 register blocks; else up to 16 rows, each score's dot
// product split over four lanes. Keys and values are staged as bf16; the score tile reuses
// the key buffer once the scores are formed (69 KB of LDS: two workgroups per CU).
template <bool BIG>
__global__ __launch_bounds__(kAttnThreads) void attn_partial_kernel(
    const float* __restrict__ q, const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    uint4* __restrict__ k_cache, uint4* __restrict__ v_cache, const int32_t* __restrict__ cache_pos,
    int n, int H, int Hkv, int hd, int Lmax, int chunk, int rgroups, int R, float scale,
    float* __restrict__ pm, float* __restrict__ pl, float* __restrict__ po,
    float* __restrict__ out) {
  constexpr int kRows = BIG ? kMaxRowsWg : 16;
  __shared__ float s_q[kRows * kPitch];
  __shared__ uint4 s_kp[kTile * kKVPitch8];  // keys (bf16), then the score tile [position][row]
  __shared__ uint4 s_v[kTile * kKVPitch8];   // values (bf16)
  __shared__ float s_m[kRows], s_l[kRows], s_alpha[kRows];
  float* s_p = reinterpret_cast<float*>(s_kp);
  const uint16_t* s_v16 = reinterpret_cast<const uint16_t*>(s_v);
  const int tid = threadIdx.x;
  const int split = blockIdx.x, nsplit = gridDim.x;
  const int kvh = blockIdx.y / rgroups, rg = blockIdx.y % rgroups, b = blockIdx.z;
  const int G = H / Hkv;
  const int p = cache_pos[b];
  const bool valid = p >= 0 && p + n <= Lmax;
  const int L = p + n;
  const int c0 = split * chunk, c1 = min(c0 + chunk, L);
  const int r0 = rg * kMaxRowsWg, nr = min(kRows, R - r0);
  const int nr4 = (nr + 3) & ~3;
  const int hd4 = hd >> 2, hd8 = hd >> 3;
  const size_t rowbase = ((size_t)b * Hkv + kvh) * R + r0;  // partial row index of row r0
  // one chunk per row (out != nullptr): the output itself, out[b][i][h][:] for row r0 + r
  auto out_row = [&](int r) {
    const int rr = r0 + r, i = rr / G, h = kvh * G + (rr - i * G);
    return out + (((size_t)b * n + i) * H + h) * hd;
  };

  if (!valid || c0 >= L) {  // nothing visible in this chunk (or a position outside the cache)
    if (out != nullptr) {  // what the merge of empty chunks gives: 0 / 0
      for (int e = tid; e < nr * hd; e += kAttnThreads) out_row(e / hd)[e % hd] = __builtin_nanf("");
      return;
    }
    if (tid < nr) {
      pm[(rowbase + tid) * nsplit + split] = -INFINITY;
      pl[(rowbase + tid) * nsplit + split] = 0.f;
    }
    return;
  }
  // the direct rewrite: the new rows of this chunk go into the cache; the thread's first new-row
  // chunk and its first query chunk are requested together, so the two take one round trip
  const int w0 = max(c0, p);
  const int ncw = rg == 0 ? (c1 - w0) * hd8 : 0;  // 16-byte chunks of new rows to write
  {
    uint4 kw0 = make_uint4(0u, 0u, 0u, 0u), vw0 = kw0;
    size_t dst0 = 0;
    if (tid < ncw) {
      const int j = tid / hd8, c = tid - j * hd8, pos = w0 + j;
      const size_t src = (((size_t)b * n + (pos - p)) * Hkv + kvh) * hd8 + c;
      dst0 = (((size_t)b * Lmax + pos) * Hkv + kvh) * hd8 + c;
      kw0 = k_new[src];
      vw0 = v_new[src];
    }
    float4 qv = make_float4(0.f, 0.f, 0.f, 0.f);
    const int qr = tid / hd4, qd4 = tid - qr * hd4;
    if (tid < nr4 * hd4 && qr < nr) {
      const int rr = r0 + qr, i = rr / G, h = kvh * G + (rr - i * G);
      qv = reinterpret_cast<const float4*>(q + (((size_t)b * n + i) * H + h) * hd)[qd4];
    }
    if (tid < ncw) {
      k_cache[dst0] = kw0;
      v_cache[dst0] = vw0;
    }
    if (tid < nr4 * hd4)
      *reinterpret_cast<float4*>(&s_q[qr * kPitch + 4 * qd4]) =
          make_float4(qv.x * scale, qv.y * scale, qv.z * scale, qv.w * scale);
  }
  if (rg == 0) {
    for (int e = tid + kAttnThreads; e < ncw; e += kAttnThreads) {
      const int j = e / hd8, c = e - j * hd8, pos = w0 + j;
      const size_t src = (((size_t)b * n + (pos - p)) * Hkv + kvh) * hd8 + c;
      const size_t dst = (((size_t)b * Lmax + pos) * Hkv + kvh) * hd8 + c;
      k_cache[dst] = k_new[src];
      v_cache[dst] = v_new[src];
    }
  }
  // query rows (row r = token i * G + head g), scaled; padding rows are zero
  for (int e = tid + kAttnThreads; e < nr4 * hd4; e += kAttnThreads) {
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
  // output blocks of 4 rows x 4 columns; with few blocks the positions of a tile are split
  // over jg groups of threads, each accumulating its own share (summed once at the end)
  const int nob = (nr4 >> 2) * hd4;
  const int jg = BIG ? 1 : max(1, min(8, kAttnThreads / nob));
  const int jgrp = tid / nob, job = tid - jgrp * nob;  // group, block (non-BIG)
  float4 acc[kMaxOB][4];
#pragma unroll
  for (int u = 0; u < kMaxOB; ++u)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) acc[u][rr] = make_float4(0.f, 0.f, 0.f, 0.f);

  for (int t0 = c0; t0 < c1; t0 += kTile) {
    const int tn = min(kTile, c1 - t0);
    __syncthreads();  // the previous step's readers are done with s_kp, s_v
    // ---- stage keys and values (bf16): cache rows below p, new rows from p on; zero past tn.
    // Every load of the tile is issued before the first is stored.
    {
      uint4 kw[kStagePer], vw[kStagePer];
#pragma unroll
      for (int u = 0; u < kStagePer; ++u) {
        const int e = tid + u * kAttnThreads;
        const int j = e / hd8, c = e - j * hd8, pos = t0 + j;
        kw[u] = make_uint4(0u, 0u, 0u, 0u);
        vw[u] = make_uint4(0u, 0u, 0u, 0u);
        if (j < tn) {
          const size_t i = (pos < p) ? (((size_t)b * Lmax + pos) * Hkv + kvh) * hd8 + c
                                     : (((size_t)b * n + (pos - p)) * Hkv + kvh) * hd8 + c;
          kw[u] = ((pos < p) ? k_cache : k_new)[i];
          vw[u] = ((pos < p) ? v_cache : v_new)[i];
        }
      }
#pragma unroll
      for (int u = 0; u < kStagePer; ++u) {
        const int e = tid + u * kAttnThreads;
        const int j = e / hd8, c = e - j * hd8;
        if (j < kTile) {
          s_kp[j * kKVPitch8 + c] = kw[u];
          s_v[j * kKVPitch8 + c] = vw[u];
        }
      }
    }
    __syncthreads();
    // ---- scores with the causal mask (held in registers until the keys are no longer read)
    constexpr int CB = BIG ? 4 : 1;
    float sc[4][CB];   // BIG: rows 4 rb.., positions cb + 16 cc; else rows of row block rbs
    float scs[4][4];   // non-BIG: four row blocks x four rows, one position
    if (BIG) {
      const int rb = tid >> 4, cb = tid & 15;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
#pragma unroll
        for (int cc = 0; cc < CB; ++cc) sc[rr][cc] = 0.f;
      if (4 * rb < nr4) {
        for (int d8 = 0; d8 < hd8; ++d8) {
          float kf[CB][8];
#pragma unroll
          for (int cc = 0; cc < CB; ++cc) {
            const uint4 w = s_kp[(cb + 16 * cc) * kKVPitch8 + d8];
            kf[cc][0] = bf16_lo(w.x); kf[cc][1] = bf16_hi(w.x); kf[cc][2] = bf16_lo(w.y);
            kf[cc][3] = bf16_hi(w.y); kf[cc][4] = bf16_lo(w.z); kf[cc][5] = bf16_hi(w.z);
            kf[cc][6] = bf16_lo(w.w); kf[cc][7] = bf16_hi(w.w);
          }
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const float4 qa = *reinterpret_cast<const float4*>(&s_q[(4 * rb + rr) * kPitch + 8 * d8]);
            const float4 qb = *reinterpret_cast<const float4*>(&s_q[(4 * rb + rr) * kPitch + 8 * d8 + 4]);
#pragma unroll
            for (int cc = 0; cc < CB; ++cc) {
              float a = sc[rr][cc];
              a = fmaf(qa.x, kf[cc][0], a); a = fmaf(qa.y, kf[cc][1], a);
              a = fmaf(qa.z, kf[cc][2], a); a = fmaf(qa.w, kf[cc][3], a);
              a = fmaf(qb.x, kf[cc][4], a); a = fmaf(qb.y, kf[cc][5], a);
              a = fmaf(qb.z, kf[cc][6], a); a = fmaf(qb.w, kf[cc][7], a);
              sc[rr][cc] = a;
            }
          }
        }
      }
    } else {
      // position j = tid / 4; lane quarter dq takes head-dim chunks dq, dq + 4, ...
      const int j = tid >> 2, dq = tid & 3;
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) scs[rb][rr] = 0.f;
      for (int d8 = dq; d8 < hd8; d8 += 4) {
        const uint4 w = s_kp[j * kKVPitch8 + d8];
        const float kf[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                             bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          if (4 * rb < nr4) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
              const float4 qa = *reinterpret_cast<const float4*>(&s_q[(4 * rb + rr) * kPitch + 8 * d8]);
              const float4 qb = *reinterpret_cast<const float4*>(&s_q[(4 * rb + rr) * kPitch + 8 * d8 + 4]);
              float a = scs[rb][rr];
              a = fmaf(qa.x, kf[0], a); a = fmaf(qa.y, kf[1], a);
              a = fmaf(qa.z, kf[2], a); a = fmaf(qa.w, kf[3], a);
              a = fmaf(qb.x, kf[4], a); a = fmaf(qb.y, kf[5], a);
              a = fmaf(qb.z, kf[6], a); a = fmaf(qb.w, kf[7], a);
              scs[rb][rr] = a;
            }
          }
        }
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          scs[rb][rr] += __shfl_xor(scs[rb][rr], 1, kWave);
          scs[rb][rr] += __shfl_xor(scs[rb][rr], 2, kWave);
        }
    }
    __syncthreads();  // keys read: the score tile takes their place
    if (BIG) {
      const int rb = tid >> 4, cb = tid & 15;
      if (4 * rb < nr4) {
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int r = 4 * rb + rr;
          const int lim = p + (r0 + r) / G;  // last visible position of row r
#pragma unroll
          for (int cc = 0; cc < CB; ++cc) {
            const int j = cb + 16 * cc;
            // padding rows get 0 (they never enter the softmax); hidden positions -inf
            s_p[j * kPPitch + r] = (r >= nr) ? 0.f : ((j < tn && t0 + j <= lim) ? sc[rr][cc] : -INFINITY);
          }
        }
      }
    } else if ((tid & 3) == 0) {
      const int j = tid >> 2;
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if (4 * rb < nr4) {
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int r = 4 * rb + rr;
            const int lim = p + (r0 + r) / G;
            s_p[j * kPPitch + r] = (r >= nr) ? 0.f : ((j < tn && t0 + j <= lim) ? scs[rb][rr] : -INFINITY);
          }
        }
      }
    }
    __syncthreads();
    // ---- online softmax: LPR lanes per row (4 for up to 64 rows, 16 for up to 16), the tile's
    // positions split evenly over them
    {
      constexpr int LPR = BIG ? 4 : 16, PPL = kTile / LPR;
      const int r = tid / LPR, part = tid % LPR;
      float mx = -INFINITY;
      if (r < nr) {
#pragma unroll
        for (int jj = 0; jj < PPL; ++jj) mx = fmaxf(mx, s_p[(part * PPL + jj) * kPPitch + r]);
      }
#pragma unroll
      for (int m = 1; m < LPR; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, kWave));
      float m_old = -INFINITY, m_new = -INFINITY;
      if (r < nr) {
        m_old = s_m[r];
        m_new = fmaxf(m_old, mx);
      }
      float sum = 0.f;
      if (r < nr) {
#pragma unroll
        for (int jj = 0; jj < PPL; ++jj) {
          float* sp = &s_p[(part * PPL + jj) * kPPitch + r];
          const float e = (*sp > -INFINITY) ? expf(*sp - m_new) : 0.f;
          *sp = e;
          sum += e;
        }
      }
#pragma unroll
      for (int m = 1; m < LPR; m <<= 1) sum += __shfl_xor(sum, m, kWave);
      if (r < nr && part == 0) {
        const float alpha = (m_old > -INFINITY) ? expf(m_old - m_new) : 0.f;
        s_alpha[r] = alpha;
        s_m[r] = m_new;
        s_l[r] = s_l[r] * alpha + sum;
      }
    }
    __syncthreads();
    // ---- O = alpha O + P V over 4 x 4 output blocks (a thread group's share of positions)
#pragma unroll
    for (int u = 0; u < kMaxOB; ++u) {
      const int ob = BIG ? tid + u * kAttnThreads : job;
      const bool mine = BIG ? (ob < nob) : (u == 0 && jgrp < jg);
      if (mine) {
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
        const int span = kTile / jg, j0 = (BIG ? 0 : jgrp) * span, j1 = min(j0 + span, tn);
#pragma unroll 4
        for (int j = j0; j < j1; ++j) {
          const float4 pv = *reinterpret_cast<const float4*>(&s_p[j * kPPitch + 4 * rb]);
          const uint2 vw = *reinterpret_cast<const uint2*>(&s_v16[j * kKVPitch8 * 8 + 4 * d4]);
          const float vv[4] = {bf16_lo(vw.x), bf16_hi(vw.x), bf16_lo(vw.y), bf16_hi(vw.y)};
          const float pr[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            acc[u][rr].x = fmaf(pr[rr], vv[0], acc[u][rr].x);
            acc[u][rr].y = fmaf(pr[rr], vv[1], acc[u][rr].y);
            acc[u][rr].z = fmaf(pr[rr], vv[2], acc[u][rr].z);
            acc[u][rr].w = fmaf(pr[rr], vv[3], acc[u][rr].w);
          }
        }
      }
    }
  }
  // ---- this chunk's partial: max, sum and the unnormalised output per row (with one chunk,
  // the output itself: the unnormalised output over the sum, as the merge computes it)
  __syncthreads();
  if (tid < nr && out == nullptr) {
    pm[(rowbase + tid) * nsplit + split] = s_m[tid];
    pl[(rowbase + tid) * nsplit + split] = s_l[tid];
  }
  if (BIG) {
#pragma unroll
    for (int u = 0; u < kMaxOB; ++u) {
      const int ob = tid + u * kAttnThreads;
      if (ob < nob) {
        const int rb = ob / hd4, d4 = ob - rb * hd4;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int r = 4 * rb + rr;
          if (r < nr && out != nullptr) {
            const float l = s_l[r];
            const float4 a = acc[u][rr];
            reinterpret_cast<float4*>(out_row(r))[d4] = make_float4(a.x / l, a.y / l, a.z / l, a.w / l);
          } else if (r < nr) {
            reinterpret_cast<float4*>(po + ((rowbase + r) * nsplit + split) * hd)[d4] = acc[u][rr];
          }
        }
      }
    }
  } else {
    // sum the position groups' shares in order through LDS (the value buffer is free)
    float4* s_red = reinterpret_cast<float4*>(s_v);  // [group][block][4 rows]: <= 8 x 64 x 4
    if (jgrp < jg) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) s_red[(jgrp * nob + job) * 4 + rr] = acc[0][rr];
    }
    __syncthreads();
    if (tid < nob) {
      const int rb = tid / hd4, d4 = tid - rb * hd4;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        float4 t = s_red[tid * 4 + rr];
#pragma unroll 4
        for (int g2 = 1; g2 < jg; ++g2) {
          const float4 o = s_red[(g2 * nob + tid) * 4 + rr];
          t.x += o.x;
          t.y += o.y;
          t.z += o.z;
          t.w += o.w;
        }
        const int r = 4 * rb + rr;
        if (r < nr && out != nullptr) {
          const float l = s_l[r];
          reinterpret_cast<float4*>(out_row(r))[d4] = make_float4(t.x / l, t.y / l, t.z / l, t.w / l);
        } else if (r < nr) {
          reinterpret_cast<float4*>(po + ((rowbase + r) * nsplit + split) * hd)[d4] = t;
        }
      }
    }
  }
}

// One workgroup (hd threads) per query row. Every thread requests its chunks' (max, sum) and
// the first batch of chunk outputs of its column together, so the row costs about one
// memory round trip; the maximum over the chunks, the weights exp(m_c - M) (one chunk per
// thread, LDS) and the denominator follow, then each thread sums its output column over the
// chunks in order, the next batch requested before the current one is added. Chunks with no
// visible position never write their outputs: those are read but replaced by 0 (a select, so
// whatever the buffer holds there cannot reach the sum). NB chunk outputs are requested per
// batch: 8 when there are at most 8 chunks (the small decoder's), where unrolled guards for
// more would cost more than they save; all of them, in one batch and one memory round trip,
// up to 64 chunks (a 4096-row cache); else 32 per batch.
template <int NB>
__device__ __forceinline__ void combine_row(int n, int H, int Hkv, int hd, int R, int nsplit,
                                            const float* __restrict__ pm,
                                            const float* __restrict__ pl,
                                            const float* __restrict__ po, float* __restrict__ out,
                                            float* s_w, float* s_red) {
  const int row = blockIdx.x;  // (b, kvh, r)
  const int r = row % R, bk = row / R, kvh = bk % Hkv, b = bk / Hkv;
  const int G = H / Hkv, i = r / G, h = kvh * G + (r - i * G);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const float* m = pm + (size_t)row * nsplit;
  const float* l = pl + (size_t)row * nsplit;
  const float* o = po + (size_t)row * nsplit * hd + (tid < hd ? tid : 0);
  constexpr bool kOneBatch = NB == kOneBatchMax;  // every chunk's output in the first batch
  constexpr int kPer = kMaxSplits / kMaxHd;  // chunks per thread for the max and the weights
  static_assert(kMaxSplits % kMaxHd == 0, "whole chunks per thread");
  float mv[kPer], lv[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int sp = tid + u * kMaxHd;
    mv[u] = sp < nsplit ? m[sp] : -INFINITY;
    lv[u] = sp < nsplit ? l[sp] : 0.f;
  }
  float ov[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) ov[u] = u < nsplit ? o[(size_t)u * hd] : 0.f;

  float mx = -INFINITY;
#pragma unroll
  for (int u = 0; u < kPer; ++u) mx = fmaxf(mx, mv[u]);
  for (int k = 1; k < kWave; k <<= 1) mx = fmaxf(mx, __shfl_xor(mx, k, kWave));
  if (lane == 0) s_red[wave] = mx;
  __syncthreads();
  float M = s_red[0];
  for (int w = 1; w < kMaxHd / kWave; ++w) M = fmaxf(M, s_red[w]);
  __syncthreads();
  float den = 0.f;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int sp = tid + u * kMaxHd;
    if (sp < nsplit) {
      const float w = (mv[u] > -INFINITY) ? expf(mv[u] - M) : 0.f;
      s_w[sp] = w;
      den = fmaf(lv[u], w, den);
    }
  }
  for (int k = 1; k < kWave; k <<= 1) den += __shfl_xor(den, k, kWave);
  if (lane == 0) s_red[wave] = den;
  __syncthreads();
  den = 0.f;
  for (int w = 0; w < kMaxHd / kWave; ++w) den += s_red[w];
  float num = 0.f;
  for (int s0 = 0; s0 < nsplit; s0 += NB) {
    float nx[NB];
    const int s1 = s0 + NB;
    if constexpr (!kOneBatch) {
#pragma unroll
      for (int u = 0; u < NB; ++u) nx[u] = s1 + u < nsplit ? o[(size_t)(s1 + u) * hd] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      if (s0 + u < nsplit) {
        const float w = s_w[s0 + u];
        num = fmaf(w > 0.f ? ov[u] : 0.f, w, num);
      }
    }
    if constexpr (!kOneBatch) {
#pragma unroll
      for (int u = 0; u < NB; ++u) ov[u] = nx[u];
    }
  }
  if (tid < hd) out[(((size_t)b * n + i) * H + h) * hd + tid] = num / den;
}

__global__ __launch_bounds__(kMaxHd) void attn_combine_kernel(
    int n, int H, int Hkv, int hd, int R, int nsplit, const float* __restrict__ pm,
    const float* __restrict__ pl, const float* __restrict__ po, float* __restrict__ out) {
  __shared__ float s_w[kMaxSplits], s_red[kMaxHd / kWave];
  if (nsplit <= 8)
    combine_row<8>(n, H, Hkv, hd, R, nsplit, pm, pl, po, out, s_w, s_red);
  else if (nsplit <= kOneBatchMax)
    combine_row<kOneBatchMax>(n, H, Hkv, hd, R, nsplit, pm, pl, po, out, s_w, s_red);
  else
    combine_row<32>(n, H, Hkv, hd, R, nsplit, pm, pl, po, out, s_w, s_red);
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
  L.chunk = Lmax <= kDirectMax ? ceil_div(Lmax, kTile) * kTile
                               : kTile * std::max(1, ceil_div(ceil_div(Lmax, kTile), kMaxSplits));
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
  const bool direct = L.nsplit == 1;  // the partial kernel writes the output; no merge
  {
    ProfScope prof("attn_partial", stream);
    if (R > 16)
      klaunch(attn_partial_kernel<true>, grid, kAttnThreads, 0, stream, 
          q, reinterpret_cast<const uint4*>(k_new), reinterpret_cast<const uint4*>(v_new),
          reinterpret_cast<uint4*>(k_cache), reinterpret_cast<uint4*>(v_cache), cache_pos, n, H,
          Hkv, hd, Lmax, L.chunk, L.rgroups, R, scale, pm, pl, po, direct ? out : nullptr);
    else
      klaunch(attn_partial_kernel<false>, grid, kAttnThreads, 0, stream, 
          q, reinterpret_cast<const uint4*>(k_new), reinterpret_cast<const uint4*>(v_new),
          reinterpret_cast<uint4*>(k_cache), reinterpret_cast<uint4*>(v_cache), cache_pos, n, H,
          Hkv, hd, Lmax, L.chunk, L.rgroups, R, scale, pm, pl, po, direct ? out : nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (direct) return hipSuccess;
  ProfScope prof("attn_combine", stream);
  klaunch(attn_combine_kernel, B * Hkv * R, kMaxHd, 0, stream, n, H, Hkv, hd, R, L.nsplit, pm, pl, po,
                                                          out);
  return hipGetLastError();
}

hipError_t launch_kv_rollback(int32_t* cache_pos, const int32_t* accept_len, int B, int n,
                              hipStream_t stream) {
  ProfScope prof("kv_rollback", stream);
  klaunch(kv_rollback_kernel, ceil_div(B, 256), 256, 0, stream, cache_pos, accept_len, B, n);
  return hipGetLastError();
}

}  // namespace sirius
