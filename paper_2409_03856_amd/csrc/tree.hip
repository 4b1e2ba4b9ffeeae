// Tree drafting step on gfx950 (Sec. 4, hardware-friendly tree building): from the sparse
// model's logits at the Wc current leaves of each tree, keep the W expansions (parent leaf,
// token) of largest cumulative log-likelihood, ties to the lower parent slot, then the lower
// token id; the new leaves come out best first.
//
// Only a leaf's W most likely tokens can be among the W best expansions (the parent's
// cumulative value is common to its tokens), so:
//
//  tree_topw_kernel    grid (splits, B * Wc): each workgroup streams one segment of one leaf's
//                      logit row once and keeps, per thread, the running softmax statistics
//                      (max, sum of exp((v - max) / T) in fp64) and the W largest logits
//                      (lower token first on ties) in registers; four wave merges of the
//                      statistics in a fixed order, W block-argmax rounds for the lists.
//  tree_select_kernel  one workgroup per tree: per leaf, the split statistics merged in a fixed
//                      order give log-likelihood (v - max) / T - log(sum), the split lists give
//                      the leaf's W most likely tokens (W wave-argmax rounds); the Wc x W
//                      candidates are ranked in W more rounds.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

constexpr int kTopThreads = 256;
constexpr int kKW = 16;          // tree width and current-leaf limit (list length in registers)
constexpr int kSegMin = 2048;    // logits per workgroup at least
constexpr int kMaxSplits = 64;   // segments per leaf row at most (candidates per lane <= 16)
constexpr int kTargetBlocks = 2048;

// candidate order: larger value first, then lower token
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

struct Best {  // a wave-argmax candidate: value, token, owner lane
  float v;
  int i, lane;
};

__device__ __forceinline__ Best wave_best(Best b) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    Best o;
    o.v = __shfl_xor(b.v, m, kWave);
    o.i = __shfl_xor(b.i, m, kWave);
    o.lane = __shfl_xor(b.lane, m, kWave);
    if (better(o.v, o.i, b.v, b.i)) b = o;
  }
  return b;
}

__global__ __launch_bounds__(kTopThreads) void tree_topw_kernel(
    const float* __restrict__ logits, int V, int seg, int W, float c, float* __restrict__ rm,
    double* __restrict__ rs, float* __restrict__ rv, int* __restrict__ ri) {
  __shared__ float s_v[kTopThreads * kKW];
  __shared__ int s_i[kTopThreads * kKW];
  __shared__ float s_m[kTopThreads / kWave];
  __shared__ double s_s[kTopThreads / kWave];
  __shared__ Best s_b[kTopThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int split = blockIdx.x, row = blockIdx.y, splits = gridDim.x;
  const int lo = split * seg, hi = min(V, lo + seg);
  const float* L = logits + (size_t)row * V;

  float m = -INFINITY;
  double s = 0.0;
  float tv[kKW];  // the thread's W best so far, best first; (thv, thi) is the W-th
  int ti[kKW];
  float thv = -INFINITY;
  int thi = 0x7fffffff;
#pragma unroll
  for (int p = 0; p < kKW; ++p) {
    tv[p] = -INFINITY;
    ti[p] = 0x7fffffff;
  }
  for (int i = lo + tid; i < hi; i += kTopThreads) {
    const float v = L[i];
    if (v > m) {
      if (s > 0.0) s *= (double)exp2f((m - v) * c);
      m = v;
    }
    s += (double)exp2f((v - m) * c);
    if (better(v, i, thv, thi)) {  // insert, keeping the list sorted
      bool done = false;
#pragma unroll
      for (int p = kKW - 1; p >= 0; --p) {
        if (p < W && !done) {
          if (p > 0 && better(v, i, tv[p - 1], ti[p - 1])) {
            tv[p] = tv[p - 1];
            ti[p] = ti[p - 1];
          } else {
            tv[p] = v;
            ti[p] = i;
            done = true;
          }
        }
      }
#pragma unroll
      for (int p = 0; p < kKW; ++p)
        if (p == W - 1) {
          thv = tv[p];
          thi = ti[p];
        }
    }
  }

  // softmax statistics: wave tree, then the four waves in order
#pragma unroll
  for (int k = 1; k < kWave; k <<= 1) {
    const float om = __shfl_xor(m, k, kWave);
    const double os = __shfl_xor(s, k, kWave);
    const float mm = fmaxf(m, om);
    double ns = 0.0;
    if (s > 0.0) ns += s * (double)exp2f((m - mm) * c);
    if (os > 0.0) ns += os * (double)exp2f((om - mm) * c);
    m = mm;
    s = ns;
  }
  if (lane == 0) {
    s_m[wave] = m;
    s_s[wave] = s;
  }
#pragma unroll
  for (int p = 0; p < kKW; ++p) {
    s_v[tid * kKW + p] = tv[p];
    s_i[tid * kKW + p] = ti[p];
  }
  __syncthreads();
  const size_t o = (size_t)row * splits + split;
  if (tid == 0) {
    float am = s_m[0];
    double as = s_s[0];
    for (int w = 1; w < kTopThreads / kWave; ++w) {
      const float mm = fmaxf(am, s_m[w]);
      double ns = 0.0;
      if (as > 0.0) ns += as * (double)exp2f((am - mm) * c);
      if (s_s[w] > 0.0) ns += s_s[w] * (double)exp2f((s_m[w] - mm) * c);
      am = mm;
      as = ns;
    }
    rm[o] = am;
    rs[o] = as;
  }
  // the workgroup's W best: W rounds of a block argmax over the threads' list heads
  int head = 0;
  for (int round = 0; round < W; ++round) {
    Best b;
    b.v = head < W ? s_v[tid * kKW + head] : -INFINITY;
    b.i = head < W ? s_i[tid * kKW + head] : 0x7fffffff;
    b.lane = tid;
    b = wave_best(b);
    if (lane == 0) s_b[wave] = b;
    __syncthreads();
    Best w0 = s_b[0];
    for (int w = 1; w < kTopThreads / kWave; ++w)
      if (better(s_b[w].v, s_b[w].i, w0.v, w0.i)) w0 = s_b[w];
    if (tid == w0.lane) ++head;
    if (tid == 0) {
      rv[o * kKW + round] = w0.v;
      ri[o * kKW + round] = w0.i;
    }
    __syncthreads();  // s_b is rewritten next round
  }
}

__global__ __launch_bounds__(kTopThreads) void tree_select_kernel(
    int Wc, int W, int splits, float c, float inv_t, const float* __restrict__ rm,
    const double* __restrict__ rs, const float* __restrict__ rv, const int* __restrict__ ri,
    const float* __restrict__ cum_in, int32_t* __restrict__ tokens, int32_t* __restrict__ parents,
    float* __restrict__ cum_out) {
  constexpr int kPer = kMaxSplits * kKW / kWave;  // candidates per lane at most
  __shared__ double s_sc[kKW * kKW];  // leaf-major candidates: score, token
  __shared__ int s_tk[kKW * kKW];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int b = blockIdx.x;
  for (int w = wave; w < Wc; w += kTopThreads / kWave) {  // one wave per leaf
    const size_t row = (size_t)b * Wc + w;
    // statistics of the leaf row: lanes merge splits lane, lane + 64, ..., then a wave tree
    float m = -INFINITY;
    double s = 0.0;
    for (int sp = lane; sp < splits; sp += kWave) {
      const float om = rm[row * splits + sp];
      const double os = rs[row * splits + sp];
      const float mm = fmaxf(m, om);
      double ns = 0.0;
      if (s > 0.0) ns += s * (double)exp2f((m - mm) * c);
      if (os > 0.0) ns += os * (double)exp2f((om - mm) * c);
      m = mm;
      s = ns;
    }
#pragma unroll
    for (int k = 1; k < kWave; k <<= 1) {
      const float om = __shfl_xor(m, k, kWave);
      const double os = __shfl_xor(s, k, kWave);
      const float mm = fmaxf(m, om);
      double ns = 0.0;
      if (s > 0.0) ns += s * (double)exp2f((m - mm) * c);
      if (os > 0.0) ns += os * (double)exp2f((om - mm) * c);
      m = mm;
      s = ns;
    }
    const double lse = log(s);  // log of sum exp((v - m) / T)
    const double base = cum_in != nullptr ? (double)cum_in[row] : 0.0;
    // the leaf's W most likely tokens among its splits' lists
    const int n = splits * W;
    float cv[kPer];
    int ci[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int j = lane + kWave * u;
      const bool ok = j < n;
      const size_t src = (row * splits + (ok ? j / W : 0)) * kKW + (ok ? j % W : 0);
      cv[u] = ok ? rv[src] : -INFINITY;
      ci[u] = ok ? ri[src] : 0x7fffffff;
    }
    for (int round = 0; round < W; ++round) {
      Best bb;
      bb.v = -INFINITY;
      bb.i = 0x7fffffff;
      bb.lane = lane;
      int slot = -1;
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        if (better(cv[u], ci[u], bb.v, bb.i)) {
          bb.v = cv[u];
          bb.i = ci[u];
          slot = u;
        }
      }
      const Best win = wave_best(bb);
      if (lane == win.lane) {
#pragma unroll
        for (int u = 0; u < kPer; ++u)
          if (u == slot) {
            cv[u] = -INFINITY;
            ci[u] = 0x7fffffff;
          }
      }
      if (lane == 0) {
        const double lp = ((double)win.v - (double)m) * (double)inv_t - lse;
        s_sc[w * kKW + round] = (win.i == 0x7fffffff) ? -INFINITY : base + lp;
        s_tk[w * kKW + round] = win.i;
      }
    }
  }
  __syncthreads();
  // rank the Wc x W candidates: larger score, then lower parent, then lower token
  if (wave == 0) {
    constexpr int kC = kKW * kKW / kWave;  // candidates per lane
    double sv[kC];
    int sp_[kC], st[kC];
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int j = lane + kWave * u;  // j = leaf * W + rank
      const bool ok = j < Wc * W;
      const int leaf = ok ? j / W : 0, rank = ok ? j % W : 0;
      // a leaf with fewer than W tokens (V < W) leaves empty entries: they rank last
      st[u] = ok ? s_tk[leaf * kKW + rank] : 0x7fffffff;
      sv[u] = ok ? s_sc[leaf * kKW + rank] : -INFINITY;
      sp_[u] = st[u] != 0x7fffffff ? leaf : 0x7fffffff;
    }
    for (int round = 0; round < W; ++round) {
      double bv = -INFINITY;
      int bp = 0x7fffffff, bt = 0x7fffffff, slot = -1;
#pragma unroll
      for (int u = 0; u < kC; ++u) {
        const bool bt_ = sv[u] > bv || (sv[u] == bv && (sp_[u] < bp || (sp_[u] == bp && st[u] < bt)));
        if (bt_) {
          bv = sv[u];
          bp = sp_[u];
          bt = st[u];
          slot = u;
        }
      }
      int owner = lane;
#pragma unroll
      for (int k = 1; k < kWave; k <<= 1) {
        const double ov = __shfl_xor(bv, k, kWave);
        const int op = __shfl_xor(bp, k, kWave), ot = __shfl_xor(bt, k, kWave);
        const int oo = __shfl_xor(owner, k, kWave);
        if (ov > bv || (ov == bv && (op < bp || (op == bp && ot < bt)))) {
          bv = ov;
          bp = op;
          bt = ot;
          owner = oo;
        }
      }
      if (lane == owner) {
#pragma unroll
        for (int u = 0; u < kC; ++u)
          if (u == slot) {
            sv[u] = -INFINITY;
            sp_[u] = 0x7fffffff;
            st[u] = 0x7fffffff;
          }
      }
      if (lane == 0) {
        tokens[(size_t)b * W + round] = bt;
        parents[(size_t)b * W + round] = bp;
        cum_out[(size_t)b * W + round] = (float)bv;
      }
    }
  }
}

}  // namespace

TreeBuildLayout tree_build_layout(int B, int Wc, int V) {
  TreeBuildLayout L{};
  const int rows = std::max(1, B * Wc);
  int splits = ceil_div(kTargetBlocks, rows);
  splits = std::max(1, std::min(std::min(splits, ceil_div(V, kSegMin)), kMaxSplits));
  L.splits = splits;
  const size_t n = (size_t)rows * splits;
  Carve c;
  L.rm = c.take(n * sizeof(float));
  L.rs = c.take(n * sizeof(double));
  L.rv = c.take(n * kKW * sizeof(float));
  L.ri = c.take(n * kKW * sizeof(int));
  L.total = c.off;
  return L;
}

hipError_t launch_tree_build(const float* logits, int B, int Wc, int V, const float* cum_ll, int W,
                             float temperature, int32_t* tokens, int32_t* parents,
                             float* cum_out, char* ws, const TreeBuildLayout& L,
                             hipStream_t stream) {
  if (W < 1 || W > kKW || Wc < 1 || Wc > kKW) return hipErrorInvalidValue;
  const int splits = L.splits;
  const int seg = ceil_div(V, splits);
  float* rm = reinterpret_cast<float*>(ws + L.rm);
  double* rs = reinterpret_cast<double*>(ws + L.rs);
  float* rv = reinterpret_cast<float*>(ws + L.rv);
  int* ri = reinterpret_cast<int*>(ws + L.ri);
  const float c = (float)(1.4426950408889634 / (double)temperature);
  {
    ProfScope prof("tree_topw", stream);
    tree_topw_kernel<<<dim3(splits, B * Wc), kTopThreads, 0, stream>>>(logits, V, seg, W, c, rm, rs,
                                                                     rv, ri);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ProfScope prof("tree_select", stream);
  tree_select_kernel<<<B, kTopThreads, 0, stream>>>(Wc, W, splits, c, (float)(1.0 / temperature),
                                                    rm, rs, rv, ri, cum_ll, tokens, parents,
                                                    cum_out);
  return hipGetLastError();
}

}  // namespace sirius
