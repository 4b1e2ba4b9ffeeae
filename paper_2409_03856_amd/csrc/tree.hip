// Tree drafting step on gfx950 (Sec. 4, hardware-friendly tree building): from the sparse
// model's logits at the Wc current leaves of each tree, keep the W expansions (parent leaf,
// token) of largest cumulative log-likelihood, ties to the lower parent slot, then the lower
// token id; the new leaves come out best first.
//
// Only a leaf's W most likely tokens can be among the W best expansions (the parent's
// cumulative value is common to its tokens), and within a leaf the order of log-likelihoods is
// the order of the raw logits. A candidate is a 64-bit key that orders (logit descending, token
// ascending): the logit's bits mapped to an order-preserving unsigned value above the
// complemented token id. Keys of one row are distinct; 0 marks an empty entry.
//
//  tree_topw_kernel    grid (splits, B * Wc): each workgroup reads one segment of one leaf's
//                      logit row once, in passes of 4096 with each thread holding a contiguous
//                      run of 16 logits (all loads in flight), keeping the running softmax
//                      statistics (max, sum of exp((v - max) / T) in fp64). The threads form G
//                      interleaved groups (G the power of two at or above W); the pass's W
//                      best are at least the W-th largest group maximum, so only the keys at
//                      or above that bound (usually a handful) are gathered and ranked by
//                      counting together with the running W best.
//  tree_select_kernel  one 1024-thread workgroup per tree, one wave per leaf and one lane per
//                      segment: the segment statistics merge in a fixed butterfly order into
//                      log-likelihood (v - max) / T - log(sum), W rounds of a DPP wave maximum
//                      over the segment lists' heads give the leaf's W best tokens, and the
//                      Wc x W scored candidates are ranked by counting.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "softmax.h"

namespace sirius {
namespace {

constexpr int kTopThreads = 256;
constexpr int kElems = 16;  // contiguous logits per thread per pass (the stats sum assumes 16)
constexpr int kPassElems = kTopThreads * kElems;   // 4096 logits per workgroup pass
constexpr int kKW = 16;          // tree width and current-leaf limit (list length in registers)
constexpr int kMaxSplits = 64;   // segments per leaf row at most (one lane each in the select)
constexpr int kSelThreads = 1024;
constexpr int kRankBatch = 16;   // LDS reads in flight per step of a rank-by-counting loop

__device__ __forceinline__ uint32_t ordered_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_ordered(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
// larger key = larger logit, then lower token
__device__ __forceinline__ uint64_t make_key(float v, int i) {
  return ((uint64_t)ordered_bits(v) << 32) | (uint64_t)(~(uint32_t)i);
}
__device__ __forceinline__ int key_token(uint64_t k) { return (int)(~(uint32_t)k); }
__device__ __forceinline__ float key_value(uint64_t k) { return from_ordered((uint32_t)(k >> 32)); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)v, m, kWave);
  const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, kWave);
  return ((uint64_t)hi << 32) | lo;
}

// v = max(v, v moved by one DPP step); rows outside ROWS keep v
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t max_dpp(uint64_t v) {
  const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
  const uint32_t olo = (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xf, false);
  const uint32_t ohi = (uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xf, false);
  const uint64_t o = ((uint64_t)ohi << 32) | olo;
  return o > v ? o : v;
}

// Maximum over the 64 lanes, returned to every lane; all lanes must be active. Swaps within
// quads, rotations by 4 and 8 within rows of 16, then row 0's and row 1's results broadcast
// into the rows above: lane 63 ends with the maximum.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = max_dpp<0xB1, 0xF>(v);   // quad_perm [1, 0, 3, 2]
  v = max_dpp<0x4E, 0xF>(v);   // quad_perm [2, 3, 0, 1]
  v = max_dpp<0x124, 0xF>(v);  // row_ror:4
  v = max_dpp<0x128, 0xF>(v);  // row_ror:8
  v = max_dpp<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v = max_dpp<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

// running softmax statistics, merged to the larger max
__device__ __forceinline__ void sm_merge(float& m, double& s, float om, double os, float c) {
  const float mm = fmaxf(m, om);
  double ns = 0.0;
  if (s > 0.0) ns += s * (double)exp2f((m - mm) * c);
  if (os > 0.0) ns += os * (double)exp2f((om - mm) * c);
  m = mm;
  s = ns;
}

__global__ __launch_bounds__(kTopThreads) void tree_topw_kernel(
    const float* __restrict__ logits, int V, int seg, int W, float c, float* __restrict__ rm,
    double* __restrict__ rs, uint64_t* __restrict__ rk) {
  // [0, kKW): the running W best (0 = empty); from kKW: this pass's entrants
  __shared__ uint64_t s_cand[kKW + kPassElems + kRankBatch];
  __shared__ uint64_t s_g[(kTopThreads / kWave) * kKW];  // group maxima per wave
  __shared__ uint64_t s_new[kKW];
  __shared__ uint64_t s_bound;
  __shared__ float s_m[kTopThreads / kWave];
  __shared__ double s_s[kTopThreads / kWave];
  __shared__ int s_scan[kTopThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int split = blockIdx.x, row = blockIdx.y, splits = gridDim.x;
  const int lo = split * seg, hi = min(V, lo + seg);
  const float* L = logits + (size_t)row * V;
  int G = 1;
  while (G < W) G <<= 1;

  float m = -INFINITY;
  double s = 0.0;
  if (tid < kKW) s_cand[tid] = 0;
  uint64_t run_w = 0;  // the running W-th best key (0 while fewer than W)

  for (int base = lo; base < hi; base += kPassElems) {
    const int e0 = base + tid * kElems;
    float v[kElems];
    if ((V & 3) == 0) {  // seg is a multiple of 4, so e0 and hi are too: whole float4s
      const float4* L4 = reinterpret_cast<const float4*>(L + e0);
#pragma unroll
      for (int g = 0; g < kElems / 4; ++g) {
        const float4 x = (e0 + 4 * g < hi) ? ld_stream(L4 + g)
                                           : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        v[4 * g] = x.x;
        v[4 * g + 1] = x.y;
        v[4 * g + 2] = x.z;
        v[4 * g + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < kElems; ++j) v[j] = (e0 + j < hi) ? L[e0 + j] : -INFINITY;
    }
    // softmax statistics, one rescale per pass
    float cm = m;
#pragma unroll
    for (int j = 0; j < kElems; ++j) cm = fmaxf(cm, v[j]);
    float t[kElems / 4];  // the pass's exps, summed pairwise in fp32 (16 terms, each <= 1)
#pragma unroll
    for (int g = 0; g < kElems / 4; ++g)
      t[g] = (exp2_nonpos((v[4 * g] - cm) * c) + exp2_nonpos((v[4 * g + 1] - cm) * c)) +
             (exp2_nonpos((v[4 * g + 2] - cm) * c) + exp2_nonpos((v[4 * g + 3] - cm) * c));
    double cs = (s > 0.0) ? s * (double)exp2_nonpos((m - cm) * c) : 0.0;
    if (cm > -INFINITY) cs += (double)((t[0] + t[1]) + (t[2] + t[3]));  // -inf logits add nothing
    m = cm;
    s = cs;
    // keys; the largest key of each of G thread groups (group = thread index mod G, G the
    // power of two at or above W)
    uint64_t key[kElems];
    uint64_t gk = 0;
#pragma unroll
    for (int j = 0; j < kElems; ++j) {
      key[j] = (e0 + j < hi) ? make_key(v[j], e0 + j) : 0;
      gk = key[j] > gk ? key[j] : gk;
    }
    for (int k = G; k < kWave; k <<= 1) {
      const uint64_t o = shfl_xor_u64(gk, k);
      gk = o > gk ? o : gk;
    }
    if (lane < G) s_g[wave * kKW + lane] = gk;
    if (tid == 0) s_bound = 0;
    if (tid < kKW) s_new[tid] = 0;
    __syncthreads();
    // bound: the W-th largest group maximum (W groups hold a key at least that large, so the
    // pass's W best are too), or the running W-th best if larger
    if (tid < G) {
      uint64_t gm[kKW];
#pragma unroll
      for (int g = 0; g < kKW; ++g) {
        uint64_t x = 0;
#pragma unroll
        for (int w = 0; w < kTopThreads / kWave; ++w) {
          const uint64_t y = s_g[w * kKW + g];
          x = y > x ? y : x;
        }
        gm[g] = g < G ? x : 0;
      }
      uint64_t mine = 0;
#pragma unroll
      for (int g = 0; g < kKW; ++g) mine = g == tid ? gm[g] : mine;
      int r = 0;
#pragma unroll
      for (int g = 0; g < kKW; ++g) r += gm[g] > mine;
      if (mine != 0 && r == W - 1) s_bound = mine;
    }
    __syncthreads();
    const uint64_t bound = s_bound > run_w ? s_bound : run_w;
    int n = 0;
#pragma unroll
    for (int j = 0; j < kElems; ++j) n += (key[j] != 0 && key[j] >= bound);
    int total = 0;
    int pos = kKW + block_exclusive_scan_256(n, s_scan, &total);
#pragma unroll
    for (int j = 0; j < kElems; ++j)
      if (key[j] != 0 && key[j] >= bound) s_cand[pos++] = key[j];
    const int ncand = kKW + total;
    const int npad = (ncand + kRankBatch - 1) / kRankBatch * kRankBatch;
    if (tid < npad - ncand) s_cand[ncand + tid] = 0;  // empty: never counted as larger
    __syncthreads();
    // the new running best: rank every candidate by counting (non-empty keys are distinct)
    for (int i = tid; i < ncand; i += kTopThreads) {
      const uint64_t k0 = s_cand[i];
      int r = 0;
      for (int j = 0; j < npad; j += kRankBatch) {
        uint64_t buf[kRankBatch];
#pragma unroll
        for (int q = 0; q < kRankBatch; ++q) buf[q] = s_cand[j + q];
#pragma unroll
        for (int q = 0; q < kRankBatch; ++q) r += (int)(buf[q] > k0);
      }
      if (k0 != 0 && r < W) s_new[r] = k0;
    }
    __syncthreads();
    if (tid < kKW) s_cand[tid] = s_new[tid];
    run_w = s_new[W - 1];
    __syncthreads();
  }

  // softmax statistics: butterfly within the wave, then the four waves in order
#pragma unroll
  for (int k = 1; k < kWave; k <<= 1) {
    const float om = __shfl_xor(m, k, kWave);
    const double os = __shfl_xor(s, k, kWave);
    sm_merge(m, s, om, os, c);
  }
  if (lane == 0) {
    s_m[wave] = m;
    s_s[wave] = s;
  }
  __syncthreads();
  const size_t o = (size_t)row * splits + split;
  if (tid == 0) {
    float am = s_m[0];
    double as = s_s[0];
    for (int w = 1; w < kTopThreads / kWave; ++w) sm_merge(am, as, s_m[w], s_s[w], c);
    rm[o] = am;
    rs[o] = as;
  }
  if (tid < W) rk[o * kKW + tid] = s_cand[tid];
}

__global__ __launch_bounds__(kSelThreads) void tree_select_kernel(
    int Wc, int W, int splits, float c, float inv_t, const float* __restrict__ rm,
    const double* __restrict__ rs, const uint64_t* __restrict__ rk,
    const float* __restrict__ cum_in, int32_t* __restrict__ tokens, int32_t* __restrict__ parents,
    float* __restrict__ cum_out) {
  __shared__ double s_sc[kKW * kKW];  // each leaf's W best, scored: [leaf][rank]
  __shared__ int s_tk[kKW * kKW];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int b = blockIdx.x;
  if (wave < Wc) {  // one wave per leaf, one lane per split
    const size_t row = (size_t)b * Wc + wave;
    const bool has = lane < splits;
    uint64_t lst[kKW];  // the lane's split list, best first (0 = empty)
#pragma unroll
    for (int p = 0; p < kKW; ++p)
      lst[p] = (has && p < W) ? rk[(row * splits + lane) * kKW + p] : 0;
    float m = has ? rm[row * splits + lane] : -INFINITY;
    double s = has ? rs[row * splits + lane] : 0.0;
    const float base = (cum_in != nullptr && lane == 0) ? cum_in[row] : 0.f;
    // statistics of the leaf row: butterfly merge in a fixed order
#pragma unroll
    for (int k = 1; k < kWave; k <<= 1) {
      const float om = __shfl_xor(m, k, kWave);
      const double os = __shfl_xor(s, k, kWave);
      sm_merge(m, s, om, os, c);
    }
    const double lse = log(s);  // log of sum exp((v - m) / T)
    // the leaf's W best: W rounds of a wave maximum over the list heads
    for (int r = 0; r < W; ++r) {
      const uint64_t best = wave_max_u64(lst[0]);
      const bool win = best != 0 && lst[0] == best;  // non-empty keys are distinct
#pragma unroll
      for (int p = 0; p < kKW - 1; ++p) lst[p] = win ? lst[p + 1] : lst[p];
      lst[kKW - 1] = win ? 0 : lst[kKW - 1];
      if (lane == 0) {
        const double lp = ((double)key_value(best) - (double)m) * (double)inv_t - lse;
        s_sc[wave * kKW + r] = best != 0 ? (double)base + lp : -INFINITY;
        s_tk[wave * kKW + r] = best != 0 ? key_token(best) : -1;
      }
    }
  }
  __syncthreads();
  // the W best of the Wc x W: valid first, larger score, lower parent, lower token
  const int m2 = Wc * W;
  for (int i = tid; i < m2; i += kSelThreads) {
    const int leaf = i / W, r0 = i - leaf * W;
    const double sc = s_sc[leaf * kKW + r0];
    const int tk = s_tk[leaf * kKW + r0];
    const bool ok = tk >= 0;
    int r = 0;
    for (int lj = 0; lj < Wc; ++lj) {
      double so[kKW];
      int to[kKW];
#pragma unroll
      for (int rj = 0; rj < kKW; ++rj) {
        so[rj] = s_sc[lj * kKW + rj];
        to[rj] = s_tk[lj * kKW + rj];
      }
#pragma unroll
      for (int rj = 0; rj < kKW; ++rj) {
        const bool okj = to[rj] >= 0;
        const bool tie_lower = (lj < leaf) | ((lj == leaf) & ((to[rj] < tk) | ((to[rj] == tk) & (rj < r0))));
        const bool better = (okj & !ok) | ((okj == ok) & ((so[rj] > sc) | ((so[rj] == sc) & tie_lower)));
        r += (int)((rj < W) & better);
      }
    }
    if (r < W) {
      tokens[(size_t)b * W + r] = ok ? tk : -1;
      parents[(size_t)b * W + r] = ok ? leaf : -1;
      cum_out[(size_t)b * W + r] = (float)sc;
    }
  }
}

}  // namespace

TreeBuildLayout tree_build_layout(int B, int Wc, int W, int V) {
  TreeBuildLayout L{};
  const int rows = std::max(1, B * Wc);
  int splits = ceil_div(V, kPassElems);
  splits = std::min(splits, kMaxSplits);
  L.splits = std::max(1, splits);
  const size_t n = (size_t)rows * L.splits;
  Carve c;
  L.rm = c.take(n * sizeof(float));
  L.rs = c.take(n * sizeof(double));
  L.rk = c.take(n * kKW * sizeof(uint64_t));
  L.total = c.off;
  return L;
}

hipError_t launch_tree_build(const float* logits, int B, int Wc, int V, const float* cum_ll, int W,
                             float temperature, int32_t* tokens, int32_t* parents,
                             float* cum_out, char* ws, const TreeBuildLayout& L,
                             hipStream_t stream) {
  if (W < 1 || W > kKW || Wc < 1 || Wc > kKW || L.splits > kMaxSplits)
    return hipErrorInvalidValue;
  const int splits = L.splits;
  int seg = ceil_div(V, splits);
  seg = (seg + 3) & ~3;
  float* rm = reinterpret_cast<float*>(ws + L.rm);
  double* rs = reinterpret_cast<double*>(ws + L.rs);
  uint64_t* rk = reinterpret_cast<uint64_t*>(ws + L.rk);
  const float c = (float)(1.4426950408889634 / (double)temperature);
  {
    ProfScope prof("tree_topw", stream);
    klaunch(tree_topw_kernel, dim3(splits, B * Wc), kTopThreads, 0, stream, logits, V, seg, W, c, rm, rs,
                                                                     rk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ProfScope prof("tree_select", stream);
  klaunch(tree_select_kernel, B, kSelThreads, 0, stream, Wc, W, splits, c, (float)(1.0 / temperature),
                                                    rm, rs, rk, cum_ll, tokens, parents, cum_out);
  return hipGetLastError();
}

}  // namespace sirius
