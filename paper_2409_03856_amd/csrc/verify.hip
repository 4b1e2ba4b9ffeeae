// Correction check of a drafted chunk on gfx950 (Algorithm 1; Sec. 4 "How to correct").
//
// verify_stats_kernel  grid (splits, B*R): each workgroup streams one
//                      contiguous segment of one logit row once (16-byte loads)
//                      and keeps, per thread, the running max, the sum of
//                      exp((L - max) / T) in fp64, and the first argmax. Wave
//                      shuffles and a fixed-order merge of the four waves give
//                      one partial per (row, segment).
// verify_scan_kernel   one workgroup per batch entry: merges the segments of
//                      each row in segment order, forms q_j = softmax(L_j/T)
//                      [drafted_j], finds the first j with q_j < r, and picks
//                      the corrected token (argmax of row accept_len, or of the
//                      bonus row).
//
// The pass is HBM-bound: B*R*V*4 bytes are read exactly once.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

constexpr int kVerifyThreads = 256;
constexpr int kMinSegment = 2048;    // logits per workgroup at least
constexpr int kTargetBlocks = 2048;  // enough workgroups to cover 256 CUs several times
constexpr int kMaxRows = 1024;       // R limit of the scan kernel

struct Stat {
  float m;    // running max of the raw logits
  double s;   // sum of exp2((L - m) * c)
  float bv;   // argmax value
  int bi;     // argmax index (lowest among equal values)
};

__device__ __forceinline__ void stat_merge(Stat& a, const Stat& b, float c) {
  // softmax sums: rescale both to the larger max
  const float m = fmaxf(a.m, b.m);
  double s = 0.0;
  if (a.s > 0.0) s += a.s * (double)exp2f((a.m - m) * c);
  if (b.s > 0.0) s += b.s * (double)exp2f((b.m - m) * c);
  a.m = m;
  a.s = s;
  if (b.bv > a.bv || (b.bv == a.bv && b.bi < a.bi)) {
    a.bv = b.bv;
    a.bi = b.bi;
  }
}

__device__ __forceinline__ Stat stat_shfl_xor(const Stat& v, int mask) {
  Stat o;
  o.m = __shfl_xor(v.m, mask, kWave);
  o.s = __shfl_xor(v.s, mask, kWave);
  o.bv = __shfl_xor(v.bv, mask, kWave);
  o.bi = __shfl_xor(v.bi, mask, kWave);
  return o;
}

// Fold G groups of 4 logits (group g starts at index i0[g]) into the running stat:
// one max over all of them, one rescale of the running sum, then the exps.
template <int G>
__device__ __forceinline__ void stat_fold(Stat& st, const float4* v, const int* i0, float c) {
  float m = st.m;
#pragma unroll
  for (int g = 0; g < G; ++g) m = fmaxf(fmaxf(m, fmaxf(v[g].x, v[g].y)), fmaxf(v[g].z, v[g].w));
  double s = (st.s > 0.0) ? st.s * (double)exp2f((st.m - m) * c) : 0.0;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float e[4] = {v[g].x, v[g].y, v[g].z, v[g].w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      s += (double)exp2f((e[q] - m) * c);
      if (e[q] > st.bv) {
        st.bv = e[q];
        st.bi = i0[g] + q;
      }
    }
  }
  st.m = m;
  st.s = s;
}

__device__ __forceinline__ void stat_fold1(Stat& st, float v, int i, float c) {
  const float m = fmaxf(st.m, v);
  double s = (st.s > 0.0) ? st.s * (double)exp2f((st.m - m) * c) : 0.0;
  s += (double)exp2f((v - m) * c);
  if (v > st.bv) {
    st.bv = v;
    st.bi = i;
  }
  st.m = m;
  st.s = s;
}

__global__ __launch_bounds__(kVerifyThreads) void verify_stats_kernel(
    const float* __restrict__ logits, int V, int seg, float c, float* __restrict__ pm,
    double* __restrict__ ps, float* __restrict__ pbv, int* __restrict__ pbi) {
  __shared__ Stat s_w[kVerifyThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int split = blockIdx.x, row = blockIdx.y, splits = gridDim.x;
  const int lo = split * seg;
  const int hi = min(V, lo + seg);
  const float* L = logits + (size_t)row * V;

  Stat st;
  st.m = -INFINITY;
  st.s = 0.0;
  st.bv = -INFINITY;
  st.bi = 0x7fffffff;

  if ((V & 3) == 0) {
    // 16-byte loads; seg is a multiple of 4 so lo is 16-byte aligned.
    const float4* L4 = reinterpret_cast<const float4*>(L);
    const int lo4 = lo >> 2, hi4 = (hi + 3) >> 2;  // hi is V or a multiple of 4
    int i = lo4 + tid;
    for (; i + 3 * kVerifyThreads < hi4; i += 4 * kVerifyThreads) {
      const float4 v[4] = {ld_stream(L4 + i), ld_stream(L4 + i + kVerifyThreads),
                           ld_stream(L4 + i + 2 * kVerifyThreads), ld_stream(L4 + i + 3 * kVerifyThreads)};
      const int i0[4] = {4 * i, 4 * (i + kVerifyThreads), 4 * (i + 2 * kVerifyThreads),
                         4 * (i + 3 * kVerifyThreads)};
      stat_fold<4>(st, v, i0, c);
    }
    for (; i < hi4; i += kVerifyThreads) {
      const float4 v[1] = {ld_stream(L4 + i)};
      const int i0[1] = {4 * i};
      stat_fold<1>(st, v, i0, c);
    }
  } else {
    for (int i = lo + tid; i < hi; i += kVerifyThreads) stat_fold1(st, L[i], i, c);
  }

  // Threads hold interleaved index sets, so ties are settled by index in the merge.
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    Stat o = stat_shfl_xor(st, m);
    stat_merge(st, o, c);
  }
  if (lane == 0) s_w[wave] = st;
  __syncthreads();
  if (tid == 0) {
    Stat a = s_w[0];
    for (int w = 1; w < kVerifyThreads / kWave; ++w) stat_merge(a, s_w[w], c);
    const size_t o = (size_t)row * splits + split;
    pm[o] = a.m;
    ps[o] = a.s;
    pbv[o] = a.bv;
    pbi[o] = a.bi;
  }
}

__global__ __launch_bounds__(256) void verify_scan_kernel(
    const float* __restrict__ logits, int K, int R, int V, const int32_t* __restrict__ drafted,
    float r, float c, int splits, const float* __restrict__ pm, const double* __restrict__ ps,
    const float* __restrict__ pbv, const int* __restrict__ pbi, int32_t* __restrict__ accept_len,
    int32_t* __restrict__ next_token, float* __restrict__ p_draft) {
  __shared__ float s_q[kMaxRows];
  __shared__ int s_amax[kMaxRows];
  const int b = blockIdx.x;
  for (int j = threadIdx.x; j < R; j += blockDim.x) {
    const size_t row = (size_t)b * R + j;
    Stat a;
    a.m = pm[row * splits];
    a.s = ps[row * splits];
    a.bv = pbv[row * splits];
    a.bi = pbi[row * splits];
    for (int sp = 1; sp < splits; ++sp) {
      Stat o;
      o.m = pm[row * splits + sp];
      o.s = ps[row * splits + sp];
      o.bv = pbv[row * splits + sp];
      o.bi = pbi[row * splits + sp];
      stat_merge(a, o, c);
    }
    s_amax[j] = a.bi;
    if (j < K) {
      const int tok = drafted[(size_t)b * K + j];
      float q = 0.f;
      if (tok >= 0 && tok < V) {
        const float lt = logits[row * V + tok];
        q = (float)((double)exp2f((lt - a.m) * c) / a.s);
      }
      s_q[j] = q;
      if (p_draft != nullptr) p_draft[(size_t)b * K + j] = q;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = K;
    for (int j = 0; j < K; ++j) {
      if (s_q[j] < r) {
        acc = j;
        break;
      }
    }
    accept_len[b] = acc;
    next_token[b] = (acc < K) ? s_amax[acc] : ((R == K + 1) ? s_amax[K] : -1);
  }
}

}  // namespace

VerifyLayout verify_layout(int B, int R, int V) {
  VerifyLayout L{};
  const int rows = std::max(1, B * R);
  int splits = ceil_div(kTargetBlocks, rows);
  splits = std::max(1, std::min(splits, ceil_div(V, kMinSegment)));
  L.splits = splits;
  const size_t n = (size_t)rows * splits;
  Carve c;
  L.part = c.take(n * (sizeof(float) * 2 + sizeof(double) + sizeof(int)));
  L.total = c.off;
  return L;
}

hipError_t launch_verify(const float* logits, int B, int K, int R, int V, const int32_t* drafted,
                         float r, float temperature, int32_t* accept_len, int32_t* next_token,
                         float* p_draft, char* ws, const VerifyLayout& L, hipStream_t stream) {
  if (R > kMaxRows) return hipErrorInvalidValue;
  const int splits = L.splits;
  int seg = ceil_div(V, splits);
  seg = (seg + 3) & ~3;
  const size_t n = (size_t)B * R * splits;
  char* p = ws + L.part;
  double* ps = reinterpret_cast<double*>(p);
  float* pm = reinterpret_cast<float*>(p + n * sizeof(double));
  float* pbv = pm + n;
  int* pbi = reinterpret_cast<int*>(pbv + n);
  // exp((L - m) / T) = exp2((L - m) * log2(e) / T); the factor is formed in double.
  const float c = (float)(1.4426950408889634 / (double)temperature);
  {
    ProfScope prof("verify_stats", stream);
    verify_stats_kernel<<<dim3(splits, B * R), kVerifyThreads, 0, stream>>>(logits, V, seg, c, pm,
                                                                            ps, pbv, pbi);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  ProfScope prof("verify_scan", stream);
  verify_scan_kernel<<<B, 256, 0, stream>>>(logits, K, R, V, drafted, r, c, splits, pm, ps, pbv,
                                            pbi, accept_len, next_token, p_draft);
  return hipGetLastError();
}

}  // namespace sirius
