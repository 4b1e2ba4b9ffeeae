// Correction check of a drafted chunk on gfx950 (Algorithm 1; Sec. 4 "How to correct").
//
// verify_stats_kernel  grid (splits, B*R): each workgroup streams one
//                      contiguous segment of one logit row once (16-byte loads)
//                      and keeps, per thread, the running max, the sum of
//                      exp((L - max) / T) in fp64, and the first argmax. Wave
//                      shuffles and a fixed-order merge of the four waves give
//                      one partial per (row, segment).
//                      The workgroup whose segment holds the row's drafted token
//                      also records that token's logit.
// verify_scan_kernel   one workgroup per batch entry: merges the segments of
//                      each row (lanes over segments, fixed-order butterfly),
//                      forms q_j = softmax(L_j/T)[drafted_j], finds the first
//                      j with q_j < r, and picks the corrected token (argmax of
//                      row accept_len, or of the bonus row).
//
// The pass is HBM-bound: B*R*V*4 bytes are read exactly once.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "softmax.h"

namespace sirius {
namespace {

constexpr int kVerifyThreads = 256;
constexpr int kMinSegment = 2048;    // logits per workgroup at least
constexpr int kTargetBlocks = 512;   // two workgroups per CU, each streaming several passes
constexpr int kMaxRows = 1024;       // R limit of the scan kernel
constexpr int kChunk = 8;            // float4 loads in flight per stats thread
constexpr int kScanThreads = 1024;   // scan workgroup: 16 waves
constexpr int kMaxSplits = 64;       // segments per row at most (one wave merges a row)
constexpr int kMaxTreeW = 64;        // tree width limit of the tree scan (one wave of leaves)

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

// Fold G groups of 4 logits (group g starts at index i0[g], groups in increasing index order)
// into the running stat: one max over all of them and one rescale of the running sum; the
// chunk's exps are summed pairwise in fp32 (at most 4 G terms, each at most 1) and added to the
// fp64 sum. The argmax is looked up only when the chunk raises the maximum: the first index
// holding the new maximum (ties with earlier chunks keep the earlier, lower index).
template <int G>
__device__ __forceinline__ void stat_fold(Stat& st, const float4* v, const int* i0, float c) {
  float m = st.m;
#pragma unroll
  for (int g = 0; g < G; ++g) m = fmaxf(fmaxf(m, fmaxf(v[g].x, v[g].y)), fmaxf(v[g].z, v[g].w));
  if (m > st.m) {
    int bi = st.bi;
#pragma unroll
    for (int g = G - 1; g >= 0; --g) {
      bi = (v[g].w == m) ? i0[g] + 3 : bi;
      bi = (v[g].z == m) ? i0[g] + 2 : bi;
      bi = (v[g].y == m) ? i0[g] + 1 : bi;
      bi = (v[g].x == m) ? i0[g] : bi;
    }
    st.bv = m;
    st.bi = bi;
  }
  float t[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float a = exp2_nonpos((v[g].x - m) * c) + exp2_nonpos((v[g].y - m) * c);
    const float b = exp2_nonpos((v[g].z - m) * c) + exp2_nonpos((v[g].w - m) * c);
    t[g] = a + b;
  }
#pragma unroll
  for (int w = 1; w < G; w <<= 1) {
#pragma unroll
    for (int g = 0; g + w < G; g += 2 * w) t[g] += t[g + w];
  }
  double s = (st.s > 0.0) ? st.s * (double)exp2_nonpos((st.m - m) * c) : 0.0;
  if (m > -INFINITY) s += (double)t[0];  // a chunk of -inf logits adds nothing
  st.m = m;
  st.s = s;
}

__device__ __forceinline__ void stat_fold1(Stat& st, float v, int i, float c) {
  const float m = fmaxf(st.m, v);
  double s = (st.s > 0.0) ? st.s * (double)exp2_nonpos((st.m - m) * c) : 0.0;
  if (v > -INFINITY) s += (double)exp2_nonpos((v - m) * c);
  if (v > st.bv) {
    st.bv = v;
    st.bi = i;
  }
  st.m = m;
  st.s = s;
}

__global__ __launch_bounds__(kVerifyThreads) void verify_stats_kernel(
    const float* __restrict__ logits, int V, int seg, float c, const int32_t* __restrict__ drafted,
    int K, int R, float* __restrict__ pm, double* __restrict__ ps, float* __restrict__ pbv,
    int* __restrict__ pbi, float* __restrict__ pd) {
  __shared__ Stat s_w[kVerifyThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int split = blockIdx.x, row = blockIdx.y, splits = gridDim.x;
  const int lo = split * seg;
  const int hi = min(V, lo + seg);
  const float* L = logits + (size_t)row * V;
  // the drafted token of this row, if it falls in this segment: its logit goes to pd
  const int j = row % R;
  const int tok = (j < K) ? drafted[(size_t)(row / R) * K + j] : -1;
  const bool mine = tok >= lo && tok < hi;
  const float lt = (mine && tid == 0) ? L[tok] : -INFINITY;

  Stat st;
  st.m = -INFINITY;
  st.s = 0.0;
  st.bv = -INFINITY;
  st.bi = 0x7fffffff;

  if ((V & 3) == 0) {
    // 16-byte loads, kChunk per thread in flight; seg is a multiple of 4 so lo is 16-byte
    // aligned. Groups of 4 logits in a chunk are folded with one rescale per chunk.
    // Two chunks are in flight per thread: the next chunk's loads are issued before this one is
    // folded, so the exps of one chunk overlap the loads of the next. Every lane issues every
    // load (past the segment it re-reads the segment's last 16 bytes), which keeps the waits
    // exact; the values past the segment are then replaced by -inf, which changes neither the
    // max, the sum nor the argmax.
    const float4* L4 = reinterpret_cast<const float4*>(L);
    const int lo4 = lo >> 2, hi4 = (hi + 3) >> 2;  // hi is V or a multiple of 4
    constexpr int kStep = kChunk * kVerifyThreads;
    auto issue = [&](float4(&v)[kChunk], int i) {
#pragma unroll
      for (int g = 0; g < kChunk; ++g) {
        const int k = i + g * kVerifyThreads;
        v[g] = ld_stream(L4 + (k < hi4 ? k : hi4 - 1));
      }
    };
    auto fold = [&](float4(&v)[kChunk], int i) {
      int i0[kChunk];
#pragma unroll
      for (int g = 0; g < kChunk; ++g) {
        const int k = i + g * kVerifyThreads;
        const bool in = k < hi4;
        v[g].x = in ? v[g].x : -INFINITY;
        v[g].y = in ? v[g].y : -INFINITY;
        v[g].z = in ? v[g].z : -INFINITY;
        v[g].w = in ? v[g].w : -INFINITY;
        i0[g] = 4 * k;
      }
      stat_fold<kChunk>(st, v, i0, c);
    };
    float4 va[kChunk], vb[kChunk];
    const int i_first = lo4 + tid;
    issue(va, i_first);
    for (int i = i_first; i < hi4; i += 2 * kStep) {
      issue(vb, i + kStep);
      fold(va, i);
      if (i + kStep >= hi4) break;
      issue(va, i + 2 * kStep);
      fold(vb, i + kStep);
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
    pd[o] = lt;
  }
}

__device__ __forceinline__ float drafted_q(const Stat& a, float lt, float c) {
  return (lt > -INFINITY) ? (float)((double)exp2f((lt - a.m) * c) / a.s) : 0.f;
}

// Merges the split partials of rows [0, R) of batch entry b. A row's splits sit on a group of
// S2 lanes (S2 = splits rounded up to a power of two), so a wave covers 64 / S2 rows per pass;
// the group's butterfly merge has a fixed order. The drafted token's logit comes from the
// split that holds it (-inf if none: an id outside [0, V), which then gets q = 0). Writes the
// row's argmax to s_amax[j] and, for rows j < Kd, q_j to s_q[j] (and q_out, if given).
__device__ __forceinline__ void merge_rows(int b, int R, int Kd, int splits, float c,
                                           const float* __restrict__ pm,
                                           const double* __restrict__ ps,
                                           const float* __restrict__ pbv,
                                           const int* __restrict__ pbi,
                                           const float* __restrict__ pd, float* s_q, int* s_amax,
                                           float* __restrict__ q_out) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  int lg = 0;
  while ((1 << lg) < splits) ++lg;
  const int S2 = 1 << lg, rpp = kWave >> lg;
  const int sub = lane & (S2 - 1), rsub = lane >> lg;
  const int npass = (R + rpp - 1) / rpp;
  constexpr int kPB = 2;  // passes per iteration, all their loads issued before any merge
  for (int p0 = wave; p0 < npass; p0 += kPB * nw) {
    Stat a[kPB];
    float lt[kPB];
    int j[kPB];
#pragma unroll
    for (int u = 0; u < kPB; ++u) {
      j[u] = (p0 + u * nw) * rpp + rsub;
      a[u].m = -INFINITY;
      a[u].s = 0.0;
      a[u].bv = -INFINITY;
      a[u].bi = 0x7fffffff;
      lt[u] = -INFINITY;
      if (p0 + u * nw < npass && j[u] < R && sub < splits) {
        const size_t i = ((size_t)b * R + j[u]) * splits + sub;
        a[u].m = pm[i];
        a[u].s = ps[i];
        a[u].bv = pbv[i];
        a[u].bi = pbi[i];
        lt[u] = pd[i];
      }
    }
#pragma unroll
    for (int u = 0; u < kPB; ++u) {
      for (int msk = 1; msk < S2; msk <<= 1) {
        const Stat o = stat_shfl_xor(a[u], msk);
        stat_merge(a[u], o, c);
        lt[u] = fmaxf(lt[u], __shfl_xor(lt[u], msk, kWave));
      }
      if (sub == 0 && p0 + u * nw < npass && j[u] < R) {
        s_amax[j[u]] = a[u].bi;
        if (j[u] < Kd) {
          const float q = drafted_q(a[u], lt[u], c);
          s_q[j[u]] = q;
          if (q_out != nullptr) q_out[(size_t)b * Kd + j[u]] = q;
        }
      }
    }
  }
}

__global__ __launch_bounds__(kScanThreads) void verify_scan_kernel(
    int K, int R, int splits, float r, float c, const float* __restrict__ pm,
    const double* __restrict__ ps, const float* __restrict__ pbv, const int* __restrict__ pbi,
    const float* __restrict__ pd, int32_t* __restrict__ accept_len,
    int32_t* __restrict__ next_token, float* __restrict__ p_draft) {
  __shared__ float s_q[kMaxRows];
  __shared__ int s_amax[kMaxRows];
  __shared__ int s_first;
  const int b = blockIdx.x;
  if (threadIdx.x == 0) s_first = K;
  merge_rows(b, R, K, splits, c, pm, ps, pbv, pbi, pd, s_q, s_amax, p_draft);
  __syncthreads();
  // first rejection: the lowest j < K with q_j < r
  for (int j = threadIdx.x; j < K; j += blockDim.x)
    if (s_q[j] < r) atomicMin(&s_first, j);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int acc = s_first;
    accept_len[b] = acc;
    next_token[b] = (acc < K) ? s_amax[acc] : ((R == K + 1) ? s_amax[K] : -1);
  }
}

// Tree verification (Sec. 4, hardware-friendly tree building): rows [i * W + w] are the
// nodes of step i, then W bonus rows if given. Each leaf's root path is walked back through
// the parent links; its advance is the first step whose node has q < r (else K), and the leaf
// with the longest advance (lowest slot on ties) is kept.
__global__ __launch_bounds__(kScanThreads) void tree_scan_kernel(
    int K, int W, int bonus, const int32_t* __restrict__ parents, int splits, float r, float c,
    const float* __restrict__ pm, const double* __restrict__ ps, const float* __restrict__ pbv,
    const int* __restrict__ pbi, const float* __restrict__ pd, int32_t* __restrict__ best_leaf,
    int32_t* __restrict__ accept_len, int32_t* __restrict__ next_token,
    float* __restrict__ q_out) {
  __shared__ float s_q[kMaxRows];
  __shared__ int s_amax[kMaxRows];
  __shared__ int s_par[kMaxRows];
  __shared__ int s_path[kMaxRows];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int KW = K * W, R = KW + (bonus ? W : 0);
  // the parent links are requested before the merge's loads and stored after it (KW <= 1024,
  // one per thread), so both round trips overlap
  const int par = tid < KW ? parents[(size_t)b * KW + tid] : 0;
  merge_rows(b, R, KW, splits, c, pm, ps, pbv, pbi, pd, s_q, s_amax, q_out);
  if (tid < KW) s_par[tid] = par;
  __syncthreads();
  if (tid < kWave) {  // wave 0: lane w walks leaf w's path (W <= 64)
    int adv = K, w = tid;
    if (tid < W) {
      for (int i = K - 1; i >= 0; --i) {
        s_path[tid * K + i] = w;
        if (s_q[i * W + w] < r) adv = i;  // the last one set is the first on the path
        if (i > 0) {
          const int p = s_par[i * W + w];
          w = (p >= 0 && p < W) ? p : 0;  // links outside [0, W) are a caller error; stay in bounds
        }
      }
    }
    // longest advance, lowest slot on ties: the largest of adv * 128 + (127 - slot)
    int key = (tid < W) ? adv * 128 + (127 - tid) : -1;
#pragma unroll
    for (int k = 1; k < kWave; k <<= 1) key = max(key, __shfl_xor(key, k, kWave));
    if (tid == 0) {
      const int best = 127 - (key & 127), acc = key >> 7;
      best_leaf[b] = best;
      accept_len[b] = acc;
      next_token[b] = (acc < K) ? s_amax[acc * W + s_path[best * K + acc]]
                                : (bonus ? s_amax[KW + best] : -1);
    }
  }
}

}  // namespace

VerifyLayout verify_layout(int B, int R, int V) {
  VerifyLayout L{};
  const int rows = std::max(1, B * R);
  int splits = ceil_div(kTargetBlocks, rows);
  splits = std::max(1, std::min(std::min(splits, ceil_div(V, kMinSegment)), kMaxSplits));
  L.splits = splits;
  const size_t n = (size_t)rows * splits;
  Carve c;
  L.part = c.take(n * (sizeof(float) * 3 + sizeof(double) + sizeof(int)));
  L.total = c.off;
  return L;
}

namespace {

struct Parts {
  float* pm;
  double* ps;
  float* pbv;
  int* pbi;
  float* pd;
};

// Per-(row, split) softmax partials of B * R rows; rows j < Kd of each batch entry have a
// drafted token drafted[b * Kd + j] whose logit is recorded.
hipError_t launch_stats(const float* logits, int B, int R, int V, const int32_t* drafted, int Kd,
                        float c, char* ws, const VerifyLayout& L, hipStream_t stream, Parts* P,
                        const char* prof_name) {
  const int splits = L.splits;
  int seg = ceil_div(V, splits);
  seg = (seg + 3) & ~3;
  const size_t n = (size_t)B * R * splits;
  char* p = ws + L.part;
  P->ps = reinterpret_cast<double*>(p);
  P->pm = reinterpret_cast<float*>(p + n * sizeof(double));
  P->pbv = P->pm + n;
  P->pbi = reinterpret_cast<int*>(P->pbv + n);
  P->pd = reinterpret_cast<float*>(P->pbi + n);
  ProfScope prof(prof_name, stream);
  klaunch(verify_stats_kernel, dim3(splits, B * R), kVerifyThreads, 0, stream, 
      logits, V, seg, c, drafted, Kd, R, P->pm, P->ps, P->pbv, P->pbi, P->pd);
  return hipGetLastError();
}

// exp((L - m) / T) = exp2((L - m) * log2(e) / T); the factor is formed in double.
float exp2_factor(float temperature) { return (float)(1.4426950408889634 / (double)temperature); }

}  // namespace

hipError_t launch_verify(const float* logits, int B, int K, int R, int V, const int32_t* drafted,
                         float r, float temperature, int32_t* accept_len, int32_t* next_token,
                         float* p_draft, char* ws, const VerifyLayout& L, hipStream_t stream) {
  if (R > kMaxRows) return hipErrorInvalidValue;
  const float c = exp2_factor(temperature);
  Parts P;
  hipError_t e = launch_stats(logits, B, R, V, drafted, K, c, ws, L, stream, &P, "verify_stats");
  if (e != hipSuccess) return e;
  ProfScope prof("verify_scan", stream);
  klaunch(verify_scan_kernel, B, kScanThreads, 0, stream, K, R, L.splits, r, c, P.pm, P.ps, P.pbv, P.pbi, P.pd,
                                            accept_len, next_token, p_draft);
  return hipGetLastError();
}

hipError_t launch_tree_verify(const float* logits, int B, int K, int W, int V, int bonus,
                              const int32_t* tokens, const int32_t* parents, float r,
                              float temperature, int32_t* best_leaf, int32_t* accept_len,
                              int32_t* next_token, float* q, char* ws, const VerifyLayout& L,
                              hipStream_t stream) {
  const int R = K * W + (bonus ? W : 0);
  if (R > kMaxRows || W > kMaxTreeW) return hipErrorInvalidValue;
  const float c = exp2_factor(temperature);
  Parts P;
  hipError_t e = launch_stats(logits, B, R, V, tokens, K * W, c, ws, L, stream, &P, "tree_stats");
  if (e != hipSuccess) return e;
  ProfScope prof("tree_scan", stream);
  klaunch(tree_scan_kernel, B, kScanThreads, 0, stream, K, W, bonus, parents, L.splits, r, c, P.pm, P.ps, P.pbv,
                                          P.pbi, P.pd, best_leaf, accept_len, next_token, q);
  return hipGetLastError();
}

}  // namespace sirius
