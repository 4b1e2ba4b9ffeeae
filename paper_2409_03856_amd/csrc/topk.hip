// Per-token top-k FSparse on gfx950 (Sec. 3, footnote on the fine-grained implementation: the
// paper keeps the top-k gate activations per token instead of thresholding them, so every
// token has exactly the target density; up and down stay sparse as in CATS).
//
// The k kept neurons depend on all d_ff gate activations of the token, so the pass splits in
// three:
//  1. the gate pass: a = SiLU(W_gate xn) for every neuron into a [B, d_ff] buffer; the whole
//     gate is read once, as in the threshold path (batch 1: the decode kernel's gate phase
//     alone, ffn_decode.hip; 2..64 tokens with d_model % 256 == 0: cats_ring_kernel's gate
//     phase on the exact three-piece input, ffn_batch.hip; other batches: gate_kernel in
//     activation mode, ffn_gemv.hip).
//  2. topk_cut_kernel: one 1024-thread workgroup per token finds the k-th largest top-k key
//     (|a| descending, then the lower index) by a most-significant-digit radix select over the
//     bits of |a| in digits of 11, 11 and 9 bits (LDS histograms, eight copies on the first
//     digit; a block scan over the bins) until the digit holding it has at most 128 members,
//     which are placed by a
//     block scan and ranked by counting on the full key; when every value bit is decided
//     first, a block scan over the threads' contiguous index ranges settles the ties.
//  3. the keyed FFN pass: decode1_kernel (batch 1), cats_ring_kernel + down_ring_kernel
//     (batched, one pass over the tokens' union) or gate_kernel + down_kernel (other small
//     batches) read the stored activations, keep a neuron iff its key reaches the token's cut,
//     and stream W_up and W_down for the kept neurons only; reduce_kernel sums the partials
//     and writes the ascending active lists.
#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "radix_select.h"
#include "topk.h"

namespace sirius {
namespace {

constexpr int kCutThreads = 1024;
constexpr int kCutWaves = kCutThreads / kWave;  // 16
constexpr int kRankMax = 128;  // digit members ranked directly on the full key at most

// Thread t owns neurons [t * PER, t * PER + PER) of the token (contiguous, for the tie scan).
// Digit passes (radix_select.h) from bit 30 down narrow the k-th largest |a| until its digit has
// at most kRankMax
// members, which are placed in LDS by a block scan of the per-thread member counts and ranked by
// counting on the full key; when every value bit is decided first, a block scan over the
// threads' contiguous index ranges settles the ties.
template <int PER>
__global__ __launch_bounds__(kCutThreads) void topk_cut_kernel(const float* __restrict__ act,
                                                               int F, int k,
                                                               unsigned long long* __restrict__ cut) {
  __shared__ uint32_t s_hist[kHistCopies * kBinsMax];
  __shared__ unsigned long long s_cand[kRankMax];
  __shared__ int s_w[kCutWaves];
  __shared__ int s_sel[3];
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const float* a = act + (size_t)b * F;
  const int i0 = tid * PER;

  uint32_t v[PER];  // bits of |a|: for non-negative floats the bit order is the value order
  bool ok[PER];
  if ((PER & 3) == 0 && (F & 3) == 0) {  // rows start 16-byte aligned: whole float4s
    const float4* a4 = reinterpret_cast<const float4*>(a + i0);
#pragma unroll
    for (int g = 0; g < PER / 4; ++g) {
      const float4 x = (i0 + 4 * g < F) ? a4[g] : make_float4(0.f, 0.f, 0.f, 0.f);
      v[4 * g] = __float_as_uint(fabsf(x.x));
      v[4 * g + 1] = __float_as_uint(fabsf(x.y));
      v[4 * g + 2] = __float_as_uint(fabsf(x.z));
      v[4 * g + 3] = __float_as_uint(fabsf(x.w));
    }
  } else {
#pragma unroll
    for (int j = 0; j < PER; ++j) v[j] = (i0 + j < F) ? __float_as_uint(fabsf(a[i0 + j])) : 0u;
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) ok[j] = i0 + j < F;

  // activations spread over many exponents: the digits start at bit 30 (bit 31, the sign of |a|,
  // is 0) without first settling common bits, which cost a block reduction and gained nothing
  uint32_t prefix = 0u, pmask = 0x80000000u;
  int kr = k;  // rank (1-based, descending) of the wanted key among those matching the prefix
  int hib = 30;  // highest bit still open
#pragma unroll 1
  for (int pass = 0; hib >= 0; ++pass) {
    const int bits = min(kDigitBitsMax, hib + 1), shift = hib + 1 - bits;
    int cnt;
    radix_digit_pass<PER>(v, ok, shift, bits, pass == 0 ? kHistCopies : 1, prefix, pmask, kr, &cnt,
                          s_hist, s_w, s_sel);
    hib = shift - 1;
    if (hib >= 0 && cnt <= kRankMax) {  // uniform: place the digit's members, rank them
      int nm = 0, tot;
#pragma unroll
      for (int j = 0; j < PER; ++j) nm += (ok[j] && (v[j] & pmask) == prefix) ? 1 : 0;
      int pos = block_inclusive_scan_1024(nm, s_w, &tot) - nm;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (ok[j] && (v[j] & pmask) == prefix)
          s_cand[pos++] = ((unsigned long long)v[j] << 32) | (unsigned)(~(unsigned)(i0 + j));
      __syncthreads();
      if (tid < cnt) {  // cnt <= kRankMax <= kCutThreads; the keys are distinct
        const unsigned long long mine = s_cand[tid];
        int r = 0;
        for (int q = 0; q < cnt; ++q) r += (s_cand[q] > mine) ? 1 : 0;
        if (r == kr - 1) cut[b] = mine;
      }
      return;
    }
  }
  // every value bit decided: prefix is the k-th largest |a|; the first kr neurons (by index)
  // equal to it are kept
  int eq = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) eq += (i0 + j < F && v[j] == prefix) ? 1 : 0;
  int tot;
  const int incl = block_inclusive_scan_1024(eq, s_w, &tot);
  const int before = incl - eq;
  if (before < kr && kr <= incl) {
    int m = kr - before, idx = i0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (i0 + j < F && v[j] == prefix) {
        if (m == 1) idx = i0 + j;
        --m;
      }
    }
    cut[b] = ((unsigned long long)prefix << 32) | (unsigned)(~(unsigned)idx);
  }
}

hipError_t launch_cut(const float* act, int B, int F, int k, unsigned long long* cut,
                      hipStream_t s) {
  const int per = ceil_div(F, kCutThreads);
#define SIRIUS_CUT(P)                                                        \
  if (per <= P) {                                                            \
    klaunch(topk_cut_kernel<P>, B, kCutThreads, 0, s, act, F, k, cut);            \
    return hipGetLastError();                                                \
  }
  SIRIUS_CUT(1)
  SIRIUS_CUT(2)
  SIRIUS_CUT(4)
  SIRIUS_CUT(8)
  SIRIUS_CUT(16)
  SIRIUS_CUT(32)
  SIRIUS_CUT(64)
#undef SIRIUS_CUT
  return hipErrorInvalidValue;  // d_ff above 65536
}

}  // namespace

TopkLayout topk_layout(int B, int d, int F) {
  TopkLayout L{};
  Carve c;
  L.act = c.take((size_t)B * F * sizeof(float));
  L.cut = c.take((size_t)B * sizeof(unsigned long long));
  L.ffn = c.take(B <= 1 ? decode1_layout(d, F).total
                        : (batch_path_ok(B, d, F) ? batch_layout(B, d, F, 3).total
                                                  : gemv_layout(B, d, F).total));
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_topk(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, int k, float norm_eps,
                           const float* resid, float* y, int32_t* active_idx, int32_t* active_cnt,
                           char* ws, const TopkLayout& L, hipStream_t stream) {
  if (B < 1 || k < 1 || k > F) return hipErrorInvalidValue;
  float* act = reinterpret_cast<float*>(ws + L.act);
  unsigned long long* cut = reinterpret_cast<unsigned long long*>(ws + L.cut);
  char* fws = ws + L.ffn;
  const bool batch = B >= 2 && batch_path_ok(B, d, F);
  const BatchLayout BL = batch ? batch_layout(B, d, F, 3) : BatchLayout{};
  hipError_t e = B == 1 ? launch_decode1_act(x, wg, d, F, norm_eps, act, stream)
                 : batch ? launch_batch_act(x, B, wg, d, F, norm_eps, act, fws, BL, stream)
                         : launch_gate_act(x, B, wg, d, F, norm_eps, act, stream);
  if (e != hipSuccess) return e;
  {
    ProfScope prof("topk_cut", stream);
    if ((e = launch_cut(act, B, F, k, cut, stream)) != hipSuccess) return e;
  }
  if (B == 1)
    return launch_ffn_decode1(x, wg, wu, wd, d, F, kFfnModeTopK, 0.f, norm_eps, resid, y,
                              active_idx, active_cnt, fws, decode1_layout(d, F), stream, act, cut);
  if (batch)  // one pass over the batch: the up and down rows of the tokens' union
    return launch_ffn_batch(x, B, wg, wu, wd, d, F, kFfnModeTopK, 0.f, norm_eps, resid, y,
                            active_idx, active_cnt, fws, BL, stream, act, cut);
  const GemvLayout G = gemv_layout(B, d, F);
  for (int b0 = 0; b0 < B; b0 += G.bc) {
    const int nb = std::min(G.bc, B - b0);
    e = launch_ffn_gemv(x + (size_t)b0 * d, nb, wg, wu, wd, d, F, kFfnModeTopK, 0.f, norm_eps,
                        resid ? resid + (size_t)b0 * d : nullptr, y + (size_t)b0 * d,
                        active_idx ? active_idx + (size_t)b0 * F : nullptr,
                        active_cnt ? active_cnt + b0 : nullptr, fws, G, stream,
                        act + (size_t)b0 * F, cut + b0);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sirius
