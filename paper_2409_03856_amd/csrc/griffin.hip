// Coarse-grained (prompt-fixed) neuron selection on gfx950 (Sec. 2.1; Appendix A.1).
//
//  griffin_z_kernel       z[t, i] = SiLU(x_t . W_gate[i]) * (x_t . W_up[i]) for the
//                         T prompt tokens: both products in one MFMA pass
//                         (v_mfma_f32_16x16x32_bf16, exact bf16 products, fp32
//                         accumulation). Workgroup tile 128 tokens x 128 neurons
//                         (eight waves), K staged through LDS in double-buffered
//                         32-wide slices (XOR-swizzled 64-byte rows), two slices in
//                         flight, two workgroups per CU;
//                         the token tiles of a neuron tile run on one XCD together so
//                         its weights are read from HBM once. For the plain statistic
//                         the epilogue writes only per-tile sums of z^2 (fp64); the
//                         normalised variant stores Z.
//  griffin_rownorm_kernel ||z_t||^2 per token (normalised variant only).
//  griffin_score_kernel   s_i = sqrt(sum_t z_ti^2 / ||z_t||^2) (normalised variant only).
//  griffin_tile_score_kernel  plain statistic: s_i = sqrt of the tile sums in order.
//  griffin_topk_kernel    one workgroup: the k-th largest score by a bitwise search and
//                         the k neurons of largest score (equal scores: lower index first)
//                         in ascending index order.
//  condense_kernel        copies the selected rows of the three matrices.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

constexpr int kGT = 128;           // tokens per workgroup tile
constexpr int kGN = 128;           // neurons per workgroup tile
constexpr int kGThreads = 512;     // eight waves: 2 (tokens) x 4 (neurons) wave tiles
constexpr int kGK = 32;            // K slice per LDS stage
constexpr int kLdsRow = kGK;       // LDS row (bf16 elements): 64 bytes, chunks XOR-swizzled
constexpr int kTopkThreads = 1024;
constexpr int kTopkPer = 64;       // scores per top-k thread at most: d_ff <= 65536

__device__ __forceinline__ int ceil_div_dev(int a, int b) { return (a + b - 1) / b; }

// Element offset of 16-byte chunk c (8 bf16) of LDS row r: chunk c sits at position
// c ^ ((r / 2) % 4) of the row's four, so the MFMA operand reads of 16 rows at one chunk and the
// staging writes of 16 rows x 4 chunks touch the banks evenly (a padded row pitch left 29M
// bank-conflict cycles per call in the hardware counters).
__device__ __forceinline__ int lds_at(int r, int c) { return r * kLdsRow + 8 * (c ^ ((r >> 1) & 3)); }

// 16-byte chunk (8 bf16) of row r at column k, zero outside the matrix.
__device__ __forceinline__ uint4 load_chunk(const uint16_t* base, int rows, int d, int r, int k) {
  if (r < rows && k < d) return *reinterpret_cast<const uint4*>(base + (size_t)r * d + k);
  return make_uint4(0u, 0u, 0u, 0u);
}

// Workgroup id -> (neuron tile, token tile). Workgroups are dispatched to the eight XCDs in
// turn (id % 8), and each XCD has its own L2: the token tiles of one neuron tile are given
// ids of one XCD that are dispatched together, so its weights come from HBM once and from
// that L2 for the other token tiles.
__device__ __forceinline__ void tile_of(int id, int ntn, int ntm, int* n_tile, int* m_tile) {
  const int full = (ntn / 8) * 8;  // neuron tiles placed eight at a time
  if (id < full * ntm) {
    const int xcd = id % 8, slot = id / 8;
    *m_tile = slot % ntm;
    *n_tile = xcd + 8 * (slot / ntm);
  } else {
    const int r = id - full * ntm;
    *n_tile = full + r / ntm;
    *m_tile = r % ntm;
  }
}

// Z tile (Z != nullptr) or, for the plain statistic, the tile's partial sums of z^2 over its
// tokens per neuron (part[m_tile][n], fp64) without storing Z. Tile kGT tokens x kGN neurons,
// eight waves in a 2 x 4 layout, each wave 64 tokens x 32 neurons of both products; K in
// slices of kGK staged through double-buffered LDS, each thread moving one 16-byte chunk of
// X, W_gate and W_up per slice. The global loads of slice s + 2 are issued while slice s is
// multiplied (two register sets), so each load has two slices of MFMA work to arrive in.
// Occupancy and loads in flight set its pace: at 128 VGPRs and 50 KiB of LDS two workgroups
// share a CU, so the 448 tiles of a 512-token prompt at d_ff = 14336 run in one round of the
// chip's 512 slots, with 96 KiB in flight per CU. (Four-wave 128 x 64 tiles: at two slices
// ahead three workgroups fit per CU and 128 of the 896 tiles run as a second, mostly empty
// round, about 225 us; at one slice ahead four fit, one round, about 183 us; this layout about
// 168 us.)
__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(4))) void griffin_z_kernel(const uint16_t* __restrict__ X, int T,
                                                        const uint16_t* __restrict__ Wg,
                                                        const uint16_t* __restrict__ Wu, int d,
                                                        int F, float* __restrict__ Z,
                                                        double* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) uint16_t sX[2][kGT * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sG[2][kGN * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sU[2][kGN * kLdsRow];
  __shared__ double s_part[2][kGN];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  int n_tile, m_tile;
  tile_of(blockIdx.x, ceil_div_dev(F, kGN), ceil_div_dev(T, kGT), &n_tile, &m_tile);
  const int t0 = m_tile * kGT, n0 = n_tile * kGN;
  const int wm = wave >> 2, wn = wave & 3;  // wave tile: 64 tokens x 32 neurons

  // global -> LDS per slice: X, W_gate and W_up 128 rows x 4 chunks of 16 bytes each, one chunk
  // of each per thread
  struct Stage {
    uint4 x, g, u;
  };
  auto gload = [&](int k0, Stage& st) {
    st.x = load_chunk(X, T, d, t0 + (tid >> 2), k0 + 8 * (tid & 3));
    st.g = load_chunk(Wg, F, d, n0 + (tid >> 2), k0 + 8 * (tid & 3));
    st.u = load_chunk(Wu, F, d, n0 + (tid >> 2), k0 + 8 * (tid & 3));
  };
  auto sstore = [&](const Stage& st, int buf) {
    *reinterpret_cast<uint4*>(&sX[buf][lds_at(tid >> 2, tid & 3)]) = st.x;
    *reinterpret_cast<uint4*>(&sG[buf][lds_at(tid >> 2, tid & 3)]) = st.g;
    *reinterpret_cast<uint4*>(&sU[buf][lds_at(tid >> 2, tid & 3)]) = st.u;
  };

  floatx4_t accg[4][2], accu[4][2];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      accg[mt][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
      accu[mt][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    }
  const int fr = lane & 15, fc = lane >> 4;  // fragment row and 16-byte chunk
  auto compute = [&](int buf) {
    bf16x8_t a[4], bg[2], bu[2];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
      a[mt] = *reinterpret_cast<const bf16x8_t*>(&sX[buf][lds_at(wm * 64 + mt * 16 + fr, fc)]);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      bg[nt] = *reinterpret_cast<const bf16x8_t*>(&sG[buf][lds_at(wn * 32 + nt * 16 + fr, fc)]);
      bu[nt] = *reinterpret_cast<const bf16x8_t*>(&sU[buf][lds_at(wn * 32 + nt * 16 + fr, fc)]);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        accg[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bg[nt], accg[mt][nt], 0, 0, 0);
        accu[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bu[nt], accu[mt][nt], 0, 0, 0);
      }
  };

  const int nk = (d + kGK - 1) / kGK;
  Stage s0, s1;  // register sets of slices 2j and 2j + 1
  gload(0, s0);
  if (nk > 1) gload(kGK, s1);
  sstore(s0, 0);
  __syncthreads();
  // slice ks: its loads went into set ks % 2; this set is reloaded with slice ks + 2 as soon
  // as it has been stored, and the other set (slice ks + 1) is stored after the MFMAs
  for (int ks = 0; ks < nk; ks += 2) {
    if (ks + 2 < nk) gload((ks + 2) * kGK, s0);
    compute(0);
    if (ks + 1 < nk) sstore(s1, 1);
    __syncthreads();
    if (ks + 1 < nk) {  // uniform over the block
      if (ks + 3 < nk) gload((ks + 3) * kGK, s1);
      compute(1);
      if (ks + 2 < nk) sstore(s0, 0);
      __syncthreads();
    }
  }

  // C layout: lane holds column (neuron) lane % 16 and rows (tokens) 4*(lane/16) + i.
  if (Z != nullptr) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int n = n0 + wn * 32 + nt * 16 + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + wm * 64 + mt * 16 + 4 * (lane >> 4) + i;
          if (t < T && n < F) Z[(size_t)t * F + n] = silu(accg[mt][nt][i]) * accu[mt][nt][i];
        }
      }
    return;
  }
  // sum of z^2 over this tile's tokens, per neuron, in a fixed order: the lane's 16 rows,
  // then the four lane groups, then the two token halves of the tile. Tokens past T have zero
  // inputs, so their z is 0.
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    double acc = 0.0;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double z = (double)(silu(accg[mt][nt][i]) * accu[mt][nt][i]);
        acc += z * z;
      }
    acc += __shfl_xor(acc, 16, kWave);
    acc += __shfl_xor(acc, 32, kWave);
    if (lane < 16) s_part[wm][wn * 32 + nt * 16 + lane] = acc;
  }
  __syncthreads();
  if (tid < kGN && n0 + tid < F) part[(size_t)m_tile * F + n0 + tid] = s_part[0][tid] + s_part[1][tid];
}

__global__ __launch_bounds__(256) void griffin_rownorm_kernel(const float* __restrict__ Z, int F,
                                                              float* __restrict__ rn2) {
  __shared__ double s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const float* zr = Z + (size_t)blockIdx.x * F;
  double s = 0.0;
  for (int i = tid; i < F; i += 256) s += (double)zr[i] * (double)zr[i];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, kWave);
  if (lane == 0) s_w[wave] = s;
  __syncthreads();
  if (tid == 0) rn2[blockIdx.x] = (float)(((s_w[0] + s_w[1]) + s_w[2]) + s_w[3]);
}

__global__ __launch_bounds__(256) void griffin_score_kernel(const float* __restrict__ Z, int T,
                                                            int F, const float* __restrict__ rn2,
                                                            float* __restrict__ scores) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= F) return;
  double s = 0.0;
  for (int t = 0; t < T; ++t) {
    const double z = (double)Z[(size_t)t * F + i];
    if (rn2 == nullptr) {
      s += z * z;
    } else {
      const double n2 = (double)rn2[t];
      if (n2 > 0.0) s += z * z / n2;
    }
  }
  scores[i] = (float)sqrt(s);
}

// Block-wide exclusive scan for 1024 threads (16 waves).
__device__ __forceinline__ int scan1024(int v, int* s_tmp, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += t;
  }
  if (lane == kWave - 1) s_tmp[wave] = incl;
  __syncthreads();
  int off = 0, tot = 0;
  for (int w = 0; w < 16; ++w) {
    if (w < wave) off += s_tmp[w];
    tot += s_tmp[w];
  }
  *total = tot;
  __syncthreads();
  return off + incl - v;
}

// s_i = sqrt(sum over the token tiles, in order, of the tile sums of z^2): the plain
// statistic, from the product kernel's partials (spread over many CUs: one CU cannot read
// the partials quickly enough on its own).
__global__ __launch_bounds__(256) void griffin_tile_score_kernel(const double* __restrict__ part,
                                                                 int ntm, int F,
                                                                 float* __restrict__ scores) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= F) return;
  double a = 0.0;
  for (int m = 0; m < ntm; ++m) a += part[(size_t)m * F + i];
  scores[i] = (float)sqrt(a);
}

// Block-wide sum over 1024 threads; s_tmp holds 16 ints and is written once per call, so
// consecutive calls alternate between two such arrays.
__device__ __forceinline__ int sum1024(int v, int* s_tmp) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  if (lane == 0) s_tmp[wave] = v;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += s_tmp[w];
  return tot;
}

// The k-th largest score and the ascending top-k list in one workgroup. Wave w owns
// neurons [w W, w W + W) (W = d_ff / 16 rounded up to 64) and its lane l the neurons
// w W + l + 64 j (coalesced loads), all in registers (J = W / 64 <= PER). The k-th largest is
// the largest bit pattern u with at least k scores at or above it (non-negative floats order
// like their bit patterns), built one bit at a time from the top with a block-wide count per
// bit. The list is then written in ascending order: per-wave totals give each wave's base,
// and inside a wave ballots over the lanes, slot j after slot j - 1. Equal scores at the
// k-th value are taken lowest index first.
template <int PER>
__global__ __launch_bounds__(kTopkThreads) void griffin_topk_kernel(const float* __restrict__ scores,
                                                                    int F, int k,
                                                                    int32_t* __restrict__ sel) {
  __shared__ int s_tmp[2][16];
  __shared__ int s_gt[16], s_eq[16], s_take[16];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int W = ((F + 15) / 16 + kWave - 1) / kWave * kWave;
  const int J = W / kWave;
  const int ib = wave * W + lane;  // neuron of slot j: ib + 64 j
  float v[PER];  // -1 marks slots past d_ff (scores are >= 0)
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = ib + kWave * j;
    v[j] = (j < J && i < F) ? scores[i] : -1.0f;
  }

  uint32_t prefix = 0u;
  for (int b = 30; b >= 0; --b) {
    const uint32_t cand = prefix | (1u << b);
    int c = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) c += (v[j] >= 0.0f && __float_as_uint(v[j]) >= cand) ? 1 : 0;
    if (sum1024(c, s_tmp[b & 1]) >= k) prefix = cand;  // uniform over the block
  }
  const float kth = __uint_as_float(prefix);

  // per-wave counts, then each wave's eq offset and take base
  int gt = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    gt += (v[j] > kth) ? 1 : 0;
    eq += (v[j] == kth) ? 1 : 0;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    gt += __shfl_xor(gt, m, kWave);
    eq += __shfl_xor(eq, m, kWave);
  }
  if (lane == 0) {
    s_gt[wave] = gt;
    s_eq[wave] = eq;
  }
  __syncthreads();
  int n_gt = 0, eq_before = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) {
    n_gt += s_gt[w];
    eq_before += (w < wave) ? s_eq[w] : 0;
  }
  const int need_eq = k - n_gt;  // equal scores taken, lowest index first
  if (lane == 0) s_take[wave] = gt + min(max(need_eq - eq_before, 0), eq);
  __syncthreads();
  int run = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) run += (w < wave) ? s_take[w] : 0;
  int eq_run = eq_before;
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (j < J) {  // uniform over the block
      const bool is_eq = v[j] == kth;
      const unsigned long long me = __ballot(is_eq);
      const int eq_rank = eq_run + __popcll(me & below);
      eq_run += __popcll(me);
      const bool take = v[j] > kth || (is_eq && eq_rank < need_eq);
      const unsigned long long mt = __ballot(take);
      const int pos = run + __popcll(mt & below);
      run += __popcll(mt);
      if (take && pos < k) sel[pos] = ib + kWave * j;
    }
  }
}

__global__ __launch_bounds__(256) void condense_kernel(const uint4* __restrict__ wg,
                                                       const uint4* __restrict__ wu,
                                                       const uint4* __restrict__ wd, int nch, int F,
                                                       const int32_t* __restrict__ sel,
                                                       uint4* __restrict__ wgc, uint4* __restrict__ wuc,
                                                       uint4* __restrict__ wdc) {
  const int j = blockIdx.x;
  const uint4* src = blockIdx.y == 0 ? wg : (blockIdx.y == 1 ? wu : wd);
  uint4* dst = blockIdx.y == 0 ? wgc : (blockIdx.y == 1 ? wuc : wdc);
  const int r = sel[j];
  if (r < 0 || r >= F) return;  // sel comes from device memory; never gather outside the matrix
  const size_t row = (size_t)r;
  for (int c = threadIdx.x; c < nch; c += 256) dst[(size_t)j * nch + c] = src[row * nch + c];
}

}  // namespace

GriffinLayout griffin_layout(int T, int d, int F) {
  (void)d;
  GriffinLayout L{};
  Carve c;
  L.z = c.take((size_t)T * F * sizeof(float));  // used by the normalised variant only
  L.rownorm = c.take((size_t)T * sizeof(float));
  L.part = c.take((size_t)ceil_div(T, kGT) * F * sizeof(double));
  L.scores = c.take((size_t)F * sizeof(float));
  L.total = c.off;
  return L;
}

hipError_t launch_griffin(const uint16_t* xp, int T, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, int d, int F, int k, int normalize, int32_t* sel,
                          float* scores_out, uint16_t* wgc, uint16_t* wuc, uint16_t* wdc, char* ws,
                          const GriffinLayout& L, hipStream_t stream) {
  if (F > kTopkThreads * kTopkPer) return hipErrorInvalidValue;
  float* Z = normalize ? reinterpret_cast<float*>(ws + L.z) : nullptr;
  float* rn2 = reinterpret_cast<float*>(ws + L.rownorm);
  double* part = reinterpret_cast<double*>(ws + L.part);
  float* scores = reinterpret_cast<float*>(ws + L.scores);
  const int ntn = ceil_div(F, kGN), ntm = ceil_div(T, kGT);
  hipError_t e;
  {
    ProfScope prof("griffin_z", stream);
    klaunch(griffin_z_kernel, ntn * ntm, kGThreads, 0, stream, xp, T, wg, wu, d, F, Z, part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  float* sc = scores_out != nullptr ? scores_out : scores;
  if (normalize) {  // the normalised variant needs every z of a token first
    {
      ProfScope prof("griffin_rownorm", stream);
      klaunch(griffin_rownorm_kernel, T, 256, 0, stream, Z, F, rn2);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    ProfScope prof("griffin_score", stream);
    klaunch(griffin_score_kernel, ceil_div(F, 256), 256, 0, stream, Z, T, F, rn2, sc);
  } else {
    ProfScope prof("griffin_score", stream);
    klaunch(griffin_tile_score_kernel, ceil_div(F, 256), 256, 0, stream, part, ntm, F, sc);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  {
    ProfScope prof("griffin_topk", stream);
    const int per = ceil_div(ceil_div(F, 16), kWave);  // slots per lane
    if (per <= 16)
      klaunch(griffin_topk_kernel<16>, 1, kTopkThreads, 0, stream, sc, F, k, sel);
    else if (per <= 32)
      klaunch(griffin_topk_kernel<32>, 1, kTopkThreads, 0, stream, sc, F, k, sel);
    else
      klaunch(griffin_topk_kernel<64>, 1, kTopkThreads, 0, stream, sc, F, k, sel);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  ProfScope prof("condense", stream);
  klaunch(condense_kernel, dim3(k, 3), 256, 0, stream, 
      reinterpret_cast<const uint4*>(wg), reinterpret_cast<const uint4*>(wu),
      reinterpret_cast<const uint4*>(wd), d / 8, F, sel, reinterpret_cast<uint4*>(wgc),
      reinterpret_cast<uint4*>(wuc), reinterpret_cast<uint4*>(wdc));
  return hipGetLastError();
}

}  // namespace sirius
