// Coarse-grained (prompt-fixed) neuron selection on gfx950 (Sec. 2.1; Appendix A.1).
//
//  griffin_z_kernel       z[t, i] = SiLU(x_t . W_gate[i]) * (x_t . W_up[i]) for the
//                         T prompt tokens: both products in one MFMA pass
//                         (v_mfma_f32_16x16x32_bf16, exact bf16 products, fp32
//                         accumulation). Workgroup tile 256 tokens x 112 neurons (eight
//                         waves of 64 x 56, two per SIMD, one workgroup per CU: the 256
//                         tiles of a 512-token prompt at d_ff = 14336 fill the chip once),
//                         K through a five-slot LDS ring of 32-wide stages filled by direct
//                         global-to-LDS loads, the next stage's operands read while the
//                         current one is multiplied; the token tiles of a neuron tile run on
//                         one XCD together so its weights are read from HBM once. For the
//                         plain statistic the epilogue writes only per-tile sums of z^2
//                         (fp64); the normalised variant stores Z.
//  griffin_rownorm_kernel ||z_t||^2 per token (normalised variant only).
//  griffin_score_kernel   s_i = sqrt(sum_t z_ti^2 / ||z_t||^2) (normalised variant only).
//  griffin_tile_score_kernel  plain statistic: s_i = sqrt of the tile sums in order.
//  griffin_topk_kernel    one workgroup: the k-th largest score by a radix select (the bits
//                         every score shares, then digits of at most 11 bits below them,
//                         radix_select.h) and the k neurons of largest
//                         score (equal scores: lower index first) in ascending index order.
//  condense_kernel        copies the selected rows of the three matrices.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "radix_select.h"
#include "ring.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

constexpr int kTopkThreads = 1024;
constexpr int kTopkPer = 64;       // scores per top-k thread at most: d_ff <= 65536

// griffin_z tile: 256 tokens x 112 neurons, both products (224 output columns), eight waves of
// 64 tokens x 56 neurons each (4 x 2), one workgroup (two waves per SIMD) per CU.
constexpr int kZT = 256;                  // tokens per workgroup tile
constexpr int kZN = 112;                  // neurons per workgroup tile
constexpr int kZWT = 64;                  // tokens per wave
constexpr int kZWB = 7;                   // column blocks per wave: 7 x (8 gate + 8 up columns)
constexpr int kZMB = kZWT / 16;           // 16-token blocks per wave
constexpr int kZThreads = 512;
constexpr int kZK = 32;                   // K per ring stage: one 64-byte LDS row per token or weight row
constexpr int kZRowsW = 2 * kZN;          // 224 weight rows per stage (gate and up, interleaved by 8)
constexpr int kZRows = kZT + kZRowsW;     // 480 rows per stage
constexpr int kZSlotBytes = kZRows * 64;  // 30 KiB per stage
constexpr int kZSlots = 5;                // ring depth: four stages in flight while one is multiplied
constexpr int kZPieces = kZRows * 4;      // 16-byte pieces per stage: 1920
// direct loads per thread per stage: pieces q * 512 + tid for q = 0..3; the fourth exists for
// the first 384 threads only (waves 0..5), so the per-wave load count is 4 or 3 (wave-uniform)
constexpr int kZLoads = (kZPieces + kZThreads - 1) / kZThreads;
constexpr int kZFullWaves = (kZPieces - (kZLoads - 1) * kZThreads) / kWave;
static_assert(kZLoads == 4 && kZFullWaves == 6, "the ring's wait counts assume four or three loads per thread");
static_assert(kZSlots * kZSlotBytes <= 160 * 1024, "the ring fits in LDS");
static_assert(kZSlots <= 5, "wait_later counts at most four later stages");

__device__ __forceinline__ int ceil_div_dev(int a, int b) { return (a + b - 1) / b; }

// 16 zero bytes in global memory: the source of the K-tail chunks of griffin_z's direct loads
__device__ __align__(16) uint4 g_zero_chunk[1] = {{0u, 0u, 0u, 0u}};

// Position of 16-byte chunk c of LDS row r among the row's four: c ^ ((r / 2) % 4). An MFMA operand
// read (16 consecutive rows x the four chunks, one 16-byte chunk per lane) then touches the banks
// evenly; a padded row pitch left 29M bank-conflict cycles per call in the hardware counters. The
// map is its own inverse, so a direct load writing position p fetches chunk p ^ ((r / 2) % 4).
__device__ __forceinline__ int z_pos(int r, int c) { return c ^ ((r >> 1) & 3); }

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

// SiLU of a gate product in griffin_z's epilogue: exp through v_exp_f32 and a v_rcp_f32
// reciprocal (each within about 1 ulp) instead of the range-reduced expf and IEEE division
__device__ __forceinline__ float z_silu(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g * 1.4426950408889634f));
}

// Z tile (Z != nullptr) or, for the plain statistic, the tile's partial sums of z^2 over its
// tokens per neuron (part[m_tile][n], fp64) without storing Z.
//
// Tile kZT tokens x kZN neurons. The MFMAs take weight rows as the M side and tokens as the N
// side, and the weight rows of the tile alternate gate and up: row 2p of block j (16 rows) is
// the gate row of neuron n0 + 8j + p, row 2p + 1 its up row. A lane of a 16 x 16 result holds
// four consecutive rows of one token column, so it holds the gate and up products of two
// neurons side by side: every lane forms z from its own registers. Wave (wm, wn) multiplies
// weight blocks 7 wn .. + 6 by token rows 64 wm .. + 63: 7 x 4 v_mfma_f32_16x16x32_bf16 per K
// stage into 112 fp32 accumulators per lane. The two waves of a SIMD take turns on its MFMA
// unit.
//
// K goes through a five-slot LDS ring of 32-wide stages (30 KiB each) filled by direct
// global-to-LDS 16-byte loads (three or four per thread per stage, no staging registers): while
// stage b is multiplied, stages b + 2 .. b + 5 are in flight and the operands of stage b + 1 are
// read from LDS into a second register set, so the LDS reads of the next stage overlap this
// stage's MFMAs. One barrier per stage: after it, every wave has finished reading stage b (its
// register copy is complete) and every load of stage b + 1 has landed, so stage b's slot is
// refilled with stage b + 5.
//
// Rows past T or d_ff load a valid row (T - 1, d_ff - 1) whose products are never used; in a K
// tail (d_model % 32 != 0) the chunks past d_model are loaded from a block of zeros.
__global__ __launch_bounds__(kZThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void griffin_z_kernel(
    const uint16_t* __restrict__ X, int T, const uint16_t* __restrict__ Wg,
    const uint16_t* __restrict__ Wu, int d, int F, float* __restrict__ Z,
    double* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) unsigned char s_ring[kZSlots * kZSlotBytes];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  int n_tile, m_tile;
  tile_of(blockIdx.x, ceil_div_dev(F, kZN), ceil_div_dev(T, kZT), &n_tile, &m_tile);
  const int t0 = m_tile * kZT, n0 = n_tile * kZN;
  const int wm = wave >> 1, wn = wave & 1;  // token quarter, neuron half
  const int nblk = ceil_div_dev(d, kZK);

  // this thread's loads of a stage: slot piece g = q * 512 + tid, row g / 4, position g % 4,
  // holding chunk z_pos(row, position) of that row; a wave instruction covers 16 whole rows, so
  // the row kind (token or weight) is uniform over it
  const bool full_wave = wave < kZFullWaves;  // issues a fourth load per stage
  const uint16_t* src[kZLoads];
  int chunk_k[kZLoads];  // K offset of the chunk within a stage (elements)
  int lds_off[kZLoads];
#pragma unroll
  for (int q = 0; q < kZLoads; ++q) {
    const int g = min(q * kZThreads + tid, kZPieces - 1);  // past the last piece: never issued
    const int r = g >> 2, c = z_pos(r, g & 3);
    const uint16_t* row;
    if (r < kZT) {
      row = X + (size_t)min(t0 + r, T - 1) * d;
    } else {
      const int w = r - kZT;  // weight row: neuron w / 2 of the tile, gate (even) or up (odd)
      const int n = min(n0 + (w >> 1), F - 1);
      row = ((w & 1) ? Wu : Wg) + (size_t)n * d;
    }
    src[q] = row;
    chunk_k[q] = 8 * c;
    lds_off[q] = (q * kZThreads + wave * kWave) * 16;  // wave-uniform: lane l lands at + 16 l
  }
  auto issue = [&](unsigned char* slot, int b) {
    const int k0 = b * kZK;
    const bool tail = k0 + kZK > d;  // uniform: only the last stage of a K that is not a multiple of 32
#pragma unroll
    for (int q = 0; q < kZLoads; ++q) {
      if (q == kZLoads - 1 && !full_wave) break;  // wave-uniform
      const int k = k0 + chunk_k[q];
      // past d_model (the K tail) the chunk comes from a zero block, so those products vanish
      const void* gp = (tail && k >= d) ? static_cast<const void*>(g_zero_chunk) : static_cast<const void*>(src[q] + k);
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(slot + lds_off[q]));
      __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 0);
    }
  };
  // wait until at most `later` stages of this thread's loads are still in flight
  auto wait_later = [&](int later) {
    if (full_wave) {
      switch (later) {
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<kZLoads>(); break;
        case 2: wait_vm<2 * kZLoads>(); break;
        case 3: wait_vm<3 * kZLoads>(); break;
        default: wait_vm<4 * kZLoads>(); break;
      }
    } else {
      switch (later) {
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<kZLoads - 1>(); break;
        case 2: wait_vm<2 * (kZLoads - 1)>(); break;
        case 3: wait_vm<3 * (kZLoads - 1)>(); break;
        default: wait_vm<4 * (kZLoads - 1)>(); break;
      }
    }
  };

  // operand fragments of one stage: lane l reads row R0 + l % 16, chunk l / 16 of each 16-row block
  const int fr = lane & 15, fc = lane >> 4;
  struct Frag {
    bf16x8_t a[kZMB];  // token blocks
    bf16x8_t b[kZWB];  // weight blocks
  };
  auto read_frag = [&](const unsigned char* slot, Frag& f) {
#pragma unroll
    for (int mt = 0; mt < kZMB; ++mt) {
      const int r = wm * kZWT + 16 * mt + fr;
      f.a[mt] = *reinterpret_cast<const bf16x8_t*>(slot + r * 64 + 16 * z_pos(r, fc));
    }
#pragma unroll
    for (int nb = 0; nb < kZWB; ++nb) {
      const int r = kZT + 16 * (kZWB * wn + nb) + fr;
      f.b[nb] = *reinterpret_cast<const bf16x8_t*>(slot + r * 64 + 16 * z_pos(r, fc));
    }
  };

  floatx4_t acc[kZMB][kZWB];  // [token block][weight block]: rows = weights, columns = tokens
#pragma unroll
  for (int mt = 0; mt < kZMB; ++mt)
#pragma unroll
    for (int nb = 0; nb < kZWB; ++nb) acc[mt][nb] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  auto mfma = [&](const Frag& f) {
#pragma unroll
    for (int nb = 0; nb < kZWB; ++nb)
#pragma unroll
      for (int mt = 0; mt < kZMB; ++mt)
        acc[mt][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.b[nb], f.a[mt], acc[mt][nb], 0, 0, 0);
  };

  // iteration b: fragments of stage b are in `cur`, stage b lives in slot b % kZSlots. Wait for
  // this thread's loads of stage b + 1 (the loads of stages b + 2 .. b + kZSlots - 1 stay in
  // flight), barrier, refill the slot of stage b with stage b + kZSlots, then multiply stage b
  // while reading stage b + 1 into `nxt`. (Past the last stage the read of `nxt` takes a slot
  // whose values go unused: no branch separates these reads from the MFMAs, so they stay in
  // flight while the MFMAs issue.)
  int slot_b = 0;  // slot of stage b
  auto next_slot = [](int sl) { return sl + 1 == kZSlots ? 0 : sl + 1; };
  auto step = [&](Frag& cur, Frag& nxt, int b) {
    if (b + 1 < nblk) wait_later(min(kZSlots - 2, nblk - 2 - b));
    ring_barrier();
    const int slot_n = next_slot(slot_b);
    if (b + kZSlots < nblk) issue(s_ring + slot_b * kZSlotBytes, b + kZSlots);
    read_frag(s_ring + slot_n * kZSlotBytes, nxt);
    mfma(cur);
    slot_b = slot_n;
  };
  for (int p = 0; p < kZSlots; ++p)
    if (p < nblk) issue(s_ring + p * kZSlotBytes, p);  // uniform
  wait_later(min(kZSlots - 1, nblk - 1));  // stage 0 landed
  ring_barrier();
  Frag f0, f1;
  read_frag(s_ring, f0);
  int b = 0;
  for (; b + 1 < nblk; b += 2) {
    step(f0, f1, b);
    step(f1, f0, b + 1);
  }
  if (b < nblk) step(f0, f1, b);

  // C layout of a 16 x 16 block: lane l holds token column l % 16 and weight rows 4 (l / 16) + i,
  // i = 0..3: the gate and up products of neurons 8 nb + 2 (l / 16) (i = 0, 1) and
  // 8 nb + 2 (l / 16) + 1 (i = 2, 3).
  const int tcol = lane & 15, grp = lane >> 4;
  if (Z != nullptr) {
#pragma unroll
    for (int nb = 0; nb < kZWB; ++nb) {
      const int n = n0 + 8 * (kZWB * wn + nb) + 2 * grp;
#pragma unroll
      for (int mt = 0; mt < kZMB; ++mt) {
        const int t = t0 + wm * kZWT + 16 * mt + tcol;
        const floatx4_t& c = acc[mt][nb];
        if (t < T && n < F) Z[(size_t)t * F + n] = z_silu(c[0]) * c[1];
        if (t < T && n + 1 < F) Z[(size_t)t * F + n + 1] = z_silu(c[2]) * c[3];
      }
    }
    return;
  }
  // sum of z^2 over this tile's tokens, per neuron, in a fixed order: the lane's 4 tokens, then
  // the 16 token columns (xor tree), then the four token quarters of the tile. Tokens past T
  // are left out.
  __syncthreads();  // every wave is done with the ring: its first slot holds the wave sums
  double* s_part = reinterpret_cast<double*>(s_ring);  // [token quarter][kZN]
#pragma unroll
  for (int nb = 0; nb < kZWB; ++nb) {
    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int mt = 0; mt < kZMB; ++mt) {
      const int t = t0 + wm * kZWT + 16 * mt + tcol;
      const floatx4_t& c = acc[mt][nb];
      const double z0 = (double)(z_silu(c[0]) * c[1]);
      const double z1 = (double)(z_silu(c[2]) * c[3]);
      if (t < T) {
        s0 += z0 * z0;
        s1 += z1 * z1;
      }
    }
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) {
      s0 += __shfl_xor(s0, m, kWave);
      s1 += __shfl_xor(s1, m, kWave);
    }
    if (tcol == 0) {
      const int nl = 8 * (kZWB * wn + nb) + 2 * grp;
      s_part[wm * kZN + nl] = s0;
      s_part[wm * kZN + nl + 1] = s1;
    }
  }
  __syncthreads();
  if (tid < kZN && n0 + tid < F)
    part[(size_t)m_tile * F + n0 + tid] =
        ((s_part[tid] + s_part[kZN + tid]) + s_part[2 * kZN + tid]) + s_part[3 * kZN + tid];
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

// The k-th largest score and the ascending top-k list in one workgroup. Wave w owns
// neurons [w W, w W + W) (W = d_ff / 16 rounded up to 64) and its lane l the neurons
// w W + l + 64 j (coalesced loads), all in registers (J = W / 64 <= PER). The k-th largest
// score comes from the radix select over the scores' bit patterns (non-negative floats order
// like their bit patterns; the bits every score shares first, then digits right below them);
// a 31-step bitwise search with a block-wide count per bit took 28 us at d_ff = 14336. The list
// is then written in ascending order: per-wave totals give each wave's base, and inside a wave
// ballots over the lanes, slot j after slot j - 1. Equal scores at the
// k-th value are taken lowest index first.
template <int PER>
__global__ __launch_bounds__(kTopkThreads) void griffin_topk_kernel(const float* __restrict__ scores,
                                                                    int F, int k,
                                                                    int32_t* __restrict__ sel) {
  __shared__ uint32_t s_hist[kHistCopies * kBinsMax];
  __shared__ int s_w[2 * kSelWaves], s_sel[3];
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

  // the k-th largest score: three digit passes of the radix select settle every value bit
  uint32_t u[PER];
  bool ok[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    ok[j] = v[j] >= 0.0f;
    u[j] = __float_as_uint(v[j]);
  }
  uint32_t prefix, pmask;
  int kr = k, cnt;
  int hib = radix_common_bits<PER>(u, ok, prefix, pmask, s_w);  // highest bit still open
#pragma unroll 1
  for (int pass = 0; hib >= 0; ++pass) {
    const int bits = min(kDigitBitsMax, hib + 1), shift = hib + 1 - bits;
    radix_digit_pass<PER>(u, ok, shift, bits, pass == 0 ? kHistCopies : 1, prefix, pmask, kr,
                          &cnt, s_hist, s_w, s_sel);
    hib = shift - 1;
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
  L.part = c.take((size_t)ceil_div(T, kZT) * F * sizeof(double));
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
  const int ntn = ceil_div(F, kZN), ntm = ceil_div(T, kZT);
  hipError_t e;
  {
    ProfScope prof("griffin_z", stream);
    klaunch(griffin_z_kernel, ntn * ntm, kZThreads, 0, stream, xp, T, wg, wu, d, F, Z, part);
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
