// Multi-token SwiGLU FFN on MFMA (gfx950) for 2..64 tokens with d_model % 256 == 0: dense and
// condensed decode of small batches, the full model's parallel pass over a drafted chunk or tree,
// and per-token threshold (CATS) and top-k sparsity of batched tokens. The weights are streamed
// once per call whatever the batch (up to four 16-token MFMA tiles share every weight byte), so
// the call stays HBM-bound: at 16 tokens the products are 2 flops per weight byte per token,
// far below the bf16 MFMA ridge (about 300).
//
//  prep_pieces_kernel  x -> optional RMSNorm -> PX bf16 pieces, zero-padded to whole 16-token
//                      tiles. PX = 1: x rounded to bf16 (the full model's pass, as before).
//                      PX = 3: x = hi + mid + lo exactly (each piece the bf16 rounding of what
//                      the previous ones leave), so the MFMA products of the three pieces sum to
//                      the fp32 product: the threshold, top-k and small-batch paths keep fp32
//                      inputs.
//  gu_ring_kernel      dense: H = SiLU(X W_gate^T) * (X W_up^T) for one segment of at most 56
//                      neurons per workgroup; gate rows, up rows and the x pieces of every
//                      token tile move into an LDS ring by direct global-to-LDS loads, two to
//                      four K blocks in flight; wave (tile, product) multiplies with
//                      v_mfma_f32_16x16x32_bf16.
//  gu_unit_kernel      the same for 8..16 tokens with d_model a multiple of 2048: the weights
//                      move through LDS in units of 16 rows x 2048 columns, each row's 4 KiB
//                      requested by one wave with consecutive 1 KiB direct loads (the order in
//                      which HBM streams a row fastest), x held in registers.
//  cats_unit_kernel    the same modes as cats_ring_kernel for at most 4 tokens with d_model a
//                      multiple of 2048 on the unit layout: the three pieces of the four tokens
//                      are the 12 rows of one MFMA operand tile, held in registers.
//  cats_ring_kernel    per-token sparsity over one segment: the gate rows alone through the ring
//                      (threshold mode and the top-k gate pass), SiLU, the per-token keep
//                      decision (|a| > t, or the top-k key against the token's cut), the union of
//                      the tokens' kept neurons compacted in ascending order with a wave ballot,
//                      then the up rows of that union only through the ring; h = a u where the
//                      token keeps the neuron, 0 elsewhere, stored per segment position. Up rows
//                      outside the union are never read. Dense and condensed calls of fewer than
//                      8 tokens run here too, every neuron kept, so that a threshold below 0
//                      gives the dense result bit for bit.
//  down_ring_kernel    Y_partial over one 256-column tile and one range of 64-position blocks of
//                      the segment layout: a segment's rows (dense) or its union rows (gathered
//                      by index), so W_down rows outside the union are never read.
//                      The W_down rows of a block and the hi/lo h fragments move into an LDS
//                      ring by direct loads.
//  reduce_kernel       (ffn_gemv.hip) y = resid + the partials in a fixed order; the per-token
//                      ascending kept lists from the per-segment lists.
//
// Every sum has a fixed order and no kernel uses atomics: results are bitwise reproducible.
#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "ring.h"
#include "topk.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

constexpr int kBT = 512;                 // threads per workgroup: eight waves
constexpr int kSegN = 56;                // neurons per segment at most
constexpr int kSegPad = 64;              // segment positions (whole 16-neuron tiles, one down block)
constexpr int kLdsRing = 150 * 1024;     // LDS the rings may take
constexpr int kDnCols = 256;             // output columns per down workgroup
constexpr int kDnBlock = 64;             // rows per down block

// 16 zero bytes in global memory: the source of direct loads past d_model (a K tail)
__device__ __align__(16) uint4 g_zero16[1] = {{0u, 0u, 0u, 0u}};

__device__ __forceinline__ int swz(int r, int c) { return c ^ (r & 7); }

// vmcnt wait until at most `later` blocks of L loads each are still in flight (later <= 10)
template <int L>
__device__ __forceinline__ void wait_later(int later) {
  switch (later) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<L>(); break;
    case 2: wait_vm<(2 * L > 63 ? 63 : 2 * L)>(); break;
    case 3: wait_vm<(3 * L > 63 ? 63 : 3 * L)>(); break;
    case 4: wait_vm<(4 * L > 63 ? 63 : 4 * L)>(); break;
    case 5: wait_vm<(5 * L > 63 ? 63 : 5 * L)>(); break;
    case 6: wait_vm<(6 * L > 63 ? 63 : 6 * L)>(); break;
    case 7: wait_vm<(7 * L > 63 ? 63 : 7 * L)>(); break;
    case 8: wait_vm<(8 * L > 63 ? 63 : 8 * L)>(); break;
    case 9: wait_vm<(9 * L > 63 ? 63 : 9 * L)>(); break;
    default: wait_vm<(10 * L > 63 ? 63 : 10 * L)>(); break;
  }
}

// Geometry of an LDS ring (compile-time): ROWS rows of KS bf16 per slot (KS * 2 bytes), as many
// slots (at most 12) as fit in LDS bytes. Slots hold only rows that carry data (the real tokens
// of a batch rounded up to a token class, not a whole 16-token tile), so small batches get deep
// rings and many weight bytes in flight.
template <int ROWS, int KS, int LDS>
struct RingGeom {
  static constexpr int kRowBytes = KS * 2;
  static constexpr int kCpr = kRowBytes / 16;   // 16-byte chunks per row
  static constexpr int kRowQuant = kWave / kCpr; // rows per wave instruction
  static constexpr int kRows = (ROWS + kRowQuant - 1) / kRowQuant * kRowQuant;
  static constexpr int kSlotBytes = kRows * kRowBytes;
  static constexpr int kPieces = kRows * kCpr;
  static constexpr int kLoads = (kPieces + kBT - 1) / kBT;
  static constexpr int kFullWaves = (kPieces - (kLoads - 1) * kBT) / kWave;
  static constexpr int slots_for() {
    int s = LDS / kSlotBytes;
    if (s > 12) s = 12;
    while (s > 2 && (s - 2) * kLoads > 63) --s;  // vmcnt range of the waits
    return s;
  }
  static constexpr int kSlots = slots_for();
  static_assert(kSlots >= 3, "at least two blocks in flight");
  static_assert(kLoads <= 8, "loads per thread");
};

// LDS ring filled by 16-byte direct global-to-LDS loads from kBT threads. A wave instruction
// writes 64 consecutive 16-byte pieces, i.e. kRowQuant whole rows, so a lane fetches the chunk
// that its piece holds under the swizzle c ^ (r & 7); the 16-row MFMA operand reads of one chunk
// are then spread over the banks. Piece q * kBT + tid is load q of thread tid; the last load
// exists for the first kFullWaves waves only, so every wave knows its own count and the ring
// waits on exact vmcnt values. Row pointers come from row_of(r); nullptr marks a row of zeros
// (rows past the data), whose pieces all come from one 16-byte zero block in the cache.
template <class G>
struct Ring {
  const uint16_t* src[G::kLoads];
  int kofs[G::kLoads];
  int lds[G::kLoads];
  bool full;  // wave-uniform: this wave issues the last load
  template <class RowOf>
  __device__ __forceinline__ Ring(int tid, int wave, RowOf row_of) {
    full = wave < G::kFullWaves;
#pragma unroll
    for (int q = 0; q < G::kLoads; ++q) {
      const int gp = min(q * kBT + tid, G::kPieces - 1);  // past the last piece: never issued
      const int r = gp / G::kCpr, c = swz(r, gp % G::kCpr);
      src[q] = row_of(r);
      kofs[q] = 8 * c;
      lds[q] = (q * kBT + wave * kWave) * 16;  // wave-uniform: lane l lands at + 16 l
    }
  }
  // w_rows: the slot's first rows hold weights (read once: non-temporal loads)
  __device__ __forceinline__ void issue(unsigned char* slot, int blk, int d, int w_rows) {
    const int k0 = blk * (G::kRowBytes / 2);
    const bool tail = k0 + G::kRowBytes / 2 > d;  // uniform
    const int w_pieces = w_rows * G::kCpr;
    const int wbase = __builtin_amdgcn_readfirstlane(threadIdx.x & ~(kWave - 1));
#pragma unroll
    for (int q = 0; q < G::kLoads; ++q) {
      if (q == G::kLoads - 1 && !full) break;  // wave-uniform
      const int k = k0 + kofs[q];
      const void* gp = (src[q] == nullptr || (tail && k >= d)) ? static_cast<const void*>(g_zero16)
                                                                : static_cast<const void*>(src[q] + k);
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(slot + lds[q]));
      if (q * kBT + wbase < w_pieces)
        __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 2);
      else
        __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 0);
    }
  }
  // at most `later` blocks of this wave's loads still in flight
  __device__ __forceinline__ void wait(int later) {
    if (full) wait_later<G::kLoads>(later);
    else wait_later<G::kLoads - 1>(later);
  }
};

// Runs the ring over nblk K blocks: compute(slot) for each block in order, with the kSlots - 1
// blocks after it in flight. Block b: wait for it, barrier (every wave is done reading block
// b - 1, whose slot is refilled with block b + kSlots - 1), compute.
template <class G, class R, class Compute>
__device__ __forceinline__ void run_ring(unsigned char* ring, R& rg, int nblk, int d, int w_rows,
                                         Compute compute) {
  constexpr int S = G::kSlots, SB = G::kSlotBytes;
  static_assert(S - 2 <= 10, "wait_l covers ten later blocks");
#pragma unroll
  for (int p = 0; p < S - 1; ++p)
    if (p < nblk) rg.issue(ring + p * SB, p, d, w_rows);
  int slot = 0, refill = S - 1;
  for (int b = 0; b < nblk; ++b) {
    rg.wait(min(S - 2, nblk - 1 - b));
    ring_barrier();
    if (b + S - 1 < nblk) rg.issue(ring + refill * SB, b + S - 1, d, w_rows);
    compute(ring + slot * SB);
    slot = slot + 1 == S ? 0 : slot + 1;
    refill = refill + 1 == S ? 0 : refill + 1;
  }
}

// ---- x -> optional RMSNorm -> PX bf16 pieces [PX][Mpad][d]; one workgroup per padded row.
template <int PX>
__global__ __launch_bounds__(256) void prep_pieces_kernel(const float* __restrict__ x, int B, int d,
                                                          int mpad, float norm_eps,
                                                          uint16_t* __restrict__ xp) {
  constexpr int kPer = 8;  // d_model <= 8192: 2048 float4 per row over 256 threads
  __shared__ float s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int m = blockIdx.x;
  const int nv4 = d >> 2;
  if (m >= B) {  // uniform over the block: padded rows are zero in every piece
#pragma unroll
    for (int p = 0; p < PX; ++p) {
      uint2* out = reinterpret_cast<uint2*>(xp + ((size_t)p * mpad + m) * d);
      for (int i = tid; i < nv4; i += 256) out[i] = make_uint2(0u, 0u);
    }
    return;
  }
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)m * d);
  float4 v[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    v[u] = (i < nv4) ? xr[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (norm_eps >= 0.f) {
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      ss = fmaf(v[u].x, v[u].x, ss);
      ss = fmaf(v[u].y, v[u].y, ss);
      ss = fmaf(v[u].z, v[u].z, ss);
      ss = fmaf(v[u].w, v[u].w, ss);
    }
    ss = wave_sum(ss);
    if (lane == 0) s_w[wave] = ss;
    __syncthreads();
    const float tot = ((s_w[0] + s_w[1]) + s_w[2]) + s_w[3];
    const float inv = 1.0f / sqrtf(tot / (float)d + norm_eps);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      v[u].x *= inv;
      v[u].y *= inv;
      v[u].z *= inv;
      v[u].w *= inv;
    }
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    if (i >= nv4) continue;
    float r[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
    for (int p = 0; p < PX; ++p) {
      uint32_t b[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        b[e] = f32_to_bf16(r[e]);
        r[e] -= __uint_as_float(b[e] << 16);  // exact: the remainder of a bf16 rounding
      }
      reinterpret_cast<uint2*>(xp + ((size_t)p * mpad + m) * d)[i] =
          make_uint2(b[0] | (b[1] << 16), b[2] | (b[3] << 16));
    }
  }
}

// Segment geometry: nseg segments of np neurons over n_rows rows, np a multiple of 4 of at most
// 56, small enough that there are at least 256 segments (one workgroup per CU) when n_rows allows.
struct Seg {
  int nseg, np;
};
constexpr int kSegTarget = 256;
__host__ __device__ inline Seg seg_of(int n_rows) {
  int np = (n_rows + kSegTarget - 1) / kSegTarget;
  np = (np + 3) & ~3;
  if (np > kSegN) np = kSegN;
  if (np < 4) np = 4;
  return Seg{(n_rows + np - 1) / np, np};
}

// h = SiLU(g) u as a bf16 pair (hi, lo): hi = bf16(h), lo = bf16(h - hi)
__device__ __forceinline__ void store_h(uint16_t* hhi, uint16_t* hlo, size_t at, float h) {
  const uint32_t hi = f32_to_bf16(h);
  const float lo = h - __uint_as_float(hi << 16);
  hhi[at] = (uint16_t)hi;
  hlo[at] = (uint16_t)f32_to_bf16(lo);
}

// h positions [npos, hs) of every token row lie past the last segment but inside the last down
// block; the last workgroup of a gate/up launch writes zeros there (hs - npos < 64)
__device__ __forceinline__ void zero_h_tail(uint16_t* hhi, uint16_t* hlo, int hs, int npos,
                                            int mpad) {
  const int tail = hs - npos;
  for (int i = threadIdx.x; i < mpad * tail; i += blockDim.x) {
    const size_t at = (size_t)(i / tail) * hs + npos + i % tail;
    hhi[at] = 0;
    hlo[at] = 0;
  }
}

// Token classes: a batch of B tokens occupies TB slot rows per input piece (B rounded up to 4, 8,
// 16, 32, 48 or 64); rows past B load zeros. MFMA tiles are 16 tokens: MT = ceil(TB / 16).
__host__ __device__ inline int token_class(int B) {
  return B <= 4 ? 4 : (B <= 8 ? 8 : (B <= 16 ? 16 : (B <= 32 ? 32 : (B <= 48 ? 48 : 64))));
}
// K per ring block: 128 (256-byte rows) when three slots fit in the LDS budget, else 64
constexpr int ks_for(int rows, int lds) { return rows * 256 * 3 <= lds ? 128 : 64; }
// LDS for the rings of the gate/up kernels (dynamic), next to their own static arrays
constexpr int kGuLds = 144 * 1024;
constexpr int kCatsLds = 124 * 1024;

// NPM: neurons per segment at most (kSegN, or kSegSmall for short segments, whose smaller slots
// leave room for a deeper ring)
constexpr int kSegSmall = 32;
template <int TB, int NPM>
struct GuGeom {
  static constexpr int kRowsData = 2 * NPM + TB;
  using G = RingGeom<kRowsData, ks_for(kRowsData, kGuLds), kGuLds>;
};
template <int TB, int NPM>
struct CatsGeom {
  static constexpr int kRowsData = NPM + 3 * TB;
  using G = RingGeom<kRowsData, ks_for(kRowsData, kCatsLds), kCatsLds>;
};
template <int TB, int NPM>
struct AllGeom {
  static constexpr int kRowsData = 2 * NPM + 3 * TB;
  using G = RingGeom<kRowsData, ks_for(kRowsData, kCatsLds), kCatsLds>;
};

// ---- dense gate/up on the bf16-rounded input: one workgroup per segment of np neurons over
// F16 rows (rows past d_ff give h = 0). Slot rows: gate rows [0, np), up rows [np, 2 np), then
// TB token rows (zeros past B). Wave w: 16-neuron tile w / 2 of the gate (w even) or up (w odd)
// rows; its A operand for tile mt reads token row min(16 mt + r, TB - 1), so a tile's padding
// tokens (never stored) repeat a loaded row instead of occupying slot rows.
template <int TB, int NPM>
__global__ __launch_bounds__(kBT) void gu_ring_kernel(const uint16_t* __restrict__ xp, int B,
                                                      const uint16_t* __restrict__ wg,
                                                      const uint16_t* __restrict__ wu, int d,
                                                      int F, int hs, int np, int sp,
                                                      uint16_t* __restrict__ hhi,
                                                      uint16_t* __restrict__ hlo) {
  using G = typename GuGeom<TB, NPM>::G;
  constexpr int MT = (TB + 15) / 16, KS = G::kRowBytes / 2;
  extern __shared__ __attribute__((aligned(16))) unsigned char ring[];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int n0 = blockIdx.x * np;
  const int x0 = 2 * np;  // first token row of a slot
  const int nblk = (d + KS - 1) / KS;
  Ring<G> rg(tid, wave, [&](int r) -> const uint16_t* {
    if (r < x0) {
      const int j = r < np ? r : r - np;
      const int n = min(n0 + j, F - 1);  // rows past d_ff: a valid row, h = 0 there
      return (r < np ? wg : wu) + (size_t)n * d;
    }
    if (r < x0 + B) return xp + (size_t)(r - x0) * d;
    return nullptr;
  });

  const int tau = wave >> 1, mu = wave & 1;
  const bool active = 16 * tau < np;
  const int wrow = mu * np + 16 * tau + fr;  // B operand row (past np: never stored)
  floatx4_t acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  run_ring<G>(ring, rg, nblk, d, x0, [&](const unsigned char* slot) {
    if (!active) return;
    constexpr int kSteps = KS / 32;
    bf16x8_t bw[kSteps], ax[kSteps][MT];
#pragma unroll
    for (int i = 0; i < kSteps; ++i) {  // every operand of the block first, then the MFMAs
      const int c = 4 * i + grp;
      bw[i] = *reinterpret_cast<const bf16x8_t*>(slot + wrow * G::kRowBytes + 16 * swz(wrow, c));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int xr = x0 + min(16 * mt + fr, TB - 1);
        ax[i][mt] = *reinterpret_cast<const bf16x8_t*>(slot + xr * G::kRowBytes + 16 * swz(xr, c));
      }
    }
#pragma unroll
    for (int i = 0; i < kSteps; ++i)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ax[i][mt], bw[i], acc[mt], 0, 0, 0);
  });

  // epilogue: the up wave of each tile hands its sums to the gate wave through LDS
  __syncthreads();  // every wave is done with the ring
  floatx4_t* s_up = reinterpret_cast<floatx4_t*>(ring);  // [tile][mt][lane]
  if (active && mu == 1) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) s_up[(tau * MT + mt) * kWave + lane] = acc[mt];
  }
  __syncthreads();
  // h goes to the segment's positions [0, sp) (sp >= np, whole 16-neuron tiles): position j of
  // segment s holds neuron s np + j, and h = 0 at the positions past the segment's rows, past
  // d_ff and for the padding tokens, so the down pass can take whole 64-position blocks
  if (mu == 0 && 16 * tau < sp) {
    const int j = 16 * tau + fr, n = n0 + j;
    const bool real = active && j < np && n < F;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4_t u4 = active ? s_up[(tau * MT + mt) * kWave + lane] : floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * grp + r;
        // C layout: lane holds neuron fr and tokens 4 (lane / 16) + r
        store_h(hhi, hlo, (size_t)m * hs + (size_t)blockIdx.x * sp + j,
                (real && m < B) ? silu(acc[mt][r]) * u4[r] : 0.f);
      }
    }
  }
  if (blockIdx.x == gridDim.x - 1) zero_h_tail(hhi, hlo, hs, gridDim.x * sp, 16 * MT);
}

// ---- dense gate/up of 8..16 tokens on the bf16-rounded input with d_model a multiple of 2048.
// HBM streams a weight row fastest when its bytes are requested close together in time: one wave
// reading a row's aligned 4 KiB with consecutive 1 KiB loads moves about 6.8 TB/s over the chip,
// the same bytes requested 256 or 512 bytes per row per instruction, or spread over later
// instructions, 5.0-6.0. The ring kernel above requests each row 256 bytes per K block; this one
// moves the weights through LDS in units of 16 rows x 2048 columns, wave w requesting row w of
// the unit with four consecutive 1 KiB direct loads, two unit buffers (128.5 KiB of LDS).
// Segment rows: gate rows [0, np), up rows [np, 2 np), padded to whole 16-row tiles with zero
// rows; units go tile by tile with the K spans inner, so a row's spans are requested in
// consecutive units. Wave w multiplies K steps 4 w .. 4 w + 3 of every unit (x in registers for
// the whole call, the weights from LDS) into one partial per tile; the 16 partials are summed in
// wave order at the end, so the result does not depend on timing.
constexpr int kUnitThreads = 1024;                  // 16 waves: one row of a unit each
constexpr int kUnitWaves = kUnitThreads / kWave;
constexpr int kUnitK = 2048;                        // columns per unit (4 KiB of a row)
constexpr int kUnitRowBytes = kUnitK * 2 + 16;      // LDS row stride: the 16 rows of an MFMA
                                                    // operand read lie in distinct banks
constexpr int kUnitBytes = 16 * kUnitRowBytes;      // 65792
constexpr int kUnitLds = 2 * kUnitBytes;            // 131584
constexpr int kUnitTiles = (2 * kSegN + 15) / 16;   // 16-row tiles per segment at most (7)
constexpr int kUnitLoads = kUnitK * 2 / 1024;       // 1 KiB loads per wave per unit (4)
constexpr int kUnitSteps = kUnitK / 32 / kUnitWaves;  // 32-wide K steps per wave per unit (4)
static_assert(kUnitWaves * kUnitTiles * kWave * 16 + kUnitTiles * 16 * 16 * 4 <= kUnitLds,
              "the end-of-call reduction fits in the unit buffers");
__device__ __align__(16) uint16_t g_zero_row[kUnitK];  // source of the padding rows

// x operand (A) of this wave's K steps in every span: row fr of the tile from `row` (16 rows of
// d columns), zero where `ok` is false (the load is issued anyway, from row 0, so every wave's
// load count is the same)
template <int NSPAN>
__device__ __forceinline__ void unit_x(bf16x8_t (&xa)[NSPAN][kUnitSteps], const uint16_t* row,
                                       bool ok) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6, grp = lane >> 4;
#pragma unroll
  for (int s = 0; s < NSPAN; ++s)
#pragma unroll
    for (int j = 0; j < kUnitSteps; ++j) {
      uint4 v = *reinterpret_cast<const uint4*>(row + s * kUnitK + 32 * (kUnitSteps * wave + j) + 8 * grp);
      if (!ok) v = make_uint4(0u, 0u, 0u, 0u);
      xa[s][j] = as_bf16x8(v);
    }
}

// The unit pipeline: T (<= TMAX) tiles of 16 rows, row r of the sequence from row_of(r) (wave-
// uniform; nullptr: a zero row), units (tile u / NSPAN, span u % NSPAN) in two LDS buffers, wave w
// requesting row w of every unit; acc[t] = this wave's K steps of tile t. Then the waves'
// partials are summed in wave order into res[16 t + row][x row] (fp32, in LDS past the partials),
// and the unit buffers are free again. A row's result does not depend on its place in the
// sequence: the same loads, steps and sums give it wherever it sits.
template <int NSPAN, int TMAX, class RowOf>
__device__ __forceinline__ float* unit_pass(unsigned char* lds_u, int T, RowOf row_of,
                                            const bf16x8_t (&xa)[NSPAN][kUnitSteps]) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int U = T * NSPAN;
  auto issue = [&](int u) {
    const int t = u / NSPAN, sp_ = u - t * NSPAN;
    const uint16_t* row = row_of(__builtin_amdgcn_readfirstlane(16 * t + wave));  // wave-uniform
    const uint16_t* src = row != nullptr ? row + sp_ * kUnitK : g_zero_row;
    unsigned char* dst = lds_u + (u & 1) * kUnitBytes + wave * kUnitRowBytes;
#pragma unroll
    for (int q = 0; q < kUnitLoads; ++q) {
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(dst + q * 1024));  // lane l lands at + 16 l
      __builtin_amdgcn_global_load_lds(src + q * 512 + 8 * lane, lp, 16, 0, 2);
    }
  };
  floatx4_t acc[TMAX];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) acc[t] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  issue(0);
  if (U > 1) issue(1);
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    if (t >= T) break;  // uniform
#pragma unroll
    for (int s = 0; s < NSPAN; ++s) {
      const int u = t * NSPAN + s;
      // this wave's loads of unit u have landed (unit u + 1 still in flight), then every wave's
      if (u + 1 < U) wait_vm<kUnitLoads>();
      else wait_vm<0>();
      ring_barrier();
      const unsigned char* buf = lds_u + (u & 1) * kUnitBytes;
      bf16x8_t bw[kUnitSteps];  // B operand: weight row fr of the tile
#pragma unroll
      for (int j = 0; j < kUnitSteps; ++j)
        bw[j] = *reinterpret_cast<const bf16x8_t*>(
            buf + fr * kUnitRowBytes + 2 * (32 * (kUnitSteps * wave + j) + 8 * grp));
#pragma unroll
      for (int j = 0; j < kUnitSteps; ++j)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[s][j], bw[j], acc[t], 0, 0, 0);
      if (u + 2 < U) {
        ring_barrier();  // every wave is done reading buffer u & 1
        issue(u + 2);
      }
    }
  }
  // the waves' partials summed in wave order: red[w][t][lane], then res
  __syncthreads();
  floatx4_t* red = reinterpret_cast<floatx4_t*>(lds_u);
  float* res = reinterpret_cast<float*>(lds_u + kUnitWaves * TMAX * kWave * 16);
#pragma unroll
  for (int t = 0; t < TMAX; ++t)
    if (t < T) red[(wave * TMAX + t) * kWave + lane] = acc[t];
  __syncthreads();
  if (tid < T * kWave) {
    const int t = tid >> 6, l = tid & (kWave - 1);
    floatx4_t v = red[t * kWave + l];
#pragma unroll
    for (int w = 1; w < kUnitWaves; ++w) v += red[(w * TMAX + t) * kWave + l];
    // C layout: lane l holds weight row (l & 15) of the tile and x rows 4 (l >> 4) + e
#pragma unroll
    for (int e = 0; e < 4; ++e) res[(16 * t + (l & 15)) * 16 + 4 * (l >> 4) + e] = v[e];
  }
  __syncthreads();
  return res;
}

template <int NSPAN>  // d_model / 2048
__global__ __launch_bounds__(kUnitThreads) void gu_unit_kernel(
    const uint16_t* __restrict__ xp, int B, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int hs, int np, int sp,
    uint16_t* __restrict__ hhi, uint16_t* __restrict__ hlo) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_u[];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int n0 = blockIdx.x * np;
  // x operand: token rows (rows past B are zero in xp)
  bf16x8_t xa[NSPAN][kUnitSteps];
  unit_x<NSPAN>(xa, xp + (size_t)(lane & 15) * d, true);
  const float* res = unit_pass<NSPAN, kUnitTiles>(
      lds_u, (2 * np + 15) >> 4,
      [&](int r) -> const uint16_t* {
        return r < np       ? wg + (size_t)min(n0 + r, F - 1) * d
               : r < 2 * np ? wu + (size_t)min(n0 + r - np, F - 1) * d
                            : nullptr;
      },
      xa);
  // h at the segment's positions [0, sp), as the ring kernel writes it: neuron n0 + j, zero past
  // the segment's rows, past d_ff and for the padding tokens
  for (int i = tid; i < 16 * sp; i += kUnitThreads) {
    const int m = i / sp, j = i - m * sp;
    const bool real = j < np && n0 + j < F && m < B;
    store_h(hhi, hlo, (size_t)m * hs + (size_t)blockIdx.x * sp + j,
            real ? silu(res[j * 16 + m]) * res[(np + j) * 16 + m] : 0.f);
  }
  if (blockIdx.x == gridDim.x - 1) zero_h_tail(hhi, hlo, hs, gridDim.x * sp, 16);
}

// ---- per-token sparse gate/up of at most 4 tokens on the exact input (threshold, top-k gate pass,
// top-k keyed pass, every neuron kept), d_model a multiple of 2048, on the unit pipeline: the
// three bf16 pieces of the four tokens are the 12 rows of one MFMA operand tile (row 4 p + m), so
// the whole input stays in registers. Phase A streams the segment's gate rows, phase B the up rows
// of the tokens' union; keep decisions, lists and h as cats_ring_kernel forms them. A row's sum is
// its three pieces' sums added in piece order. With every neuron kept the gate and up rows go in
// one pass (each row's result is the same wherever it sits in the sequence), so a threshold below
// 0 still gives the dense result bit for bit.
constexpr int kCatsUnitTokens = 4;
constexpr int kCatsUnitTiles = (kSegN + 15) / 16;  // 16-row tiles of one phase (4)
constexpr int kModeThr = 0, kModeAct = 1, kModeKeyed = 2, kModeAll = 3;

__device__ __forceinline__ float piece_sum(const float* res, int row, int m) {
  return (res[row * 16 + m] + res[row * 16 + 4 + m]) + res[row * 16 + 8 + m];
}

template <int NSPAN, int MODE>
__global__ __launch_bounds__(kUnitThreads) void cats_unit_kernel(
    const uint16_t* __restrict__ xp, int B, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int np, float t, float* __restrict__ act,
    const unsigned long long* __restrict__ cut, uint16_t* __restrict__ hhi,
    uint16_t* __restrict__ hlo, int hs, int sp, int32_t* __restrict__ uidx,
    int32_t* __restrict__ ucnt, int32_t* __restrict__ bidx, int32_t* __restrict__ bcnt) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_u[];
  __shared__ float s_a[kCatsUnitTokens][kSegPad];         // a = SiLU(g) per token and position
  __shared__ unsigned long long s_keep[kCatsUnitTokens];  // kept positions per token
  __shared__ int s_u[kSegPad];                            // union positions, ascending
  __shared__ int s_nu;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int seg = blockIdx.x, nseg = gridDim.x;
  const int r0 = seg * np;
  const int nr = min(np, F - r0);  // neurons of this segment (>= 1)
  constexpr int kMpad = 16;        // rows of xp per piece and of h

  // x operand: row 4 p + m = piece p of token m (rows 12..15 and tokens past B: zero)
  bf16x8_t xa[NSPAN][kUnitSteps];
  {
    const int fr = lane & 15, pc = fr >> 2, m = fr & 3;
    const bool ok = fr < 12 && m < B;
    unit_x<NSPAN>(xa, xp + ((size_t)(ok ? pc : 0) * kMpad + (ok ? m : 0)) * d, ok);
  }

  if (MODE == kModeAll) {  // gate rows [0, np), up rows [np, 2 np) in one pass
    const float* res = unit_pass<NSPAN, kUnitTiles>(
        lds_u, (2 * np + 15) >> 4,
        [&](int r) -> const uint16_t* {
          return r < np       ? wg + (size_t)(r0 + min(r, nr - 1)) * d
                 : r < 2 * np ? wu + (size_t)(r0 + min(r - np, nr - 1)) * d
                              : nullptr;
        },
        xa);
    for (int i = tid; i < kMpad * sp; i += kUnitThreads) {
      const int m = i / sp, k = i - m * sp;
      const float h = (m < B && k < nr) ? silu(piece_sum(res, k, m)) * piece_sum(res, np + k, m) : 0.f;
      store_h(hhi, hlo, (size_t)m * hs + (size_t)seg * sp + k, h);
    }
    // the kept list of every neuron, as the threshold path writes it for t < 0
    if (tid < nr) uidx[seg * sp + tid] = r0 + tid;
    if (tid == 0) ucnt[seg] = nr;
    if (seg == nseg - 1) zero_h_tail(hhi, hlo, hs, nseg * sp, kMpad);
    return;
  }

  // ---- phase A: the gate (threshold mode and the top-k gate pass) or the stored activations
  if (MODE != kModeKeyed) {
    const float* res = unit_pass<NSPAN, kCatsUnitTiles>(
        lds_u, (np + 15) >> 4,
        [&](int r) -> const uint16_t* {
          return r < np ? wg + (size_t)(r0 + min(r, nr - 1)) * d : nullptr;
        },
        xa);
    for (int i = tid; i < kCatsUnitTokens * kSegPad; i += kUnitThreads) {
      const int m = i / kSegPad, j = i - m * kSegPad;
      if (j < np) {
        const float a = silu(piece_sum(res, j, m));
        if (MODE == kModeAct) {
          if (m < B && j < nr) act[(size_t)m * F + r0 + j] = a;
        } else {
          s_a[m][j] = a;
        }
      }
    }
    if (MODE == kModeAct) return;  // uniform
  } else {
    for (int i = tid; i < kCatsUnitTokens * kSegPad; i += kUnitThreads) {
      const int m = i / kSegPad, j = i - m * kSegPad;
      s_a[m][j] = (m < B && j < nr) ? act[(size_t)m * F + r0 + j] : 0.f;
    }
  }
  __syncthreads();

  // ---- keep decisions per token (a wave ballot over the segment's positions), per-token lists
  if (wave < kCatsUnitTokens) {
    const int m = wave;
    const float a = s_a[m][lane];
    bool keep = false;
    if (m < B && lane < nr) {
      if (MODE == kModeKeyed) keep = topk_key(a, r0 + lane) >= cut[m];
      else keep = fabsf(a) > t;
    }
    const unsigned long long mk = __ballot(keep);
    if (lane == 0) s_keep[m] = mk;
    if (m < B && bidx != nullptr) {
      if (keep) bidx[((size_t)m * nseg + seg) * kSegPad + __popcll(mk & ((1ull << lane) - 1ull))] = r0 + lane;
      if (lane == 0) bcnt[m * nseg + seg] = __popcll(mk);
    }
  }
  __syncthreads();
  // ---- union of the tokens' kept positions, ascending
  if (wave == 0) {
    unsigned long long un = 0ull;
    for (int m = 0; m < B && m < kCatsUnitTokens; ++m) un |= s_keep[m];
    const bool in = (un >> lane) & 1ull;
    const int pos = __popcll(un & ((1ull << lane) - 1ull));
    if (in) {
      s_u[pos] = lane;
      uidx[seg * sp + pos] = r0 + lane;
    }
    if (lane == 0) {
      s_nu = __popcll(un);
      ucnt[seg] = __popcll(un);
    }
  }
  __syncthreads();
  const int nu = s_nu;

  // ---- phase B: the up rows of the union only; h = a u where the token keeps the neuron
  const float* res = nullptr;
  if (nu > 0)  // uniform
    res = unit_pass<NSPAN, kCatsUnitTiles>(
        lds_u, (nu + 15) >> 4,
        [&](int k) -> const uint16_t* { return k < nu ? wu + (size_t)(r0 + s_u[k]) * d : nullptr; },
        xa);
  for (int i = tid; i < kMpad * sp; i += kUnitThreads) {
    const int m = i / sp, k = i - m * sp;
    float h = 0.f;
    if (m < B && k < nu) {
      const int j = s_u[k];
      if ((s_keep[m] >> j) & 1ull) h = s_a[m][j] * piece_sum(res, k, m);
    }
    store_h(hhi, hlo, (size_t)m * hs + (size_t)seg * sp + k, h);  // 0 past nu
  }
  if (seg == nseg - 1) zero_h_tail(hhi, hlo, hs, nseg * sp, kMpad);
}

// ---- every neuron kept (the dense and condensed FFN of small batches on the exact input) in one
// ring pass over the segment's gate rows [0, np), up rows [np, 2 np) and the token rows (piece p,
// token m) at 2 np + p TB + m. Wave w keeps the gate and up sums of 16-neuron tile w & 3 over the
// K steps of half w >> 2 of each block, in the order in which the two-phase segment kernel below
// forms them (same K blocks, steps, pieces and token tiles; the halves added in the same order),
// so its results are bitwise those of the threshold path with t < 0, with one pass over K instead
// of two.
template <int TB, int NPM>
__global__ __launch_bounds__(kBT) void all_ring_kernel(
    const uint16_t* __restrict__ xp, int B, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int np, uint16_t* __restrict__ hhi,
    uint16_t* __restrict__ hlo, int hs, int sp, int32_t* __restrict__ uidx,
    int32_t* __restrict__ ucnt) {
  using G = typename AllGeom<TB, NPM>::G;
  static_assert(G::kRowBytes == CatsGeom<TB, NPM>::G::kRowBytes,
                "the K blocks of the two-phase kernel, and so its sums");
  constexpr int MT = (TB + 15) / 16, KS = G::kRowBytes / 2;
  constexpr int kMpad = 16 * MT;
  extern __shared__ __attribute__((aligned(16))) unsigned char ring[];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int seg = blockIdx.x, nseg = gridDim.x;
  const int r0 = seg * np;
  const int nr = min(np, F - r0);  // neurons of this segment (>= 1)
  const int nblk = (d + KS - 1) / KS;
  const int tau = wave & 3, kap = wave >> 2;
  constexpr int kSteps = KS / 32;
  constexpr int kHalf = kSteps / 2;
  const int x0 = 2 * np;  // first token row of a slot

  Ring<G> rg(tid, wave, [&](int r) -> const uint16_t* {
    if (r < np) return wg + (size_t)(r0 + min(r, nr - 1)) * d;
    if (r < x0) return wu + (size_t)(r0 + min(r - np, nr - 1)) * d;
    if (r < x0 + 3 * TB) {
      const int p = (r - x0) / TB, m = (r - x0) % TB;
      return m < B ? xp + ((size_t)p * kMpad + m) * d : nullptr;
    }
    return nullptr;
  });
  floatx4_t accg[MT], accu[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    accg[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    accu[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }
  const int wrow = 16 * tau + fr;  // past np: never stored
  const bool active = 16 * tau < np;
  run_ring<G>(ring, rg, nblk, d, x0, [&](const unsigned char* slot) {
    if (!active) return;
    bf16x8_t bg[kHalf], bu[kHalf], ax[kHalf][3][MT];
#pragma unroll
    for (int i2 = 0; i2 < kHalf; ++i2) {
      const int c = 4 * (kap * kHalf + i2) + grp;
      bg[i2] = *reinterpret_cast<const bf16x8_t*>(slot + wrow * G::kRowBytes + 16 * swz(wrow, c));
      bu[i2] = *reinterpret_cast<const bf16x8_t*>(slot + (np + wrow) * G::kRowBytes + 16 * swz(np + wrow, c));
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int xr = x0 + p * TB + min(16 * mt + fr, TB - 1);
          ax[i2][p][mt] = *reinterpret_cast<const bf16x8_t*>(slot + xr * G::kRowBytes + 16 * swz(xr, c));
        }
    }
#pragma unroll
    for (int i2 = 0; i2 < kHalf; ++i2)
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          accg[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ax[i2][p][mt], bg[i2], accg[mt], 0, 0, 0);
          accu[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ax[i2][p][mt], bu[i2], accu[mt], 0, 0, 0);
        }
  });
  // the second K half hands its sums to the first through LDS
  __syncthreads();
  floatx4_t* s_h = reinterpret_cast<floatx4_t*>(ring);  // [gate 0..3 | up 4..7][mt][lane]
  if (kap == 1) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      s_h[(tau * MT + mt) * kWave + lane] = accg[mt];
      s_h[((4 + tau) * MT + mt) * kWave + lane] = accu[mt];
    }
  }
  __syncthreads();
  if (kap == 0) {
    const int k = 16 * tau + fr;  // position = neuron r0 + k
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4_t og = s_h[(tau * MT + mt) * kWave + lane];
      const floatx4_t ou = s_h[((4 + tau) * MT + mt) * kWave + lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        accg[mt][r] += og[r];
        accu[mt][r] += ou[r];
        const int m = 16 * mt + 4 * grp + r;  // C layout: neuron fr, tokens 4 (lane / 16) + r
        const float h = (k < nr && m < B) ? silu(accg[mt][r]) * accu[mt][r] : 0.f;
        if (k < sp) store_h(hhi, hlo, (size_t)m * hs + seg * sp + k, h);
      }
    }
  }
  // the kept list of every neuron, as the two-phase kernel writes it for t < 0
  if (tid < nr) uidx[seg * sp + tid] = r0 + tid;
  if (tid == 0) ucnt[seg] = nr;
  if (seg == nseg - 1) zero_h_tail(hhi, hlo, hs, nseg * sp, kMpad);
}

// ---- per-token sparse gate/up over one segment (threshold, top-k gate pass, top-k keyed pass,
// every neuron kept) on the exact input. Slot rows: the segment's gate (phase A) or union up
// (phase B) rows [0, np), then the token rows (piece p, token m) at np + p TB + m (zeros past B).
// Wave w: 16-neuron tile w & 3, K steps of half w >> 2 of each block; the halves are added in a
// fixed order. The A operand for piece p and tile mt reads token row min(16 mt + r, TB - 1).
// (The modes are those of cats_unit_kernel above. kModeAll keeps every neuron: the dense and
// condensed FFN of small batches on the exact input, through the same kernels, and so the same
// sums, as the threshold path with t < 0.)

template <int TB, int MODE, int NPM>
__global__ __launch_bounds__(kBT) void cats_ring_kernel(
    const uint16_t* __restrict__ xp, int B, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int np, float t, float* __restrict__ act,
    const unsigned long long* __restrict__ cut, uint16_t* __restrict__ hhi,
    uint16_t* __restrict__ hlo, int hs, int sp, int32_t* __restrict__ uidx,
    int32_t* __restrict__ ucnt, int32_t* __restrict__ bidx, int32_t* __restrict__ bcnt) {
  using G = typename CatsGeom<TB, NPM>::G;
  constexpr int MT = (TB + 15) / 16, KS = G::kRowBytes / 2;
  constexpr int kMpad = 16 * MT;
  extern __shared__ __attribute__((aligned(16))) unsigned char ring[];
  __shared__ float s_a[kMpad][kSegPad];             // a = SiLU(g) per token and position
  __shared__ unsigned long long s_keep[kMpad];      // kept positions per token
  __shared__ int s_u[kSegPad];                      // union positions, ascending
  __shared__ int s_nu;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int seg = blockIdx.x, nseg = gridDim.x;
  const int r0 = seg * np;
  const int nr = min(np, F - r0);  // neurons of this segment (>= 1)
  const int nblk = (d + KS - 1) / KS;
  const int tau = wave & 3, kap = wave >> 2;
  constexpr int kSteps = KS / 32;  // 32-wide K steps per block
  static_assert(kSteps % 2 == 0 || kSteps == 2, "the K steps split in two halves");
  constexpr int kHalf = kSteps / 2;

  // ring over the segment's rows w_row(j), j < np, and the token pieces; per-wave sums, the
  // second K half added into the first
  auto ring_pass = [&](auto w_row, floatx4_t (&acc)[MT]) {
    Ring<G> rg(tid, wave, [&](int r) -> const uint16_t* {
      if (r < np) return w_row(r);
      if (r < np + 3 * TB) {
        const int p = (r - np) / TB, m = (r - np) % TB;
        return m < B ? xp + ((size_t)p * kMpad + m) * d : nullptr;
      }
      return nullptr;
    });
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    const int wrow = 16 * tau + fr;  // past np: never stored
    const bool active = 16 * tau < np;  // a tile past the segment's rows skips its MFMAs
    run_ring<G>(ring, rg, nblk, d, np, [&](const unsigned char* slot) {
      if (!active) return;
      bf16x8_t bw[kHalf], ax[kHalf][3][MT];
#pragma unroll
      for (int i2 = 0; i2 < kHalf; ++i2) {  // every operand of the block first, then the MFMAs
        const int c = 4 * (kap * kHalf + i2) + grp;
        bw[i2] = *reinterpret_cast<const bf16x8_t*>(slot + wrow * G::kRowBytes + 16 * swz(wrow, c));
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int xr = np + p * TB + min(16 * mt + fr, TB - 1);
            ax[i2][p][mt] = *reinterpret_cast<const bf16x8_t*>(slot + xr * G::kRowBytes + 16 * swz(xr, c));
          }
      }
#pragma unroll
      for (int i2 = 0; i2 < kHalf; ++i2)
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ax[i2][p][mt], bw[i2], acc[mt], 0, 0, 0);
    });
    // the second K half hands its sums to the first through LDS (the ring is free afterwards)
    __syncthreads();
    floatx4_t* s_h = reinterpret_cast<floatx4_t*>(ring);  // [tile][mt][lane]
    if (kap == 1) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) s_h[(tau * MT + mt) * kWave + lane] = acc[mt];
    }
    __syncthreads();
    if (kap == 0) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const floatx4_t o = s_h[(tau * MT + mt) * kWave + lane];
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[mt][r] += o[r];
      }
    }
    __syncthreads();  // the ring may be refilled by the next pass
  };

  // ---- phase A: the gate (threshold mode and the top-k gate pass) or the stored activations
  if (MODE != kModeKeyed) {
    floatx4_t acc[MT];
    ring_pass([&](int j) { return wg + (size_t)(r0 + min(j, nr - 1)) * d; }, acc);
    if (kap == 0) {
      const int j = 16 * tau + fr;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * mt + 4 * grp + r;  // C layout: neuron fr, tokens 4 (lane / 16) + r
          const float a = silu(acc[mt][r]);
          if (MODE == kModeAct) {
            if (m < B && j < nr) act[(size_t)m * F + r0 + j] = a;
          } else {
            s_a[m][j] = a;
          }
        }
    }
    if (MODE == kModeAct) return;  // uniform
    __syncthreads();
  } else {
    for (int i = tid; i < kMpad * kSegPad; i += kBT) {
      const int m = i / kSegPad, j = i % kSegPad;
      s_a[m][j] = (m < B && j < nr) ? act[(size_t)m * F + r0 + j] : 0.f;
    }
    __syncthreads();
  }

  // ---- keep decisions per token (a wave ballot over the segment's positions), per-token lists
  for (int m = wave; m < kMpad; m += kBT / kWave) {
    const float a = s_a[m][lane];
    bool keep = false;
    if (m < B && lane < nr) {
      if (MODE == kModeKeyed) keep = topk_key(a, r0 + lane) >= cut[m];
      else if (MODE == kModeAll) keep = true;
      else keep = fabsf(a) > t;
    }
    const unsigned long long mk = __ballot(keep);
    if (lane == 0) s_keep[m] = mk;
    if (m < B && bidx != nullptr) {
      if (keep) bidx[((size_t)m * nseg + seg) * kSegPad + __popcll(mk & ((1ull << lane) - 1ull))] = r0 + lane;
      if (lane == 0) bcnt[m * nseg + seg] = __popcll(mk);
    }
  }
  __syncthreads();
  // ---- union of the tokens' kept positions, ascending
  if (wave == 0) {
    unsigned long long un = 0ull;
    for (int m = 0; m < B && m < kMpad; ++m) un |= s_keep[m];
    const bool in = (un >> lane) & 1ull;
    const int pos = __popcll(un & ((1ull << lane) - 1ull));
    if (in) {
      s_u[pos] = lane;
      uidx[seg * sp + pos] = r0 + lane;
    }
    if (lane == 0) {
      s_nu = __popcll(un);
      ucnt[seg] = __popcll(un);
    }
  }
  __syncthreads();
  const int nu = s_nu;

  // ---- phase B: the up rows of the union only; h = a u where the token keeps the neuron
  floatx4_t acc[MT];
  if (nu > 0) {  // uniform
    // union rows past nu load the segment's first union row again (in L2, never stored)
    ring_pass([&](int k) { return wu + (size_t)(r0 + s_u[min(k, nu - 1)]) * d; }, acc);
  }
  if (kap == 0) {
    const int k = 16 * tau + fr;  // union position
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * grp + r;
        float h = 0.f;
        if (k < nu) {
          const int j = s_u[k];
          if ((s_keep[m] >> j) & 1ull) h = s_a[m][j] * acc[mt][r];
        }
        if (k < sp) store_h(hhi, hlo, (size_t)m * hs + seg * sp + k, h);  // 0 past nu
      }
  }
  if (seg == nseg - 1) zero_h_tail(hhi, hlo, hs, nseg * sp, kMpad);
}

// ---- down product: Y_partial[rho][m][c] over one 256-column tile and one range of 64-row blocks.
// Block b is positions 64 b .. + 63 of the segment layout (segment s owns positions s sp .. +
// sp - 1, sp in {16, 32, 64}). Whole segments (GATHER = 0, the dense gate/up kernel): position
// s sp + k is W_down row s np + k for k < np (and below d_ff). Kept lists (GATHER = 1): it is row
// uidx[s sp + k] for k < ucnt[s]. Any other position has no row (h = 0 there; W_down row 0 is
// loaded, an L2 hit). The 64-row blocks of whole segments measured faster than blocks of 64
// consecutive neurons (dense 16-token pass at the Llama-3-8B layer: 22.6 against 27.2 us).
// Slot: the block's 64 W_down rows over the tile (512 bytes each; chunk c of row r at
// c ^ 2 ((r / 8) % 4), so the 16-bit B-operand gathers of one instruction touch 32 banks), then
// the hi/lo h fragments in A-operand lane order. Wave w: columns 32 w .. + 31 (two 16-column tiles).
template <int MT>
struct DnShape {
  static constexpr int kWBytes = kDnBlock * kDnCols * 2;             // 32 KiB
  static constexpr int kHBytes = 2 * MT * 2 * kWave * 16;            // hi/lo x tiles x 2 K steps
  static constexpr int kSlotBytes = kWBytes + kHBytes;
  static constexpr int kPieces = kSlotBytes / 16;
  static constexpr int kWPieces = kWBytes / 16;
  static constexpr int kLoads = (kPieces + kBT - 1) / kBT;
  static constexpr int kFullWaves = (kPieces - (kLoads - 1) * kBT) / kWave;
  static constexpr int kSlotsMax = kLdsRing / kSlotBytes;
  static constexpr int kSlots = kSlotsMax > 4 ? 4 : kSlotsMax;
  static_assert(kPieces % kWave == 0 && kWPieces % kWave == 0, "whole wave instructions");
  static_assert(kSlots >= 3, "at least two blocks in flight");
};

__device__ __forceinline__ int dr_pos(int row, int chunk) { return chunk ^ (((row >> 3) & 3) << 1); }

template <int MT, int GATHER>
__global__ __launch_bounds__(kBT) void down_ring_kernel(
    const uint16_t* __restrict__ hhi, const uint16_t* __restrict__ hlo, int hs,
    const uint16_t* __restrict__ wd, int d, int F, int B, int nblocks, int gr, int nseg, int np,
    int sp, const int32_t* __restrict__ uidx, const int32_t* __restrict__ ucnt,
    float* __restrict__ part) {
  using DS = DnShape<MT>;
  __shared__ __attribute__((aligned(16))) unsigned char ring[DS::kSlots * DS::kSlotBytes];
  __shared__ int s_rows[16 * kDnBlock];  // the range's W_down row indices (gathered blocks)
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  // workgroups go to the eight XCDs in turn (id % 8); when the grid divides evenly, XCD j takes
  // the consecutive (tile, range) indices [j N / 8, (j + 1) N / 8), so the column tiles of a
  // range share one L2 and its h fragments come from HBM once
  const int ncols = d / kDnCols, N = ncols * gr;
  const int L = blockIdx.x;
  const int idx = (N % 8 == 0) ? (L % 8) * (N / 8) + L / 8 : L;
  const int c0 = (idx % ncols) * kDnCols, rho = idx / ncols;
  const int b_lo = (int)(((long long)nblocks * rho) / gr);
  const int nb = (int)(((long long)nblocks * (rho + 1)) / gr) - b_lo;

  {  // row indices of the range's blocks (at most 16 blocks of 64 positions)
    for (int i = tid; i < nb * kDnBlock; i += kBT) {
      const int pos = b_lo * kDnBlock + i, s = pos / sp, k = pos % sp;
      // a position past its segment's rows (h = 0 there) reads W_down row 0, an L2 hit; the
      // kept lists give the rows of a gathered segment, neuron s np + k those of a whole one
      int n = 0;
      if (GATHER) n = (s < nseg && k < ucnt[s]) ? uidx[s * sp + k] : 0;
      else if (s < nseg && k < np && s * np + k < F) n = s * np + k;
      s_rows[i] = n;
    }
    __syncthreads();
  }
  // this thread's pieces of a block: piece g = q * 512 + tid; below kWPieces: W_down row g / 32,
  // position g % 32 holding chunk dr_pos(row, position) of the tile's columns; above: h fragment
  // (which, mt, step, lane) = hg / (MT 128), (hg / 128) % MT, (hg / 64) % 2, hg % 64
  const bool full = wave < DS::kFullWaves;
  int lds_off[DS::kLoads], wrow[DS::kLoads], wchunk[DS::kLoads];
  const uint16_t* hsrc[DS::kLoads];
#pragma unroll
  for (int q = 0; q < DS::kLoads; ++q) {
    const int g = min(q * kBT + tid, DS::kPieces - 1);
    lds_off[q] = (q * kBT + wave * kWave) * 16;
    if (g < DS::kWPieces) {
      wrow[q] = g >> 5;
      wchunk[q] = dr_pos(g >> 5, g & 31);
      hsrc[q] = nullptr;
    } else {
      const int hg = g - DS::kWPieces;
      const int which = hg / (MT * 128), mt = (hg / 128) % MT, st = (hg >> 6) & 1, l = hg & 63;
      wrow[q] = -1;
      wchunk[q] = 0;
      hsrc[q] = (which ? hlo : hhi) + (size_t)(16 * mt + (l & 15)) * hs + 32 * st + 8 * (l >> 4);
    }
  }
  auto issue = [&](unsigned char* slot, int b) {
    const int blk = b_lo + b;
#pragma unroll
    for (int q = 0; q < DS::kLoads; ++q) {
      if (q == DS::kLoads - 1 && !full) break;  // wave-uniform
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(slot + lds_off[q]));
      const int g0 = __builtin_amdgcn_readfirstlane(q * kBT + wave * kWave);
      if (g0 < DS::kWPieces) {
        const int n = s_rows[b * kDnBlock + wrow[q]];
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(wd + (size_t)n * d + c0 + 8 * wchunk[q]), lp, 16, 0, 2);
      } else {
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(hsrc[q] + (size_t)blk * kDnBlock), lp, 16, 0, 0);
      }
    }
  };

  const int nbv = lane & 15, gq = lane >> 4;
  floatx4_t acc[2][MT];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const unsigned char* slot) {
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      bf16x8_t ahi[MT], alo[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        ahi[mt] = as_bf16x8(*reinterpret_cast<const uint4*>(slot + DS::kWBytes + 16 * (((0 * MT + mt) * 2 + st) * kWave + lane)));
        alo[mt] = as_bf16x8(*reinterpret_cast<const uint4*>(slot + DS::kWBytes + 16 * (((1 * MT + mt) * 2 + st) * kWave + lane)));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = 32 * wave + 16 * j + nbv;
        uint32_t bw[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int ra = 32 * st + 8 * gq + 2 * jj, rb = ra + 1;
          const uint32_t e0 = *reinterpret_cast<const uint16_t*>(slot + ra * 512 + 16 * dr_pos(ra, col >> 3) + 2 * (col & 7));
          const uint32_t e1 = *reinterpret_cast<const uint16_t*>(slot + rb * 512 + 16 * dr_pos(rb, col >> 3) + 2 * (col & 7));
          bw[jj] = e0 | (e1 << 16);
        }
        const bf16x8_t bop = as_bf16x8(make_uint4(bw[0], bw[1], bw[2], bw[3]));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[mt], bop, acc[j][mt], 0, 0, 0);
          acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[mt], bop, acc[j][mt], 0, 0, 0);
        }
      }
    }
  };
#pragma unroll
  for (int p = 0; p < DS::kSlots - 1; ++p)
    if (p < nb) issue(ring + p * DS::kSlotBytes, p);
  int slot = 0, refill = DS::kSlots - 1;
  for (int b = 0; b < nb; ++b) {
    const int later = min(DS::kSlots - 2, nb - 1 - b);
    if (full) wait_later<DS::kLoads>(later);
    else wait_later<DS::kLoads - 1>(later);
    ring_barrier();
    if (b + DS::kSlots - 1 < nb) issue(ring + refill * DS::kSlotBytes, b + DS::kSlots - 1);
    compute(ring + slot * DS::kSlotBytes);
    slot = slot + 1 == DS::kSlots ? 0 : slot + 1;
    refill = refill + 1 == DS::kSlots ? 0 : refill + 1;
  }

  // C layout: lane holds column c0 + 32 wave + 16 j + lane % 16 and tokens 4 (lane / 16) + r
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = c0 + 32 * wave + 16 * j + nbv;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * gq + r;
        if (m < B) part[((size_t)rho * B + m) * d + c] = acc[j][mt][r];
      }
  }
}

int batch_mt(int B) { return (B + 15) / 16; }

}  // namespace

bool batch_path_ok(int B, int d, int F) {
  return B >= 2 && B <= 64 && d % kDnCols == 0 && d <= 8192 && F >= 1 && F <= 65536;
}

BatchLayout batch_layout(int B, int d, int F, int px) {
  BatchLayout L{};
  const int mt = batch_mt(B);
  L.mpad = 16 * mt;
  L.px = px;
  const int ncols = d / kDnCols;
  // one layout for every mode: segments of np consecutive neurons, each owning sp positions
  // (whole MFMA tiles) of h, the kept list and the down blocks
  const Seg s = seg_of(F);
  L.nseg = s.nseg;
  L.np = s.np;
  L.sp = s.np <= 16 ? 16 : (s.np <= 32 ? 32 : kSegPad);
  L.nblocks = (L.nseg * L.sp + kDnBlock - 1) / kDnBlock;
  L.hs = L.nblocks * kDnBlock;
  // down ranges: about 256 workgroups in all, at most 16 blocks per range (the gathered row list)
  L.gr = std::max(1, std::min(L.nblocks, 256 / ncols));
  while ((L.nblocks + L.gr - 1) / L.gr > 16) ++L.gr;
  Carve c;
  L.xp = c.take((size_t)px * L.mpad * d * 2);
  L.hhi = c.take((size_t)L.mpad * L.hs * 2);
  L.hlo = c.take((size_t)L.mpad * L.hs * 2);
  L.uidx = c.take((size_t)L.hs * 4);
  L.ucnt = c.take((size_t)L.nseg * 4);
  L.bidx = c.take((size_t)B * L.nseg * kSegPad * 4);
  L.bcnt = c.take((size_t)B * L.nseg * 4);
  L.part = c.take((size_t)L.gr * B * d * 4);
  L.total = c.off;
  return L;
}

namespace {

// Lets a kernel take up to `bytes` of dynamic LDS (once per kernel, on its first launch).
hipError_t allow_dynamic_lds(const void* kernel, int bytes) {
  return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

template <int TB, int NPM>
hipError_t launch_gu_np(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                        const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                        uint16_t* hlo) {
  using G = typename GuGeom<TB, NPM>::G;
  static const hipError_t attr =
      allow_dynamic_lds(reinterpret_cast<const void*>(gu_ring_kernel<TB, NPM>), kGuLds);
  if (attr != hipSuccess) return attr;
  klaunch(gu_ring_kernel<TB, NPM>, L.nseg, kBT, (uint32_t)(G::kSlots * G::kSlotBytes), stream, xp, B,
          wg, wu, d, F, L.hs, L.np, L.sp, hhi, hlo);
  return hipGetLastError();
}
template <int NSPAN>
hipError_t launch_gu_unit_n(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                            const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                            uint16_t* hlo) {
  static const hipError_t attr =
      allow_dynamic_lds(reinterpret_cast<const void*>(gu_unit_kernel<NSPAN>), kUnitLds);
  if (attr != hipSuccess) return attr;
  klaunch(gu_unit_kernel<NSPAN>, L.nseg, kUnitThreads, (uint32_t)kUnitLds, stream, xp, B, wg, wu, d,
          F, L.hs, L.np, L.sp, hhi, hlo);
  return hipGetLastError();
}
// the unit kernel takes one 16-token tile and d_model = 2048, 4096, 6144 or 8192
bool gu_unit_ok(int B, int d) { return B <= 16 && d % kUnitK == 0 && d <= 4 * kUnitK; }
hipError_t launch_gu_unit(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                          const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                          uint16_t* hlo) {
  switch (d / kUnitK) {
    case 1: return launch_gu_unit_n<1>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 2: return launch_gu_unit_n<2>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 3: return launch_gu_unit_n<3>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 4: return launch_gu_unit_n<4>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    default: return hipErrorInvalidValue;
  }
}
// short segments (np <= kSegSmall) of the small token classes take the deeper ring
template <int TB>
hipError_t launch_gu(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                     const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                     uint16_t* hlo) {
  if (TB <= 16 && L.np <= kSegSmall)
    return launch_gu_np<TB, (TB <= 16 ? kSegSmall : kSegN)>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
  return launch_gu_np<TB, kSegN>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
}

template <int TB, int MODE, int NPM>
hipError_t launch_cats_np(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                          const uint16_t* wg, const uint16_t* wu, int d, int F, float t, float* act,
                          const unsigned long long* cut, uint16_t* hhi, uint16_t* hlo,
                          int32_t* uidx, int32_t* ucnt, int32_t* bidx, int32_t* bcnt) {
  using G = typename CatsGeom<TB, NPM>::G;
  static const hipError_t attr =
      allow_dynamic_lds(reinterpret_cast<const void*>(cats_ring_kernel<TB, MODE, NPM>), kCatsLds);
  if (attr != hipSuccess) return attr;
  klaunch(cats_ring_kernel<TB, MODE, NPM>, L.nseg, kBT, (uint32_t)(G::kSlots * G::kSlotBytes), stream,
          xp, B, wg, wu, d, F, L.np, t, act, cut, hhi, hlo, L.hs, L.sp, uidx, ucnt, bidx, bcnt);
  return hipGetLastError();
}
template <int TB, int MODE>
hipError_t launch_cats(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                       const uint16_t* wg, const uint16_t* wu, int d, int F, float t, float* act,
                       const unsigned long long* cut, uint16_t* hhi, uint16_t* hlo,
                       int32_t* uidx, int32_t* ucnt, int32_t* bidx, int32_t* bcnt) {
  if (TB <= 16 && L.np <= kSegSmall)
    return launch_cats_np<TB, MODE, (TB <= 16 ? kSegSmall : kSegN)>(L, stream, xp, B, wg, wu, d, F, t, act,
                                                                     cut, hhi, hlo, uidx, ucnt, bidx, bcnt);
  return launch_cats_np<TB, MODE, kSegN>(L, stream, xp, B, wg, wu, d, F, t, act, cut, hhi, hlo, uidx,
                                         ucnt, bidx, bcnt);
}

template <int TB, int NPM>
hipError_t launch_all_np(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                         const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                         uint16_t* hlo, int32_t* uidx, int32_t* ucnt) {
  using G = typename AllGeom<TB, NPM>::G;
  static const hipError_t attr =
      allow_dynamic_lds(reinterpret_cast<const void*>(all_ring_kernel<TB, NPM>), kCatsLds);
  if (attr != hipSuccess) return attr;
  klaunch(all_ring_kernel<TB, NPM>, L.nseg, kBT, (uint32_t)(G::kSlots * G::kSlotBytes), stream, xp, B,
          wg, wu, d, F, L.np, hhi, hlo, L.hs, L.sp, uidx, ucnt);
  return hipGetLastError();
}

hipError_t launch_gu_tb(int B, const BatchLayout& L, hipStream_t stream, const uint16_t* xp,
                        const uint16_t* wg, const uint16_t* wu, int d, int F, uint16_t* hhi,
                        uint16_t* hlo) {
  switch (token_class(B)) {
    case 4: return launch_gu<4>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 8: return launch_gu<8>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 16: return launch_gu<16>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 32: return launch_gu<32>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    case 48: return launch_gu<48>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
    default: return launch_gu<64>(L, stream, xp, B, wg, wu, d, F, hhi, hlo);
  }
}

// the unit kernel of the exact-input modes: at most 4 tokens, d_model = 2048, 4096, 6144 or 8192
bool cats_unit_ok(int B, int d) {
  return B <= kCatsUnitTokens && d % kUnitK == 0 && d <= 4 * kUnitK;
}
template <int NSPAN, int MODE>
hipError_t launch_cats_unit_n(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                              const uint16_t* wg, const uint16_t* wu, int d, int F, float t,
                              float* act, const unsigned long long* cut, uint16_t* hhi,
                              uint16_t* hlo, int32_t* uidx, int32_t* ucnt, int32_t* bidx,
                              int32_t* bcnt) {
  static const hipError_t attr =
      allow_dynamic_lds(reinterpret_cast<const void*>(cats_unit_kernel<NSPAN, MODE>), kUnitLds);
  if (attr != hipSuccess) return attr;
  klaunch(cats_unit_kernel<NSPAN, MODE>, L.nseg, kUnitThreads, (uint32_t)kUnitLds, stream, xp, B, wg,
          wu, d, F, L.np, t, act, cut, hhi, hlo, L.hs, L.sp, uidx, ucnt, bidx, bcnt);
  return hipGetLastError();
}
template <int MODE>
hipError_t launch_cats_unit(const BatchLayout& L, hipStream_t stream, const uint16_t* xp, int B,
                            const uint16_t* wg, const uint16_t* wu, int d, int F, float t,
                            float* act, const unsigned long long* cut, uint16_t* hhi,
                            uint16_t* hlo, int32_t* uidx, int32_t* ucnt, int32_t* bidx,
                            int32_t* bcnt) {
#define SIRIUS_CATS_UNIT(NS)                                                                   \
  case NS:                                                                                     \
    return launch_cats_unit_n<NS, MODE>(L, stream, xp, B, wg, wu, d, F, t, act, cut, hhi, hlo, \
                                        uidx, ucnt, bidx, bcnt);
  switch (d / kUnitK) {
    SIRIUS_CATS_UNIT(1) SIRIUS_CATS_UNIT(2) SIRIUS_CATS_UNIT(3) SIRIUS_CATS_UNIT(4)
    default:
      return hipErrorInvalidValue;
  }
#undef SIRIUS_CATS_UNIT
}

template <int MODE>
hipError_t launch_cats_tb(int B, const BatchLayout& L, hipStream_t stream, const uint16_t* xp,
                          const uint16_t* wg, const uint16_t* wu, int d, int F, float t,
                          float* act, const unsigned long long* cut, uint16_t* hhi, uint16_t* hlo,
                          int32_t* uidx, int32_t* ucnt, int32_t* bidx, int32_t* bcnt) {
  if (cats_unit_ok(B, d))
    return launch_cats_unit<MODE>(L, stream, xp, B, wg, wu, d, F, t, act, cut, hhi, hlo, uidx, ucnt,
                                  bidx, bcnt);
#define SIRIUS_CATS_TB(TBV)                                                                     \
  case TBV:                                                                                     \
    return launch_cats<TBV, MODE>(L, stream, xp, B, wg, wu, d, F, t, act, cut, hhi, hlo, uidx,  \
                                  ucnt, bidx, bcnt);
  switch (token_class(B)) {
    SIRIUS_CATS_TB(4) SIRIUS_CATS_TB(8) SIRIUS_CATS_TB(16) SIRIUS_CATS_TB(32) SIRIUS_CATS_TB(48)
    default:
      return launch_cats<64, MODE>(L, stream, xp, B, wg, wu, d, F, t, act, cut, hhi, hlo, uidx,
                                   ucnt, bidx, bcnt);
  }
#undef SIRIUS_CATS_TB
}

}  // namespace

hipError_t launch_ffn_batch(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                            const uint16_t* wd, int d, int F, int mode, float t, float norm_eps,
                            const float* resid, float* y, int32_t* active_idx,
                            int32_t* active_cnt, char* ws, const BatchLayout& L,
                            hipStream_t stream, const float* act,
                            const unsigned long long* cut) {
  if (!batch_path_ok(B, d, F) || L.mpad != 16 * batch_mt(B)) return hipErrorInvalidValue;
  // the segment kernels (gate pass, then the up rows of the kept union) serve every call on the
  // exact input: threshold, top-k, and dense / condensed small batches with every neuron kept
  const bool exact = L.px == 3;
  if (mode != kFfnModeDense && !exact) return hipErrorInvalidValue;
  if (mode == kFfnModeTopK && (act == nullptr || cut == nullptr)) return hipErrorInvalidValue;
  const int mt = L.mpad / 16;
  uint16_t* xp = reinterpret_cast<uint16_t*>(ws + L.xp);
  uint16_t* hhi = reinterpret_cast<uint16_t*>(ws + L.hhi);
  uint16_t* hlo = reinterpret_cast<uint16_t*>(ws + L.hlo);
  int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.uidx);
  int32_t* ucnt = reinterpret_cast<int32_t*>(ws + L.ucnt);
  const bool lists = mode != kFfnModeDense && active_idx != nullptr;
  int32_t* bidx = lists ? reinterpret_cast<int32_t*>(ws + L.bidx) : nullptr;
  int32_t* bcnt = lists ? reinterpret_cast<int32_t*>(ws + L.bcnt) : nullptr;
  float* part = reinterpret_cast<float*>(ws + L.part);
  const bool thr = mode == kFfnModeThreshold, topk = mode == kFfnModeTopK;
  const char* pfx_prep = "batch_prep";
  const char* pfx_gu = topk ? "batch_topk_up"
                       : thr ? "batch_cats_up"
                             : (exact ? "batch_seg_gate_up" : "batch_gate_up");
  const char* pfx_dn = "batch_down";
  const char* pfx_red = "batch_reduce";
  hipError_t e;
  {
    ProfScope prof(pfx_prep, stream);
    if (L.px == 3) klaunch(prep_pieces_kernel<3>, L.mpad, 256, 0, stream, x, B, d, L.mpad, norm_eps, xp);
    else klaunch(prep_pieces_kernel<1>, L.mpad, 256, 0, stream, x, B, d, L.mpad, norm_eps, xp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    ProfScope prof(pfx_gu, stream);
    if (!exact) {
      e = gu_unit_ok(B, d) ? launch_gu_unit(L, stream, xp, B, wg, wu, d, F, hhi, hlo)
                           : launch_gu_tb(B, L, stream, xp, wg, wu, d, F, hhi, hlo);
    } else if (thr) {
      e = launch_cats_tb<kModeThr>(B, L, stream, xp, wg, wu, d, F, t, nullptr, nullptr, hhi, hlo,
                                   uidx, ucnt, bidx, bcnt);
    } else if (topk) {
      e = launch_cats_tb<kModeKeyed>(B, L, stream, xp, wg, wu, d, F, 0.f, const_cast<float*>(act),
                                     cut, hhi, hlo, uidx, ucnt, bidx, bcnt);
    } else if (token_class(B) <= 8 && L.np <= kSegSmall && !cats_unit_ok(B, d)) {  // every neuron kept: one ring pass
      e = token_class(B) == 4
              ? launch_all_np<4, kSegSmall>(L, stream, xp, B, wg, wu, d, F, hhi, hlo, uidx, ucnt)
              : launch_all_np<8, kSegSmall>(L, stream, xp, B, wg, wu, d, F, hhi, hlo, uidx, ucnt);
    } else {
      e = launch_cats_tb<kModeAll>(B, L, stream, xp, wg, wu, d, F, 0.f, nullptr, nullptr, hhi, hlo,
                                   uidx, ucnt, bidx, bcnt);
    }
    if (e != hipSuccess) return e;
  }
  {
    ProfScope prof(pfx_dn, stream);
    const int grid = (d / kDnCols) * L.gr;
#define SIRIUS_DN(MTV)                                                                                  \
  if (mt == MTV) {                                                                                      \
    if (exact)                                                                                          \
      klaunch(down_ring_kernel<MTV, 1>, grid, kBT, 0, stream, hhi, hlo, L.hs, wd, d, F, B, L.nblocks,   \
              L.gr, L.nseg, L.np, L.sp, uidx, ucnt, part);                                              \
    else                                                                                                \
      klaunch(down_ring_kernel<MTV, 0>, grid, kBT, 0, stream, hhi, hlo, L.hs, wd, d, F, B, L.nblocks,   \
              L.gr, L.nseg, L.np, L.sp, uidx, ucnt, part);                                              \
  }
    SIRIUS_DN(1) SIRIUS_DN(2) SIRIUS_DN(3) SIRIUS_DN(4)
#undef SIRIUS_DN
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  ProfScope prof(pfx_red, stream);
  if (lists)
    return launch_reduce(part, L.gr, B, d, resid, y, stream, F, L.nseg, kSegPad, bidx, bcnt,
                         active_idx, active_cnt);
  return launch_reduce(part, L.gr, B, d, resid, y, stream);
}

hipError_t launch_batch_act(const float* x, int B, const uint16_t* wg, int d, int F,
                            float norm_eps, float* act, char* ws, const BatchLayout& L,
                            hipStream_t stream) {
  if (!batch_path_ok(B, d, F) || L.px != 3 || L.mpad != 16 * batch_mt(B)) return hipErrorInvalidValue;
  uint16_t* xp = reinterpret_cast<uint16_t*>(ws + L.xp);
  hipError_t e;
  {
    ProfScope prof("batch_topk_prep", stream);
    klaunch(prep_pieces_kernel<3>, L.mpad, 256, 0, stream, x, B, d, L.mpad, norm_eps, xp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  ProfScope prof("batch_topk_gate", stream);
  return launch_cats_tb<kModeAct>(B, L, stream, xp, wg, nullptr, d, F, 0.f, act, nullptr, nullptr,
                                  nullptr, nullptr, nullptr, nullptr, nullptr);
}

}  // namespace sirius
