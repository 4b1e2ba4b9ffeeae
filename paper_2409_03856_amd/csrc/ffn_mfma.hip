// Multi-token SwiGLU FFN on MFMA (gfx950), for batches of 8..64 tokens: the full model's
// parallel pass over a drafted chunk, and condensed / dense decode of batched tokens. Both
// products stream their weights once and stay HBM-bound at these batch sizes (16 tokens: two
// flops per weight byte per token, against a bf16 MFMA ridge near 300), so the kernels are
// organised around full-line weight reads, and v_mfma_f32_16x16x32_bf16 does the arithmetic.
//
//  prep_x_kernel   x -> RMSNorm (optional) -> bf16, zero-padded to a multiple of 16 rows.
//  gate_up_ring_kernel  H for one 16-token tile (the full model's check of a 16-token chunk):
//                  one 512-thread workgroup per segment of at most 56 neurons, weights and x
//                  moved into a four-slot LDS ring by direct global-to-LDS loads (three K
//                  blocks in flight, no staging registers); see its definition.
//  gate_up_kernel  H = SiLU(X W_gate^T) * (X W_up^T) for the other shapes (more than 16
//                  tokens, d_model not a multiple of 128). A two-wave workgroup owns 8 neurons
//                  (the MFMA tile's other 8 B-operand rows are zero), 7 workgroups per CU at
//                  d_ff = 14336. Per 256-wide K block it stages the tile's gate and up rows and
//                  the x rows in LDS with coalesced loads (512 contiguous bytes per row;
//                  reading the MFMA operand layout straight from HBM gives only 64 contiguous
//                  bytes per row per instruction and ran at about 3.6 TB/s), requests the next
//                  block, and the two waves take alternate MFMA steps of the block, reading
//                  operands with 16-byte LDS reads. (16-row tiles with wave-private staging,
//                  deeper prefetch and staggered K starts measured the same or slower.) The
//                  two waves' sums are added in a fixed order. h is stored as a pair of bf16
//                  values, hi = bf16(h) and lo = bf16(h - hi), token-major [Mpad, F16]
//                  (F16 = d_ff rounded up to 64, a whole number of down blocks; padding
//                  0): the down product takes both, which keeps about 16 significant bits
//                  of h.
//  down_ring_kernel  Y_partial for one 16-token tile with d_model % 256 == 0: one 576-thread
//                  workgroup per (256-column tile, neuron range), 64-neuron blocks of W_down
//                  and the matching h fragments moved into a four-slot LDS ring by direct
//                  global-to-LDS loads; see its definition.
//  down_kernel     Y_partial = H W_down over one neuron range and one 64-column tile.
//                  W_down is neuron-major (columns contiguous) but the MFMA B operand wants
//                  eight consecutive neurons of one column per lane, so each 64-neuron x
//                  64-column chunk is staged in LDS (rows padded to 136 bytes) and the
//                  operand is gathered with 16-bit LDS reads; the four 8-row groups of a
//                  gather fall 16 banks apart, so the gathers are conflict-free. The chunk's
//                  hi/lo h fragments are staged in LDS as well and shared by the four waves
//                  (one 16-column tile each). The next chunks' loads are kept in flight in
//                  registers while the current chunk is multiplied.
//  reduce_kernel   (ffn_gemv.hip) y = resid + the neuron-range partials in a fixed order.
#include "common.h"
#include "kernels.h"
#include "profile.h"
#include "ring.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

constexpr int kMTile = 16;     // MFMA M (tokens) and N (neurons / columns) tile
constexpr int kKBlock = 256;   // gate/up: K elements per block (8 MFMA steps of 32)
constexpr int kMaxMTiles = 4;  // batch <= 64
constexpr int kGuPitch = kKBlock * 2 + 16;  // bytes per staged gate/up row (528)
constexpr int kGuRows = 8;  // neurons per gate/up workgroup (the MFMA tile's other 8 rows are 0)
constexpr int kGuDepth = 1;  // K blocks in flight per gate/up workgroup

constexpr int kDnCols = 64;                // down: output columns per workgroup (4 waves x 16)
constexpr int kDnChunk = 64;               // down: neurons per LDS chunk (2 MFMA steps)
constexpr int kDnSteps = kDnChunk / 32;
constexpr int kDnPitch = kDnCols * 2 + 8;  // bytes per staged W_down row (136)
constexpr int kDnPrefetch = 4;             // chunks in flight per thread
constexpr int kDnTarget = 1024;            // down workgroups to aim for

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// ---- x -> optional RMSNorm -> bf16 [Mpad][d]; one workgroup per padded row. Every thread
// requests all of its (at most eight) 16-byte pieces of the row before using any of them.
__global__ __launch_bounds__(256) void prep_x_kernel(const float* __restrict__ x, int B, int d,
                                                     float norm_eps, uint16_t* __restrict__ xb) {
  constexpr int kPer = 8;  // d_model <= 8192: 2048 float4 per row over 256 threads
  __shared__ float s_w[4];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int m = blockIdx.x;
  uint2* out = reinterpret_cast<uint2*>(xb + (size_t)m * d);
  const int nv4 = d >> 2;
  if (m >= B) {  // uniform over the block
    for (int i = tid; i < nv4; i += 256) out[i] = make_uint2(0u, 0u);
    return;
  }
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)m * d);
  float4 v[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    v[u] = (i < nv4) ? xr[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float inv = 1.0f;
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
    inv = 1.0f / sqrtf(tot / (float)d + norm_eps);
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + 256 * u;
    if (i < nv4) {
      float4 w = v[u];
      if (norm_eps >= 0.f) {
        w.x *= inv;
        w.y *= inv;
        w.z *= inv;
        w.w *= inv;
      }
      out[i] = make_uint2(f32_to_bf16(w.x) | (f32_to_bf16(w.y) << 16),
                          f32_to_bf16(w.z) | (f32_to_bf16(w.w) << 16));
    }
  }
}

template <int MT>
__global__ __launch_bounds__(128) void gate_up_kernel(
    const uint16_t* __restrict__ xb, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int F16, uint16_t* __restrict__ hhi,
    uint16_t* __restrict__ hlo) {
  // one K block at a time: the tile's gate and up rows and the x rows, padded to kGuPitch
  __shared__ __attribute__((aligned(16))) unsigned char s_w[2][kGuRows * kGuPitch];
  __shared__ __attribute__((aligned(16))) unsigned char s_x[MT * kMTile * kGuPitch];
  __shared__ floatx4_t s_acc[MT][2][kWave];  // the second wave's sums: [m tile][gate/up][lane]
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int n0 = blockIdx.x * kGuRows;
  const int fr = lane & 15, grp = lane >> 4;  // MFMA fragment row, lane group
  const bool frv = fr < kGuRows;              // B-operand rows 8..15 of the tile stay zero
  const int nch = d >> 3;

  floatx4_t accg[MT], accu[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    accg[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    accu[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }
  constexpr int kSteps = kKBlock / 32;
  // staging of one block by the 128 threads, 16 bytes each per load: weight row r of the tile
  // (gate for r < 8, up for r >= 8) or x row r - 16, K chunk tid % 32 of the block
  constexpr int kRowsStaged = 2 * kGuRows + MT * kMTile;
  constexpr int kLoads = kRowsStaged * (kKBlock / 8) / 128;
  static_assert((kRowsStaged * (kKBlock / 8)) % 128 == 0, "whole loads per thread");
  const int nblk = (d + kKBlock - 1) / kKBlock;
  const int schunk = tid & 31, srow0 = tid >> 5;  // 4 rows per load round
  uint4 v[kGuDepth][kLoads];
  auto load_block = [&](int blk, uint4(&vv)[kLoads]) {
#pragma unroll
    for (int q = 0; q < kLoads; ++q) {
      const int r = srow0 + 4 * q;
      const int c = blk * (kKBlock / 8) + schunk;
      const bool cok = blk < nblk && c < nch;
      if (r < 2 * kGuRows) {
        const int row = n0 + (r & (kGuRows - 1));
        const uint4* base = reinterpret_cast<const uint4*>(r < kGuRows ? wg : wu);
        vv[q] = (cok && row < F) ? ld_stream(base + (size_t)row * nch + c) : make_uint4(0u, 0u, 0u, 0u);
      } else {
        const int m = r - 2 * kGuRows;
        vv[q] = cok ? *(reinterpret_cast<const uint4*>(xb + (size_t)m * d) + c) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };
#pragma unroll
  for (int p = 0; p < kGuDepth; ++p) load_block(p, v[p]);
  for (int b0 = 0; b0 < nblk; b0 += kGuDepth) {
#pragma unroll
    for (int p = 0; p < kGuDepth; ++p) {
      const int blk = b0 + p;
      if (blk >= nblk) break;  // uniform over the block
      __syncthreads();  // both waves are done reading the previous block
#pragma unroll
      for (int q = 0; q < kLoads; ++q) {
        const int r = srow0 + 4 * q;
        unsigned char* dst = (r < 2 * kGuRows)
                                 ? s_w[r / kGuRows] + (r & (kGuRows - 1)) * kGuPitch
                                 : s_x + (r - 2 * kGuRows) * kGuPitch;
        *reinterpret_cast<uint4*>(dst + 16 * schunk) = v[p][q];
      }
      __syncthreads();
      load_block(blk + kGuDepth, v[p]);  // in flight while the next blocks are multiplied
      // wave w takes MFMA steps w, w + 2, ... of the block
#pragma unroll
      for (int i2 = 0; i2 < kSteps / 2; ++i2) {
        const int i = 2 * i2 + wave;
        const int off = 2 * (32 * i + 8 * grp);
        uint4 vg = *reinterpret_cast<const uint4*>(s_w[0] + (frv ? fr : 0) * kGuPitch + off);
        uint4 vu = *reinterpret_cast<const uint4*>(s_w[1] + (frv ? fr : 0) * kGuPitch + off);
        if (!frv) vg = vu = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const uint4 xa = *reinterpret_cast<const uint4*>(s_x + (mt * kMTile + fr) * kGuPitch + off);
          accg[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(xa), as_bf16x8(vg), accg[mt], 0, 0, 0);
          accu[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(xa), as_bf16x8(vu), accu[mt], 0, 0, 0);
        }
      }
    }
  }

  // fixed-order sum of the two waves' steps, then the epilogue on the first wave
  if (wave == 1) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      s_acc[mt][0][lane] = accg[mt];
      s_acc[mt][1][lane] = accu[mt];
    }
  }
  __syncthreads();
  if (wave == 0 && frv) {
    // C layout: lane holds tile row lane % 16 and tokens 4 (lane / 16) + r of each m tile.
    // Rows past d_ff (up to F16) have zero weights and padded tokens zero inputs: h = 0.
    const int n = n0 + fr;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4_t og = s_acc[mt][0][lane], ou = s_acc[mt][1][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * kMTile + 4 * grp + r;
        const float g = accg[mt][r] + og[r];
        const float u = accu[mt][r] + ou[r];
        const float h = silu(g) * u;
        const uint32_t hi = f32_to_bf16(h);
        const float lo = h - __uint_as_float(hi << 16);
        hhi[(size_t)m * F16 + n] = (uint16_t)hi;
        hlo[(size_t)m * F16 + n] = (uint16_t)f32_to_bf16(lo);
      }
    }
  }
}

// ---- gate/up for one 16-token tile (B <= 16, d_model % 128 == 0, at most 56 neurons per
// segment): one 512-thread workgroup per segment of np neurons (56 at d_ff = 14336, one per
// CU). Each 128-wide K block of the segment's gate rows, up rows and the 16 x rows is moved
// into one slot of a four-slot LDS ring with direct global-to-LDS 16-byte loads, so three
// blocks (84 KiB of weights per CU) are in flight without staging registers, and the x block
// is fetched once per segment instead of once per 8 neurons. A wave instruction writes 64
// consecutive 16-byte LDS slots, so the row layout is fixed at 256 bytes per row; each lane
// therefore fetches the chunk that its slot should hold under an XOR swizzle of the chunk
// index by the row (chunk c of row r sits at position c ^ (r & 7)), which keeps the MFMA
// operand reads of 16 rows at one chunk free of bank conflicts beyond the two passes that
// 256 bytes need anyway. Wave w multiplies tile w / 2 (16 neurons) of the gate (w even) or up
// (w odd) rows: four v_mfma_f32_16x16x32_bf16 steps per block. Every lane issues every load
// (rows past the segment fetch a valid row that is never used), so the wait counts are exact.
constexpr int kRgThreads = 512;
constexpr int kRgK = 128;                        // K per ring block: 256 bytes per row
constexpr int kRgRowBytes = kRgK * 2;
constexpr int kRgRows = 128;                     // 2 npad weight rows + 16 x rows (+ unused)
constexpr int kRgSlotBytes = kRgRows * kRgRowBytes;              // 32 KiB
constexpr int kRgLoads = kRgRows * (kRgK / 8) / kRgThreads;      // direct loads per thread per block
constexpr int kRgMaxNeurons = (kRgRows - kMTile) / 2;            // 56
static_assert(kRgLoads == 4, "the wait counts below assume four loads per thread per block");

__device__ __forceinline__ int rg_pos(int row, int chunk) { return chunk ^ (row & 7); }


__global__ __launch_bounds__(kRgThreads) void gate_up_ring_kernel(
    const uint16_t* __restrict__ xb, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int F16, int np,
    uint16_t* __restrict__ hhi, uint16_t* __restrict__ hlo) {
  // four slots as four arrays, so that every LDS access names its slot
  __shared__ __attribute__((aligned(16))) unsigned char s_r0[kRgSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_r1[kRgSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_r2[kRgSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_r3[kRgSlotBytes];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int fr = lane & 15, grp = lane >> 4;
  const int npad = (np + 7) & ~7;
  const int n0 = blockIdx.x * np;
  const int nblk = d / kRgK;

  // this thread's four loads of a block: slot position g = q * 512 + tid (row g / 16,
  // position g % 16), holding logical chunk rg_pos(row, position) of that row
  const uint16_t* src[kRgLoads];
  int lds_off[kRgLoads];
#pragma unroll
  for (int q = 0; q < kRgLoads; ++q) {
    const int g = q * kRgThreads + tid;
    const int r = g >> 4, c = rg_pos(r, g & 15);
    const uint16_t* base;
    if (r < 2 * npad) {
      const int j = r < npad ? r : r - npad;
      const int n = min(n0 + min(j, np - 1), F - 1);  // rows past the segment or d_ff: any valid row
      base = (r < npad ? wg : wu) + (size_t)n * d;
    } else {
      const int t = r - 2 * npad;
      base = xb + (size_t)(t < kMTile ? t : 0) * d;  // unused rows: x row 0
    }
    src[q] = base + 8 * c;
    lds_off[q] = (q * kRgThreads + wave * kWave) * 16;  // wave-uniform: lane l lands at + 16 l
  }
  auto issue = [&](unsigned char* slot, int blk) {
#pragma unroll
    for (int q = 0; q < kRgLoads; ++q) {
      // a wave instruction covers four whole rows and 2 npad is a multiple of 16: the row
      // kind is uniform over the wave (taken from lane 0, so the branch is scalar and each
      // q issues exactly one load per wave)
      const int w0 = q * kRgThreads + wave * kWave;
      const bool weight = __builtin_amdgcn_readfirstlane(w0 >> 4) < 2 * npad;
      const void* gp = src[q] + (size_t)blk * kRgK;
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(slot + lds_off[q]));
      if (weight)
        __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 2);  // non-temporal: read once
      else
        __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 0);
    }
  };

  const int tau = wave >> 1, mu = wave & 1;
  const bool active = 16 * tau < np;
  const int wrow = mu * npad + 16 * tau + fr;  // B operand row (past np: never stored)
  const int xrow = 2 * npad + fr;              // A operand row
  floatx4_t acc = floatx4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const unsigned char* slot) {
    if (!active) return;
#pragma unroll
    for (int i = 0; i < kRgK / 32; ++i) {
      const int c = 4 * i + grp;
      const uint4 bw = *reinterpret_cast<const uint4*>(slot + wrow * kRgRowBytes + 16 * rg_pos(wrow, c));
      const uint4 ax = *reinterpret_cast<const uint4*>(slot + xrow * kRgRowBytes + 16 * rg_pos(xrow, c));
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ax), as_bf16x8(bw), acc, 0, 0, 0);
    }
  };
  // block b: wait for it (the blocks issued after it stay in flight), barrier, refill the slot
  // freed by block b - 1 with block b + 3, multiply block b
  auto step = [&](unsigned char* slot, unsigned char* refill, int b) {
    const int later = min(2, nblk - 1 - b);
    if (later >= 2) wait_vm<2 * kRgLoads>();
    else if (later == 1) wait_vm<kRgLoads>();
    else wait_vm<0>();
    ring_barrier();
    if (b + 3 < nblk) issue(refill, b + 3);
    compute(slot);
  };
  issue(s_r0, 0);
  if (nblk > 1) issue(s_r1, 1);
  if (nblk > 2) issue(s_r2, 2);
  for (int b = 0; b < nblk; b += 4) {
    step(s_r0, s_r3, b);
    if (b + 1 < nblk) step(s_r1, s_r0, b + 1);
    if (b + 2 < nblk) step(s_r2, s_r1, b + 2);
    if (b + 3 < nblk) step(s_r3, s_r2, b + 3);
  }

  // epilogue: the up wave of each tile hands its sums to the gate wave through LDS
  __syncthreads();  // every wave is done with the ring
  floatx4_t* s_up = reinterpret_cast<floatx4_t*>(s_r0);  // [tile][lane]
  if (active && mu == 1) s_up[tau * kWave + lane] = acc;
  __syncthreads();
  if (active && mu == 0) {
    const floatx4_t u4 = s_up[tau * kWave + lane];
    const int j = 16 * tau + fr, n = n0 + j;
    if (j < np && n < F16) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 4 * grp + r;
        // C layout: lane holds neuron fr and tokens 4 (lane / 16) + r; past d_ff: h = 0
        const float h = n < F ? silu(acc[r]) * u4[r] : 0.f;
        const uint32_t hi = f32_to_bf16(h);
        const float lo = h - __uint_as_float(hi << 16);
        hhi[(size_t)m * F16 + n] = (uint16_t)hi;
        hlo[(size_t)m * F16 + n] = (uint16_t)f32_to_bf16(lo);
      }
    }
  }
}

// Y_partial[rho][m][c] = sum over the neurons n of range rho of H[m][n] * W_down[n][c]
template <int MT>
__global__ __launch_bounds__(256) void down_kernel(
    const uint16_t* __restrict__ hhi, const uint16_t* __restrict__ hlo, int F16,
    const uint16_t* __restrict__ wd, int d, int F, int B, int nchunk, float* __restrict__ part) {
  constexpr int kHFrags = 2 * MT * kDnSteps * kWave;  // [hi/lo][m tile][step][lane]
  constexpr int kHPerThread = kHFrags / 256;
  static_assert(kHFrags % 256 == 0, "h fragments split evenly over the threads");
  __shared__ __attribute__((aligned(16))) unsigned char s_w[kDnChunk * kDnPitch];
  __shared__ uint4 s_h[kHFrags];

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int c0 = blockIdx.x * kDnCols, rho = blockIdx.y, gr = gridDim.y;
  const int ch_lo = (int)(((long long)nchunk * rho) / gr);
  const int ch_hi = (int)(((long long)nchunk * (rho + 1)) / gr);
  const int nch = d >> 3;  // 16-byte chunks per W_down row

  // weight staging: thread t loads rows t / 8 and t / 8 + 32 of a chunk, 16 bytes at
  // column c0 + 8 (t % 8)
  const int lr = tid >> 3, lc = tid & 7;
  const int gcol = (c0 >> 3) + lc;
  const bool colok = gcol < nch;
  auto load_w = [&](int ch, uint4(&v)[2]) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int n = ch * kDnChunk + lr + 32 * q;
      v[q] = (ch < ch_hi && colok && n < F)
                 ? ld_stream(reinterpret_cast<const uint4*>(wd) + (size_t)n * nch + gcol)
                 : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  // h fragment f = ((which * MT + mt) * kDnSteps + s) * 64 + l holds, for A-operand lane l
  // (token mt * 16 + l % 16, neuron group l / 16), neurons 32 s + 8 (l / 16) .. + 7 of the chunk
  auto load_h = [&](int ch, uint4(&v)[kHPerThread]) {
#pragma unroll
    for (int i = 0; i < kHPerThread; ++i) {
      const int f = tid + 256 * i;
      const int l = f % kWave, s = (f / kWave) % kDnSteps, mt = (f / (kWave * kDnSteps)) % MT;
      const int which = f / (kWave * kDnSteps * MT);
      const int k = ch * kDnChunk + 32 * s + 8 * (l >> 4);
      const int m = mt * kMTile + (l & 15);
      v[i] = (ch < ch_hi && k < F16)
                 ? *reinterpret_cast<const uint4*>((which ? hlo : hhi) + (size_t)m * F16 + k)
                 : make_uint4(0u, 0u, 0u, 0u);
    }
  };

  floatx4_t acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  uint4 wv[kDnPrefetch][2], hv[kDnPrefetch][kHPerThread];
#pragma unroll
  for (int p = 0; p < kDnPrefetch; ++p) {
    load_w(ch_lo + p, wv[p]);
    load_h(ch_lo + p, hv[p]);
  }
  const int nb = lane & 15, gq = lane >> 4;  // B operand: column 16 wave + nb, neuron group gq
  for (int ch = ch_lo; ch < ch_hi; ch += kDnPrefetch) {
#pragma unroll
    for (int p = 0; p < kDnPrefetch; ++p) {
      if (ch + p >= ch_hi) break;  // uniform over the block
      __syncthreads();             // the previous chunk's readers are done with s_w / s_h
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        uint2* dst = reinterpret_cast<uint2*>(s_w + (lr + 32 * q) * kDnPitch + lc * 16);
        dst[0] = make_uint2(wv[p][q].x, wv[p][q].y);
        dst[1] = make_uint2(wv[p][q].z, wv[p][q].w);
      }
#pragma unroll
      for (int i = 0; i < kHPerThread; ++i) s_h[tid + 256 * i] = hv[p][i];
      __syncthreads();
      // refill this slot with the chunk kDnPrefetch ahead
      load_w(ch + p + kDnPrefetch, wv[p]);
      load_h(ch + p + kDnPrefetch, hv[p]);
#pragma unroll
      for (int s = 0; s < kDnSteps; ++s) {
        // B operand: rows 32 s + 8 gq + j (j = 0..7) of column 16 wave + nb, from LDS
        const unsigned char* col = s_w + (32 * s + 8 * gq) * kDnPitch + (16 * wave + nb) * 2;
        uint32_t bw[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t e0 = *reinterpret_cast<const uint16_t*>(col + (2 * j) * kDnPitch);
          const uint32_t e1 = *reinterpret_cast<const uint16_t*>(col + (2 * j + 1) * kDnPitch);
          bw[j] = e0 | (e1 << 16);
        }
        const bf16x8_t bop = as_bf16x8(make_uint4(bw[0], bw[1], bw[2], bw[3]));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const bf16x8_t ahi = as_bf16x8(s_h[(mt * kDnSteps + s) * kWave + lane]);
          const bf16x8_t alo = as_bf16x8(s_h[((MT + mt) * kDnSteps + s) * kWave + lane]);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bop, acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bop, acc[mt], 0, 0, 0);
        }
      }
    }
  }

  // C layout: lane holds column c0 + 16 wave + lane % 16 and tokens 4 (lane / 16) + r
  const int c = c0 + 16 * wave + nb;
  if (c < d) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * kMTile + 4 * gq + r;
        if (m < B) part[((size_t)rho * B + m) * d + c] = acc[mt][r];
      }
  }
}

// ---- down product for one 16-token tile (B <= 16, d_model % 256 == 0): one workgroup per
// (256-column tile, neuron range), the ranges' partials added by the reduce kernel in order.
// W_down is neuron-major, so the MFMA B operand (eight consecutive neurons of one column per
// lane) is gathered from LDS with 16-bit reads. Each 64-neuron block of the range -- its 64
// W_down rows over the tile's 256 columns (32 KiB, 512 bytes per row) and the hi/lo h
// fragments of the 16 tokens (4 KiB, already in A-operand lane order) -- is moved into one
// slot of a four-slot LDS ring by direct global-to-LDS loads: 36 KiB = 2304 16-byte pieces,
// four per thread of a 576-thread workgroup (eight MFMA waves and one wave that only loads),
// so three blocks are in flight. A W_down row's 16-byte chunk c sits at position
// c ^ 2 ((row / 8) % 4): the 16-bit gathers of one instruction (16 columns of four 8-row
// groups) then touch 32 different banks.
constexpr int kDrThreads = 576;
constexpr int kDrCols = 256;
constexpr int kDrRowBytes = kDrCols * 2;
constexpr int kDrWBytes = kDnChunk * kDrRowBytes;                   // 32 KiB
constexpr int kDrHBytes = 2 * kDnSteps * kWave * 16;                // 4 KiB
constexpr int kDrSlotBytes = kDrWBytes + kDrHBytes;                 // 36 KiB
constexpr int kDrLoads = kDrSlotBytes / 16 / kDrThreads;            // 4
static_assert(kDrLoads * kDrThreads * 16 == kDrSlotBytes, "whole loads per thread");
static_assert(kDrLoads == kRgLoads, "the ring wait counts assume four loads per block");
static_assert((kDrWBytes / 16) % kWave == 0, "every wave instruction is all W_down or all h");

__device__ __forceinline__ int dr_pos(int row, int chunk) { return chunk ^ (((row >> 3) & 3) << 1); }

__global__ __launch_bounds__(kDrThreads) void down_ring_kernel(
    const uint16_t* __restrict__ hhi, const uint16_t* __restrict__ hlo, int F16,
    const uint16_t* __restrict__ wd, int d, int F, int B, int nchunk, int gr,
    float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) unsigned char s_d0[kDrSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_d1[kDrSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_d2[kDrSlotBytes];
  __shared__ __attribute__((aligned(16))) unsigned char s_d3[kDrSlotBytes];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  // workgroups go to the eight XCDs in turn (id % 8); when the grid divides evenly, XCD j takes
  // the consecutive (tile, range) indices [j N / 8, (j + 1) N / 8), so the column tiles of a
  // neuron range share one L2 and its h fragments are fetched from HBM once
  const int ncols = d / kDrCols, N = ncols * gr;
  const int L = blockIdx.x;
  const int idx = (N % 8 == 0) ? (L % 8) * (N / 8) + L / 8 : L;
  const int c0 = (idx % ncols) * kDrCols, rho = idx / ncols;
  const int ch_lo = (int)(((long long)nchunk * rho) / gr);
  const int nblk = (int)(((long long)nchunk * (rho + 1)) / gr) - ch_lo;

  // this thread's loads of a block: slot piece g = q * 576 + tid. Pieces below 2048 are W_down
  // row g / 32 (of the block's 64), position g % 32, holding chunk dr_pos(row, position) of
  // the tile's columns; the rest are h fragment (which, step, lane) = (hg / 128, hg / 64 % 2,
  // hg % 64): token lane % 16, neurons 32 step + 8 (lane / 16) .. + 7 of the block.
  const uint16_t* src[kDrLoads];
  size_t stride[kDrLoads];  // elements to the same piece of the next block
  bool wpiece[kDrLoads];
  int lds_off[kDrLoads];
#pragma unroll
  for (int q = 0; q < kDrLoads; ++q) {
    const int g = q * kDrThreads + tid;
    const int g0 = __builtin_amdgcn_readfirstlane(q * kDrThreads + wave * kWave);
    wpiece[q] = g0 < kDrWBytes / 16;
    if (wpiece[q]) {
      const int r = g >> 5, c = dr_pos(r, g & 31);
      // rows past d_ff read row d_ff - 1 (finite); their h is 0 (F16 is a multiple of 64)
      const int n = min(ch_lo * kDnChunk + r, F - 1);
      src[q] = wd + (size_t)n * d + c0 + 8 * c;
      stride[q] = (size_t)kDnChunk * d;
    } else {
      const int hg = g - kDrWBytes / 16;
      const int which = hg >> 7, st = (hg >> 6) & 1, l = hg & 63;
      src[q] = (which ? hlo : hhi) + (size_t)(l & 15) * F16 + ch_lo * kDnChunk + 32 * st + 8 * (l >> 4);
      stride[q] = kDnChunk;
    }
    lds_off[q] = (q * kDrThreads + wave * kWave) * 16;
  }
  auto issue = [&](unsigned char* slot, int b) {
#pragma unroll
    for (int q = 0; q < kDrLoads; ++q) {
      const uint16_t* gp = src[q] + (size_t)b * stride[q];
      auto* lp = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<size_t>(slot + lds_off[q]));
      if (wpiece[q]) {
        // a W_down row past d_ff stays at row d_ff - 1 in every block
        const uint16_t* gw = gp;
        if (ch_lo * kDnChunk + b * kDnChunk + ((q * kDrThreads + tid) >> 5) >= F)
          gw = wd + (size_t)(F - 1) * d + (src[q] - wd) % d;
        __builtin_amdgcn_global_load_lds(gw, lp, 16, 0, 2);
      } else {
        __builtin_amdgcn_global_load_lds(gp, lp, 16, 0, 0);
      }
    }
  };

  const int nb = lane & 15, gq = lane >> 4;
  floatx4_t acc[2] = {floatx4_t{0.f, 0.f, 0.f, 0.f}, floatx4_t{0.f, 0.f, 0.f, 0.f}};
  auto compute = [&](const unsigned char* slot) {
    if (wave >= 8) return;  // the load-only wave
#pragma unroll
    for (int st = 0; st < kDnSteps; ++st) {
      const bf16x8_t ahi = as_bf16x8(*reinterpret_cast<const uint4*>(slot + kDrWBytes + 16 * (st * kWave + lane)));
      const bf16x8_t alo = as_bf16x8(*reinterpret_cast<const uint4*>(slot + kDrWBytes + 16 * ((kDnSteps + st) * kWave + lane)));
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = 32 * wave + 16 * j + nb;
        uint32_t bw[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int r0 = 32 * st + 8 * gq + 2 * jj, r1 = r0 + 1;
          const uint32_t e0 = *reinterpret_cast<const uint16_t*>(
              slot + r0 * kDrRowBytes + 16 * dr_pos(r0, col >> 3) + 2 * (col & 7));
          const uint32_t e1 = *reinterpret_cast<const uint16_t*>(
              slot + r1 * kDrRowBytes + 16 * dr_pos(r1, col >> 3) + 2 * (col & 7));
          bw[jj] = e0 | (e1 << 16);
        }
        const bf16x8_t bop = as_bf16x8(make_uint4(bw[0], bw[1], bw[2], bw[3]));
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bop, acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bop, acc[j], 0, 0, 0);
      }
    }
  };
  auto step = [&](unsigned char* slot, unsigned char* refill, int b) {
    const int later = min(2, nblk - 1 - b);
    if (later >= 2) wait_vm<2 * kDrLoads>();
    else if (later == 1) wait_vm<kDrLoads>();
    else wait_vm<0>();
    ring_barrier();
    if (b + 3 < nblk) issue(refill, b + 3);
    compute(slot);
  };
  if (nblk > 0) issue(s_d0, 0);
  if (nblk > 1) issue(s_d1, 1);
  if (nblk > 2) issue(s_d2, 2);
  for (int b = 0; b < nblk; b += 4) {
    step(s_d0, s_d3, b);
    if (b + 1 < nblk) step(s_d1, s_d0, b + 1);
    if (b + 2 < nblk) step(s_d2, s_d1, b + 2);
    if (b + 3 < nblk) step(s_d3, s_d2, b + 3);
  }

  // C layout: lane holds column c0 + 32 wave + 16 j + lane % 16 and tokens 4 (lane / 16) + r
  if (wave < 8) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = c0 + 32 * wave + 16 * j + nb;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 4 * gq + r;
        if (m < B && c < d) part[((size_t)rho * B + m) * d + c] = acc[j][r];
      }
    }
  }
}

}  // namespace

MfmaLayout mfma_layout(int B, int d, int F) {
  MfmaLayout L{};
  L.mpad = ceil_div(B, kMTile) * kMTile;
  // h rows padded to whole 64-neuron down blocks (h = 0 past d_ff)
  L.ntiles = ceil_div(F, kDnChunk) * (kDnChunk / kMTile);
  L.f16 = L.ntiles * kMTile;
  L.cs = ceil_div(d, kDnCols);
  L.nchunk = ceil_div(F, kDnChunk);
  L.gr = std::max(1, std::min(L.nchunk, kDnTarget / L.cs));
  Carve c;
  L.xb = c.take((size_t)L.mpad * d * 2);
  L.hhi = c.take((size_t)L.mpad * L.f16 * 2);
  L.hlo = c.take((size_t)L.mpad * L.f16 * 2);
  L.part = c.take((size_t)L.gr * B * d * 4);
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_mfma(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, float norm_eps, const float* resid,
                           float* y, char* ws, const MfmaLayout& L, hipStream_t stream) {
  if (B < 1 || B > kMaxMTiles * kMTile || L.mpad != ceil_div(B, kMTile) * kMTile)
    return hipErrorInvalidValue;
  hipError_t e;
  uint16_t* xb = reinterpret_cast<uint16_t*>(ws + L.xb);
  uint16_t* hhi = reinterpret_cast<uint16_t*>(ws + L.hhi);
  uint16_t* hlo = reinterpret_cast<uint16_t*>(ws + L.hlo);
  float* part = reinterpret_cast<float*>(ws + L.part);
  const int mt = L.mpad / kMTile;
  {
    ProfScope prof("ffn_mfma_prep", stream);
    klaunch(prep_x_kernel, L.mpad, 256, 0, stream, x, B, d, norm_eps, xb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    ProfScope prof("ffn_mfma_gate_up", stream);
    // one 16-token tile with d_model a multiple of 128 and at most 56 neurons per segment
    // (d_ff <= 14336 over 256 segments): the LDS-ring kernel; otherwise 8 neurons per workgroup
    const int rg_seg = std::min(256, L.f16 / 8);
    const int rg_np = ceil_div(L.f16, rg_seg);
    if (mt == 1 && d % kRgK == 0 && rg_np <= kRgMaxNeurons) {
      klaunch(gate_up_ring_kernel, ceil_div(L.f16, rg_np), kRgThreads, 0, stream, xb, wg, wu, d, F,
              L.f16, rg_np, hhi, hlo);
    } else {
      const dim3 grid(L.f16 / kGuRows);  // every row below F16 is written (0 past d_ff)
#define SIRIUS_GU(MTV)                                                                       \
  case MTV:                                                                                  \
    klaunch(gate_up_kernel<MTV>, grid, 128, 0, stream, xb, wg, wu, d, F, L.f16, hhi, hlo);        \
    break;
      switch (mt) {
        SIRIUS_GU(1)
        SIRIUS_GU(2)
        SIRIUS_GU(3)
        SIRIUS_GU(4)
        default:
          return hipErrorInvalidValue;
      }
#undef SIRIUS_GU
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (mt == 1 && d % kDrCols == 0) {
    // one 16-token tile: the LDS-ring down kernel, same partial layout
    ProfScope prof("ffn_mfma_down", stream);
    klaunch(down_ring_kernel, (d / kDrCols) * L.gr, kDrThreads, 0, stream, hhi, hlo, L.f16, wd, d, F,
            B, L.nchunk, L.gr, part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else {
    ProfScope prof("ffn_mfma_down", stream);
    const dim3 grid(L.cs, L.gr);
#define SIRIUS_DN(MTV)                                                                        \
  case MTV:                                                                                   \
    klaunch(down_kernel<MTV>, grid, 256, 0, stream, hhi, hlo, L.f16, wd, d, F, B, L.nchunk, part); \
    break;
    switch (mt) {
      SIRIUS_DN(1)
      SIRIUS_DN(2)
      SIRIUS_DN(3)
      SIRIUS_DN(4)
      default:
        return hipErrorInvalidValue;
    }
#undef SIRIUS_DN
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  ProfScope prof("ffn_mfma_reduce", stream);
  return launch_reduce(part, L.gr, B, d, resid, y, stream);
}

}  // namespace sirius
