// Multi-token SwiGLU FFN gate/up products on MFMA (gfx950), for batches of 8..64 tokens:
// the full model's parallel pass over a drafted chunk, and condensed / dense decode of
// batched tokens.
//
//  mfma_gate_up_kernel  h[m, n] = SiLU(x_m . W_gate[n]) * (x_m . W_up[n]) with
//                       v_mfma_f32_16x16x32_bf16 (x rounded to bf16, exact products,
//                       fp32 accumulation). A wave owns 16 neurons and streams their
//                       W_gate and W_up rows straight into MFMA operand registers, 256 K
//                       elements per block and 8 MFMA steps per block. Two waves split the K
//                       blocks of one neuron tile and are summed in a fixed order. h is
//                       written in the compacted-list layout of the small-batch path (every
//                       neuron kept, tiles of 16), so the same row-split down projection and
//                       fixed-order reduce finish the FFN.
//
// The pass is HBM-bound (3 * d_ff * d_model * 2 bytes against ~6 * B * d_ff * d_model
// flops), so MFMA is used for the contraction and nothing more elaborate is needed.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;

constexpr int kMTile = 16;      // MFMA M (tokens) and N (neurons) tile
constexpr int kKBlock = 256;    // K elements per block: 4 lane groups x 64
constexpr int kMaxMTiles = 4;   // batch <= 64

// 8 fp32 -> 8 bf16 (round to nearest even), zero when out of range
__device__ __forceinline__ bf16x8_t load_x8(const float* x, int m, int B, int d, int k) {
  uint4 r = make_uint4(0u, 0u, 0u, 0u);
  if (m < B && k < d) {
    const float4 a = *reinterpret_cast<const float4*>(x + (size_t)m * d + k);
    const float4 b = *reinterpret_cast<const float4*>(x + (size_t)m * d + k + 4);
    r.x = f32_to_bf16(a.x) | (f32_to_bf16(a.y) << 16);
    r.y = f32_to_bf16(a.z) | (f32_to_bf16(a.w) << 16);
    r.z = f32_to_bf16(b.x) | (f32_to_bf16(b.y) << 16);
    r.w = f32_to_bf16(b.z) | (f32_to_bf16(b.w) << 16);
  }
  return __builtin_bit_cast(bf16x8_t, r);
}

template <int MT>
__global__ __launch_bounds__(256) void mfma_gate_up_kernel(
    const float* __restrict__ x, int B, const uint16_t* __restrict__ wg,
    const uint16_t* __restrict__ wu, int d, int F, int32_t* __restrict__ uidx,
    float* __restrict__ hbuf, int32_t* __restrict__ ucnt) {
  __shared__ floatx4_t s_acc[2][MT][2][kWave];  // [neuron tile][m tile][gate/up][lane]
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int ntile = blockIdx.x * 2 + (wave >> 1);  // two neuron tiles per workgroup
  const int khalf = wave & 1;                      // waves 0/1 and 2/3 split the K blocks
  const int n0 = ntile * kMTile;
  const int fr = lane & 15, grp = lane >> 4;  // fragment row, lane group
  const int row = n0 + fr;
  const bool rv = row < F;
  const uint16_t* wgr = wg + (size_t)row * d;
  const uint16_t* wur = wu + (size_t)row * d;

  floatx4_t accg[MT], accu[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    accg[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    accu[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }
  const int nblk = (d + kKBlock - 1) / kKBlock;
  for (int blk = khalf; blk < nblk; blk += 2) {
    // step i covers K elements [32 i, 32 i + 32) of the block, lane group grp the 8 at 8 grp:
    // the four lanes of a row read 64 contiguous bytes, steps 2j and 2j+1 a full 128-byte line
    const int kb = blk * kKBlock + 8 * grp;
    uint4 g8[8], u8[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = kb + 32 * i;
      const bool ok = rv && k < d;
      g8[i] = ok ? ld_stream(reinterpret_cast<const uint4*>(wgr + k)) : make_uint4(0u, 0u, 0u, 0u);
      u8[i] = ok ? ld_stream(reinterpret_cast<const uint4*>(wur + k)) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = kb + 32 * i;
      const bf16x8_t bg = __builtin_bit_cast(bf16x8_t, g8[i]);
      const bf16x8_t bu = __builtin_bit_cast(bf16x8_t, u8[i]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const bf16x8_t a = load_x8(x, mt * kMTile + fr, B, d, k);
        accg[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bg, accg[mt], 0, 0, 0);
        accu[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bu, accu[mt], 0, 0, 0);
      }
    }
  }

  // fixed-order sum of the two K halves, then the epilogue on the first wave of each pair
  const int pair = wave >> 1;
  if (khalf == 1) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      s_acc[pair][mt][0][lane] = accg[mt];
      s_acc[pair][mt][1][lane] = accu[mt];
    }
  }
  __syncthreads();
  if (khalf == 0 && n0 < F) {
    // C layout: lane holds neuron n0 + lane % 16 and tokens 4 * (lane / 16) + r of each m tile
    const int n = n0 + fr;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4_t og = s_acc[pair][mt][0][lane], ou = s_acc[pair][mt][1][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * kMTile + 4 * grp + r;
        if (n < F && m < B) {
          const float g = accg[mt][r] + og[r];
          const float u = accu[mt][r] + ou[r];
          hbuf[(size_t)n * B + m] = silu(g) * u;
        }
      }
    }
    if (lane < kMTile && n0 + lane < F) uidx[n0 + lane] = n0 + lane;
    if (lane == 0) ucnt[ntile] = min(kMTile, F - n0);
  }
}

}  // namespace

MfmaLayout mfma_layout(int B, int d, int F) {
  MfmaLayout L{};
  L.mpad = ceil_div(B, kMTile) * kMTile;
  L.ntiles = ceil_div(F, kMTile);
  L.cs = ceil_div(d / 8, kWave);
  L.gr = std::max(1, std::min(512 / L.cs, ceil_div(F, 32)));
  Carve c;
  L.xn = c.take((size_t)B * d * 4);
  L.uidx = c.take((size_t)L.ntiles * kMTile * 4);
  L.h = c.take((size_t)L.ntiles * kMTile * B * 4);
  L.ucnt = c.take((size_t)L.ntiles * 4);
  L.part = c.take((size_t)L.gr * std::min(B, 16) * d * 4);  // one 16-token down chunk
  L.total = c.off;
  return L;
}

hipError_t launch_ffn_mfma(const float* x, int B, const uint16_t* wg, const uint16_t* wu,
                           const uint16_t* wd, int d, int F, float norm_eps, const float* resid,
                           float* y, char* ws, const MfmaLayout& L, hipStream_t stream) {
  if (B < 1 || B > kMaxMTiles * kMTile) return hipErrorInvalidValue;
  hipError_t e;
  const float* xin = x;
  if (norm_eps >= 0.f) {  // RMSNorm once into the workspace, then the unnormalised path
    float* xn = reinterpret_cast<float*>(ws + L.xn);
    if ((e = launch_rmsnorm(x, B, d, norm_eps, xn, stream)) != hipSuccess) return e;
    xin = xn;
  }
  int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.uidx);
  float* hbuf = reinterpret_cast<float*>(ws + L.h);
  int32_t* ucnt = reinterpret_cast<int32_t*>(ws + L.ucnt);
  const dim3 grid(ceil_div(L.ntiles, 2));
  {
    ProfScope prof("ffn_mfma_gate_up", stream);
    switch (ceil_div(B, kMTile)) {
      case 1: mfma_gate_up_kernel<1><<<grid, 256, 0, stream>>>(xin, B, wg, wu, d, F, uidx, hbuf, ucnt); break;
      case 2: mfma_gate_up_kernel<2><<<grid, 256, 0, stream>>>(xin, B, wg, wu, d, F, uidx, hbuf, ucnt); break;
      case 3: mfma_gate_up_kernel<3><<<grid, 256, 0, stream>>>(xin, B, wg, wu, d, F, uidx, hbuf, ucnt); break;
      case 4: mfma_gate_up_kernel<4><<<grid, 256, 0, stream>>>(xin, B, wg, wu, d, F, uidx, hbuf, ucnt); break;
      default: return hipErrorInvalidValue;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // down projection and reduce in token chunks of at most 16 (the row-split down kernel keeps
  // 8 output columns per token per lane in registers)
  float* part = reinterpret_cast<float*>(ws + L.part);
  for (int b0 = 0; b0 < B; b0 += 16) {
    const int nb = std::min(16, B - b0);
    {
      ProfScope prof("ffn_mfma_down", stream);
      if ((e = launch_down(nb, d, L.ntiles, kMTile, L.gr, wd, uidx, hbuf + b0, B, ucnt, part,
                           stream)) != hipSuccess)
        return e;
    }
    ProfScope prof("ffn_mfma_reduce", stream);
    if ((e = launch_reduce(part, L.gr, nb, d, resid ? resid + (size_t)b0 * d : nullptr,
                           y + (size_t)b0 * d, stream)) != hipSuccess)
      return e;
  }
  return hipSuccess;
}

}  // namespace sirius
