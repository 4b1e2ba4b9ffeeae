// Radix select of the k-th largest of n non-negative fp32 values on gfx950.
//
// Non-negative IEEE floats order like their bit patterns, so the k-th largest
// is found one byte at a time, most significant first: a grid-wide histogram
// of the current byte over the values that match the bytes already fixed
// (LDS histograms merged with integer atomics, so the counts are exact),
// then a one-thread pass that fixes the next byte. Four rounds give the exact
// value. Used by the threshold calibration and by the prompt top-k.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace sirius {
namespace {

struct SelectState {
  uint32_t prefix;  // bytes fixed so far
  uint32_t mask;    // which bits of prefix are fixed
  int rem;          // rank still to find among the matching values
  int pad;
};

constexpr int kHistBlocks = 512;

__global__ void select_init_kernel(SelectState* st, int k, int* ghist) {
  const int t = threadIdx.x;
  if (t < 256) ghist[t] = 0;
  if (t == 0) {
    st->prefix = 0u;
    st->mask = 0u;
    st->rem = k;
  }
}

__global__ __launch_bounds__(256) void select_hist_kernel(const float* __restrict__ v, int n,
                                                          int shift, const SelectState* st,
                                                          int* ghist) {
  __shared__ int h[256];
  const uint32_t prefix = st->prefix, mask = st->mask;
  h[threadIdx.x] = 0;
  __syncthreads();
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const uint32_t u = __float_as_uint(v[i]);
    if ((u & mask) == prefix) atomicAdd(&h[(u >> shift) & 255u], 1);
  }
  __syncthreads();
  const int c = h[threadIdx.x];
  if (c != 0) atomicAdd(&ghist[threadIdx.x], c);
}

__global__ void select_pick_kernel(int shift, SelectState* st, int* ghist, float* out_value) {
  __shared__ int h[256];
  h[threadIdx.x] = ghist[threadIdx.x];
  ghist[threadIdx.x] = 0;  // ready for the next round
  __syncthreads();
  if (threadIdx.x == 0) {
    int rem = st->rem;
    int dsel = 0;
    for (int dg = 255; dg >= 0; --dg) {
      const int c = h[dg];
      if (c >= rem) {
        dsel = dg;
        break;
      }
      rem -= c;
    }
    st->rem = rem;
    st->prefix |= (uint32_t)dsel << shift;
    st->mask |= 255u << shift;
    if (shift == 0) out_value[0] = __uint_as_float(st->prefix);
  }
}

}  // namespace

size_t select_ws_bytes() { return 256 + 256 * sizeof(int); }

hipError_t launch_select_kth_largest(const float* v, int n, int k, float* out_value, char* ws,
                                     hipStream_t stream) {
  SelectState* st = reinterpret_cast<SelectState*>(ws);
  int* ghist = reinterpret_cast<int*>(ws + 256);
  {
    ProfScope prof("select_init", stream);
    klaunch(select_init_kernel, 1, 256, 0, stream, st, k, ghist);
  }
  const int blocks = std::max(1, std::min(kHistBlocks, ceil_div(n, 256 * 8)));
  for (int shift = 24; shift >= 0; shift -= 8) {
    {
      ProfScope prof("select_hist", stream);
      klaunch(select_hist_kernel, blocks, 256, 0, stream, v, n, shift, st, ghist);
    }
    ProfScope prof("select_pick", stream);
    klaunch(select_pick_kernel, 1, 256, 0, stream, shift, st, ghist, out_value);
  }
  return hipGetLastError();
}

}  // namespace sirius
