// Order of neurons for per-token top-k sparsity: larger |a| first, then the lower neuron
// index, as one 64-bit key (the bits of |a| order like its value; the complemented index
// breaks ties). Keys of one token are distinct, so the k-th largest key cuts exactly k.
#pragma once

#include <hip/hip_runtime.h>

namespace sirius {

__device__ __forceinline__ unsigned long long topk_key(float a, int i) {
  return ((unsigned long long)__float_as_uint(fabsf(a)) << 32) | (unsigned)(~(unsigned)i);
}

}  // namespace sirius
