// Helpers of the softmax statistics kept by the verify and tree kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace sirius {

// 2^x for x <= 0 with the hardware instruction (about 1 ulp). Results below the smallest
// normal float flush to zero: such a term is under 2^-126 of the largest term of its sum, far
// below that sum's rounding.
__device__ __forceinline__ float exp2_nonpos(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace sirius
