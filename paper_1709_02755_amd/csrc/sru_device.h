// Device helpers shared by the scan kernels and the fused projection + scan.
#pragma once

#include <hip/hip_runtime.h>

namespace sru {

// 1 / (1 + e^{-z}) (Eq. 1, 3); saturates to exactly 0 (e^{-z} = inf) and 1
// (e^{-z} underflows) instead of producing NaN.
__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

// The same sigma given zs = -z log2(e): 1 / (1 + 2^zs).  The recurrences
// fold the factor into the operands of the fma that forms a gate's
// pre-activation (v * c + u + b), which takes a multiply off the chain that
// carries c from one step to the next.  Saturates like sigmoid_fast.
constexpr float kNegLog2e = -1.44269504088896341f;
__device__ __forceinline__ float sigmoid_scaled(float zs) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(zs));
}

}  // namespace sru
