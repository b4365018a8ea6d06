// Device helpers shared by the scan kernels and the fused projection + scan.
#pragma once

#include <hip/hip_runtime.h>

namespace sru {

// 1 / (1 + e^{-z}) (Eq. 1, 3); saturates to exactly 0 (e^{-z} = inf) and 1
// (e^{-z} underflows) instead of producing NaN.
__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

}  // namespace sru
