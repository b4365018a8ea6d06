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

// The v/b gradient sums of one block of 256 threads: 64 consecutive outputs
// o = qlo * nfeat + 64 * blk + lane (q = o / nfeat selects dv_f, dv_r, db_f,
// db_r).  Wave w adds rows b = w, w + 4, ... in order, and the four wave sums
// meet in a fixed tree through `red` (256 floats of LDS), so the result does
// not depend on the launch that runs the block.  Called by all 256 threads.
__device__ __forceinline__ void vb_sum_block(const float* __restrict__ partial, int rows,
                                             int nfeat, int qlo, float* const (&out)[4],
                                             int blk, float* red) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int o = qlo * nfeat + blk * 64 + lane;
  const bool live = o < 4 * nfeat;
  const long long stride = 4LL * nfeat;
  float s = 0.f;
  if (live) {
    const float* p = partial + o;
#pragma unroll 8
    for (int b = w; b < rows; b += 4) s += p[b * stride];
  }
  red[w * 64 + lane] = s;
  __syncthreads();
  if (w == 0 && live) {
    const float t = (red[lane] + red[64 + lane]) + (red[128 + lane] + red[192 + lane]);
    const int q = o / nfeat;
    out[q][o - q * nfeat] = t;
  }
}

}  // namespace sru
