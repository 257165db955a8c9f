// Diagnostics: the matrix cores' bf16 rate as one workload sees it, for the
// measured side of the roofline's peak.  Every wave runs `iters` rounds of
// back-to-back MFMAs on independent accumulators held in registers (no
// memory traffic inside the loop): 32 accumulators of v_mfma_f32_16x16x32_bf16
// or 8 of v_mfma_f32_32x32x16_bf16 (the same 128 accumulator registers), so
// no product waits for an earlier one.  The accumulators are summed into one
// float per thread at the end, so nothing is optimised away.
#include <hip/hip_runtime.h>

#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

template <bool WIDE>
__global__ __launch_bounds__(256) void k_mfma_rate(int iters, float* sink) {
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)(threadIdx.x & 63) + 0.125f * e);
    b[e] = (__bf16)(0.0625f * e - 0.25f);
  }
  float s = 0.f;
  if constexpr (WIDE) {
    f32x16 acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 8; ++i) s += acc[i][0] + acc[i][15];
  } else {
    f32x4 acc[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[i] = zero4();
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int i = 0; i < 32; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 32; ++i) s += acc[i][0] + acc[i][3];
  }
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

hipError_t launch_mfma_rate(bool wide, int blocks, int iters, float* sink, hipStream_t st) {
  if (wide)
    hipLaunchKernelGGL(k_mfma_rate<true>, dim3(blocks), dim3(256), 0, st, iters, sink);
  else
    hipLaunchKernelGGL(k_mfma_rate<false>, dim3(blocks), dim3(256), 0, st, iters, sink);
  return hipGetLastError();
}

}  // namespace tla
