// Matrix-core throughput probe: every wave runs `iters` rounds of eight
// independent v_mfma_f32_32x32x16_f16 (no memory traffic inside the loop), so
// the kernel's duration gives the dense fp16 MFMA rate the chip sustains at
// the clock it actually runs under that load.
#include "common.h"
#include "launch.h"

namespace mte {

constexpr int kProbeChains = 8;

__global__ __launch_bounds__(256) void k_mfma_probe(int iters, float *sink) {
  const int lane = threadIdx.x & 63;
  f16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (f16)(0.001f * (lane + e));
    b[e] = (f16)(0.002f * (lane - e));
  }
  f32x16 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  sink[blockIdx.x * 256 + threadIdx.x] = s;
}

hipError_t launch_mfma_probe(int blocks, int iters, float *sink, hipStream_t s) {
  if (blocks <= 0 || iters <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_mfma_probe, dim3(blocks), dim3(256), 0, s, iters, sink);
  return hipGetLastError();
}

}  // namespace mte
