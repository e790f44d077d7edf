// Matrix-core throughput probe for the benchmark's measured-peak figure. It is
// built into its own library (libmte_probe.so), not into libmte: it measures
// the chip, it is no part of the encoder.
//
// Every wave runs `iters` rounds of eight independent v_mfma_f32_32x32x16_f16
// (no memory traffic inside the loop), so the kernel's duration gives the
// dense fp16 MFMA rate the chip sustains at the clock it actually runs under
// that load.
//
//   int mte_probe_mfma(int32_t blocks, int32_t iters, float *sink, hipStream_t stream);
//
// Enqueues `blocks` workgroups of four waves on `stream`; every wave does
// iters * 8 MFMAs of 32768 flops. sink: device float[blocks * 256], one value
// per thread, overwritten. Returns 0, -1 for a null sink or non-positive
// blocks / iters (checked before any HIP call), -3 if the launch fails.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
constexpr int kProbeChains = 8;

__global__ __launch_bounds__(256) void k_mfma_probe(int iters, float *sink) {
  const int lane = threadIdx.x & 63;
  f16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(0.001f * (lane + e));
    b[e] = (_Float16)(0.002f * (lane - e));
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

}  // namespace

extern "C" int mte_probe_mfma(int32_t blocks, int32_t iters, float *sink, hipStream_t stream) {
  if (!sink || blocks <= 0 || iters <= 0) return -1;
  hipLaunchKernelGGL(k_mfma_probe, dim3(blocks), dim3(256), 0, stream, iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
