// Shared device-side definitions for the gfx950 encoder kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mte {

typedef __bf16 bf16;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16;
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(f16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// float -> bf16 conversion rounds to nearest, ties to even (gfx950 v_cvt_pk_bf16_f32).
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }
// float -> fp16 rounds to nearest, ties to even (v_cvt_f16_f32).
template <> __device__ __forceinline__ f16 from_f32<f16>(float x) { return (f16)x; }

// A 16-byte per-lane MFMA operand fragment. For bf16 / fp16 it is one
// v_mfma_f32_32x32x16_{bf16,f16} operand (8 values, k-extent 16); for f32 it is four
// v_mfma_f32_32x32x2_f32 operands (one value each, k-extent 8 in total).
// In both cases lane l supplies row (l % 32) and k-slot group (l / 32); A and
// B fragments use the same (group, element) -> k assignment, so the dot
// product is over the same k set whatever order the hardware sums it in.
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  typedef bf16x8 type;
  static constexpr int kElems = 8;
};
template <> struct Frag<f16> {
  typedef f16x8 type;
  static constexpr int kElems = 8;
};
template <> struct Frag<float> {
  typedef f32x4 type;
  static constexpr int kElems = 4;
};

__device__ __forceinline__ void mfma32(f32x16 &acc, const bf16x8 &a, const bf16x8 &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma32(f32x16 &acc, const f16x8 &a, const f16x8 &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma32(f32x16 &acc, const f32x4 &a, const f32x4 &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], acc, 0, 0, 0);
}

// Accumulator layout of a 32x32 MFMA tile: register r of lane l holds
// row 8*(r/4) + 4*(l/32) + (r%4), column l%32.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

__device__ __forceinline__ float warp_max_xor(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, kWave));
}
__device__ __forceinline__ float warp_sum_xor(float v, int mask) {
  return v + __shfl_xor(v, mask, kWave);
}

// Waits until at most n vector-memory operations of this wave are pending.
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 0xF) | (0x7 << 4) | (0xF << 8) | ((n >> 4) << 14));
}
// The same, and until every LDS access of this wave has completed.
template <int n>
__device__ __forceinline__ void wait_vm_lds0() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 0xF) | (0x7 << 4) | (0x0 << 8) | ((n >> 4) << 14));
}

// 16-byte global -> LDS copy without a register round trip: lane i of the
// wave writes lds_base + 16*i, lds_base wave-uniform. Written as inline asm
// on purpose: the compiler's waitcnt pass treats the builtin form as LDS
// traffic and then drains every outstanding LDS read (lgkmcnt(0)) before
// the MFMAs that follow a stage's loads. The asm form is invisible to that
// pass; the kernel orders these loads itself with explicit vmcnt waits and
// barriers, and waits for all of them before it ends.
// The source is a wave-uniform base (SGPRs) plus a 32-bit lane offset, so
// each load needs one VGPR instead of a 64-bit address.
// M0 is saved and restored around the load (the compiler reserves it), and
// one wait state separates the M0 write from the load that reads it.
__device__ __forceinline__ void dma16(const void *base, uint32_t off, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(lds_base)
      : "memory");
}

}  // namespace mte
