// Row-wise kernels of the vision tower: patch extraction in merge-group
// order, LayerNorm, and the (row, column) positions of the patches.
#include "common.h"
#include "launch.h"

namespace mte {

// Patch p of image n (merge-group order: groups of merge x merge patches
// row-major over the image, patches row-major inside a group) sits at patch
// row ph = merge*gr + dr, column pw = merge*gc + dc. Its vector is the
// image's pixels under it in (channel, row, column) order, the flattening
// of a Conv2d weight [hidden, C, patch, patch].
struct PatchGeom {
  int C, H, W, patch, merge;
  int gw;            // merge groups per row: W / (patch * merge)
  int per_image;     // patches per image
};

__device__ __forceinline__ void patch_rc(const PatchGeom &g, int p, int &ph, int &pw) {
  const int mm = g.merge * g.merge;
  const int grp = p / mm, in = p % mm;
  ph = g.merge * (grp / g.gw) + in / g.merge;
  pw = g.merge * (grp % g.gw) + in % g.merge;
}

template <typename TI, typename TO>
__global__ __launch_bounds__(256) void k_patchify(const TI *__restrict__ px, TO *__restrict__ out, PatchGeom g,
                                                  size_t total) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int K = g.C * g.patch * g.patch;
  const size_t row = i / K;
  const int k = (int)(i % K);
  const int n = (int)(row / g.per_image), p = (int)(row % g.per_image);
  int ph, pw;
  patch_rc(g, p, ph, pw);
  const int c = k / (g.patch * g.patch), ky = (k / g.patch) % g.patch, kx = k % g.patch;
  const size_t src = (((size_t)n * g.C + c) * g.H + (size_t)ph * g.patch + ky) * g.W + (size_t)pw * g.patch + kx;
  out[i] = from_f32<TO>(to_f32(px[src]));
}

hipError_t launch_patchify(int in_fmt, const void *pixels, int n, int C, int H, int W, int patch, int merge,
                           int out_fmt, void *out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (H % (patch * merge) || W % (patch * merge)) return hipErrorInvalidValue;
  PatchGeom g{C, H, W, patch, merge, W / (patch * merge), (H / patch) * (W / patch)};
  const size_t total = (size_t)n * g.per_image * C * patch * patch;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (in_fmt == FMT_BF16 && out_fmt == FMT_F16)
    hipLaunchKernelGGL((k_patchify<bf16, f16>), grid, dim3(256), 0, s, (const bf16 *)pixels, (f16 *)out, g, total);
  else if (in_fmt == FMT_F32 && out_fmt == FMT_F32)
    hipLaunchKernelGGL((k_patchify<float, float>), grid, dim3(256), 0, s, (const float *)pixels, (float *)out, g,
                       total);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// pos [3, T]: t = 0, h = patch row, w = patch column of every patch.
__global__ __launch_bounds__(256) void k_patch_positions(int32_t *__restrict__ pos, int T, PatchGeom g) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= T) return;
  int ph, pw;
  patch_rc(g, i % g.per_image, ph, pw);
  pos[i] = 0;
  pos[T + i] = ph;
  pos[2 * T + i] = pw;
}

hipError_t launch_patch_positions(int32_t *pos, int n, int H, int W, int patch, int merge, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  PatchGeom g{0, H, W, patch, merge, W / (patch * merge), (H / patch) * (W / patch)};
  const int T = n * g.per_image;
  hipLaunchKernelGGL(k_patch_positions, dim3((T + 255) / 256), dim3(256), 0, s, pos, T, g);
  return hipGetLastError();
}

// LayerNorm of one row per 256-thread block: y = (x - mean) / sqrt(var + eps)
// * g + b, mean and (biased) variance over the D values, two passes over
// values held in registers (D <= 256 * kLnPer).
constexpr int kLnPer = 16;

template <typename TO>
__global__ __launch_bounds__(256) void k_layernorm(const float *__restrict__ x, const float *__restrict__ g,
                                                   const float *__restrict__ b, TO *__restrict__ y, int D,
                                                   float eps) {
  __shared__ float red[4];
  const float *xr = x + (size_t)blockIdx.x * D;
  float v[kLnPer];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kLnPer; ++k) {
    const int c = threadIdx.x + 256 * k;
    v[k] = c < D ? xr[c] : 0.f;
    s += v[k];
  }
  auto block_sum = [&](float t) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) t = warp_sum_xor(t, m);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
    __syncthreads();
    return (red[0] + red[1]) + (red[2] + red[3]);
  };
  const float mean = block_sum(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < kLnPer; ++k) {
    const int c = threadIdx.x + 256 * k;
    const float d = c < D ? v[k] - mean : 0.f;
    q += d * d;
  }
  const float rs = rsqrtf(block_sum(q) / (float)D + eps);
  TO *yr = y + (size_t)blockIdx.x * D;
#pragma unroll
  for (int k = 0; k < kLnPer; ++k) {
    const int c = threadIdx.x + 256 * k;
    if (c < D) yr[c] = from_f32<TO>((v[k] - mean) * rs * g[c] + b[c]);
  }
}

// The same with one wave per row (four rows per block) for D a multiple of
// 256: each lane holds NV 16-byte groups of the row (coalesced loads), and
// both reductions stay inside the wave.
template <typename TO, int NV>
__global__ __launch_bounds__(256) void k_layernorm_wave(const float *__restrict__ x, const float *__restrict__ g,
                                                        const float *__restrict__ b, TO *__restrict__ y, int rows,
                                                        int D, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float *xr = x + (size_t)row * D;
  f32x4 v[NV];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    v[k] = *(const f32x4 *)(xr + 4 * (lane + 64 * k));
    s += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s = warp_sum_xor(s, m);
  const float mean = s / (float)D;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float d = v[k][e] - mean;
      q += d * d;
    }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) q = warp_sum_xor(q, m);
  const float rs = rsqrtf(q / (float)D + eps);
  TO *yr = y + (size_t)row * D;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = 4 * (lane + 64 * k);
    const f32x4 gg = *(const f32x4 *)(g + c), bb = *(const f32x4 *)(b + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) yr[c + e] = from_f32<TO>((v[k][e] - mean) * rs * gg[e] + bb[e]);
  }
}

template <typename TO>
static bool layernorm_wave(const float *x, const float *g, const float *b, TO *y, int rows, int D, float eps,
                           hipStream_t s) {
  const dim3 grid((rows + 3) / 4);
  switch (D / 256) {
#define MTE_LN(nv) case nv: hipLaunchKernelGGL((k_layernorm_wave<TO, nv>), grid, dim3(256), 0, s, x, g, b, y, rows, D, eps); return true;
    MTE_LN(1) MTE_LN(2) MTE_LN(3) MTE_LN(4) MTE_LN(6) MTE_LN(8) MTE_LN(12) MTE_LN(16)
#undef MTE_LN
  }
  return false;
}

hipError_t launch_layernorm(const float *x, const float *g, const float *b, int out_fmt, void *y, int rows, int D,
                            float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (D > 256 * kLnPer) return hipErrorInvalidValue;
  if (D % 256 == 0 && ((uintptr_t)x | (uintptr_t)g | (uintptr_t)b) % 16 == 0) {
    const bool ok = out_fmt == FMT_F16 ? layernorm_wave(x, g, b, (f16 *)y, rows, D, eps, s)
                    : out_fmt == FMT_F32 ? layernorm_wave(x, g, b, (float *)y, rows, D, eps, s)
                                         : false;
    if (ok) return hipGetLastError();
  }
  if (out_fmt == FMT_F16)
    hipLaunchKernelGGL(k_layernorm<f16>, dim3(rows), dim3(256), 0, s, x, g, b, (f16 *)y, D, eps);
  else if (out_fmt == FMT_F32)
    hipLaunchKernelGGL(k_layernorm<float>, dim3(rows), dim3(256), 0, s, x, g, b, (float *)y, D, eps);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// dst row (r / group) * group_stride + r % group = src row r (float src,
// dst FMT_F32 or FMT_BF16 rounded to nearest even); other dst rows untouched.
template <typename TD>
__global__ __launch_bounds__(256) void k_scatter_rows(const float *__restrict__ src, TD *__restrict__ dst, int cols,
                                                      int group, int group_stride) {
  const int r = blockIdx.x;
  const size_t dr = (size_t)(r / group) * group_stride + r % group;
  const float *sr = src + (size_t)r * cols;
  TD *d = dst + dr * cols;
  for (int c = threadIdx.x; c < cols; c += 256) d[c] = from_f32<TD>(sr[c]);
}

hipError_t launch_scatter_rows(const float *src, int dst_fmt, void *dst, int rows, int cols, int group,
                               int group_stride, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (group <= 0 || group_stride < group) return hipErrorInvalidValue;
  if (dst_fmt == FMT_F32)
    hipLaunchKernelGGL(k_scatter_rows<float>, dim3(rows), dim3(256), 0, s, src, (float *)dst, cols, group,
                       group_stride);
  else if (dst_fmt == FMT_BF16)
    hipLaunchKernelGGL(k_scatter_rows<bf16>, dim3(rows), dim3(256), 0, s, src, (bf16 *)dst, cols, group,
                       group_stride);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace mte
