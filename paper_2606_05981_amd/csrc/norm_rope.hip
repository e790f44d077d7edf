// Row-wise kernels of the encoder: RMSNorm, per-head QK-norm + multimodal
// rotary embedding, on-device position ids, and the weight repacking used
// at encoder creation.
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace mte {

// ------------------------------------------------------------- RMSNorm
// out = x / sqrt(mean(x^2) + eps) * g, one 256-thread block per row, where
// x = in + the np partial sums parts[0..np) (pitch pstride elements), added
// in that order. copy_to (may alias in) receives x as float. OUT_FMT:
// FMT_F32, FMT_BF16 or FMT_F16 (rounded to nearest even).
struct Parts {
  const float *p;   // partial sums [np][rows, D]
  int np;           // 0 .. kMaxParts
  size_t stride;    // elements between two partial sums
};
constexpr int kMaxParts = 8;

template <typename TI>
__device__ __forceinline__ float row_in(const TI *x, const Parts &pt, size_t o) {
  float v = to_f32(x[o]);
  for (int k = 0; k < pt.np; ++k) v += pt.p[(size_t)k * pt.stride + o];
  return v;
}

template <typename TI, int OUT_FMT>
__global__ __launch_bounds__(256) void k_rmsnorm(const TI *in, float *copy_to, Parts pt,
                                                 const float *__restrict__ gain, void *__restrict__ out,
                                                 int D, float eps) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const size_t rb = (size_t)row * D;
  float ss = 0.f;
  for (int c = tid; c < D; c += 256) {
    const float v = row_in(in, pt, rb + c);
    ss += v * v;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss = warp_sum_xor(ss, m);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float rs = rsqrtf((red[0] + red[1] + red[2] + red[3]) / (float)D + eps);
  for (int c = tid; c < D; c += 256) {
    const size_t o = rb + c;
    const float v = row_in(in, pt, o);   // same thread, same element: copy_to may alias in
    if (copy_to) copy_to[o] = v;
    const float y = v * rs * gain[c];
    if constexpr (OUT_FMT == FMT_F32) {
      ((float *)out)[o] = y;
    } else if constexpr (OUT_FMT == FMT_BF16) {
      ((bf16 *)out)[o] = (bf16)y;
    } else {
      ((f16 *)out)[o] = (f16)y;
    }
  }
}

template <typename TI>
static void rmsnorm_out(int out_fmt, dim3 grid, const TI *in, float *copy_to, const Parts &pt,
                        const float *g, void *out, int D, float eps, hipStream_t s) {
  if (out_fmt == FMT_F32)
    hipLaunchKernelGGL((k_rmsnorm<TI, FMT_F32>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
  else if (out_fmt == FMT_BF16)
    hipLaunchKernelGGL((k_rmsnorm<TI, FMT_BF16>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
  else
    hipLaunchKernelGGL((k_rmsnorm<TI, FMT_F16>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
}

// Register-resident variant for D a multiple of 1024 (D <= 4096): every
// thread owns NV groups of 4 consecutive values, read once with 16-byte (or
// 8-byte bf16) loads and written with vector stores.
template <typename TI, int OUT_FMT, int NV>
__global__ __launch_bounds__(256) void k_rmsnorm_vec(const TI *in, float *copy_to, Parts pt,
                                                     const float *__restrict__ gain, void *__restrict__ out,
                                                     int D, float eps) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const size_t rb = (size_t)row * D;
  f32x4 v[NV], gv[NV];
  float ss = 0.f;
  // Every load first (input, gains, then the partial sums), so that one
  // memory latency covers them all; then the adds, in split order.
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (i * 256 + tid) * 4;
    gv[i] = *(const f32x4 *)(gain + c);
    if constexpr (std::is_same<TI, float>::value) {
      v[i] = *(const f32x4 *)(in + rb + c);
    } else {
      const bf16x4 b = *(const bf16x4 *)(in + rb + c);
      v[i] = (f32x4){(float)b[0], (float)b[1], (float)b[2], (float)b[3]};
    }
  }
  f32x4 q[kMaxParts][NV];
#pragma unroll
  for (int k = 0; k < kMaxParts; ++k)
    if (k < pt.np)
#pragma unroll
      for (int i = 0; i < NV; ++i) q[k][i] = *(const f32x4 *)(pt.p + (size_t)k * pt.stride + rb + (i * 256 + tid) * 4);
#pragma unroll
  for (int k = 0; k < kMaxParts; ++k)
    if (k < pt.np)
#pragma unroll
      for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[i][e] += q[k][i][e];
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) ss += v[i][e] * v[i][e];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss = warp_sum_xor(ss, m);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float rs = rsqrtf((red[0] + red[1] + red[2] + red[3]) / (float)D + eps);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (i * 256 + tid) * 4;
    if (copy_to) *(f32x4 *)(copy_to + rb + c) = v[i];
    f32x4 y;
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = v[i][e] * rs * gv[i][e];
    if constexpr (OUT_FMT == FMT_F32) {
      *(f32x4 *)((float *)out + rb + c) = y;
    } else if constexpr (OUT_FMT == FMT_BF16) {
      bf16x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = (bf16)y[e];
      *(bf16x4 *)((bf16 *)out + rb + c) = h;
    } else {
      f16x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = (f16)y[e];
      *(f16x4 *)((f16 *)out + rb + c) = h;
    }
  }
}

template <typename TI, int NV>
static void rmsnorm_vec(int out_fmt, dim3 grid, const TI *in, float *copy_to, const Parts &pt,
                        const float *g, void *out, int D, float eps, hipStream_t s) {
  if (out_fmt == FMT_F32)
    hipLaunchKernelGGL((k_rmsnorm_vec<TI, FMT_F32, NV>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
  else if (out_fmt == FMT_BF16)
    hipLaunchKernelGGL((k_rmsnorm_vec<TI, FMT_BF16, NV>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
  else
    hipLaunchKernelGGL((k_rmsnorm_vec<TI, FMT_F16, NV>), grid, dim3(256), 0, s, in, copy_to, pt, g, out, D, eps);
}

template <typename TI>
static void rmsnorm_dispatch(int out_fmt, dim3 grid, const TI *in, float *copy_to, const Parts &pt,
                             const float *g, void *out, int D, float eps, hipStream_t s) {
  switch (D % 1024 == 0 ? D / 1024 : 0) {
    case 1: rmsnorm_vec<TI, 1>(out_fmt, grid, in, copy_to, pt, g, out, D, eps, s); break;
    case 2: rmsnorm_vec<TI, 2>(out_fmt, grid, in, copy_to, pt, g, out, D, eps, s); break;
    case 3: rmsnorm_vec<TI, 3>(out_fmt, grid, in, copy_to, pt, g, out, D, eps, s); break;
    case 4: rmsnorm_vec<TI, 4>(out_fmt, grid, in, copy_to, pt, g, out, D, eps, s); break;
    default: rmsnorm_out<TI>(out_fmt, grid, in, copy_to, pt, g, out, D, eps, s); break;
  }
}

hipError_t launch_rmsnorm(int in_fmt, int out_fmt, const void *in, float *copy_to, const float *parts,
                          int nparts, const float *g, void *out, int rows, int D, float eps,
                          hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (parts && nparts > kMaxParts) return hipErrorInvalidValue;
  dim3 grid(rows);
  const Parts pt{parts, parts ? nparts : 0, (size_t)rows * D};
  if (in_fmt == FMT_BF16)
    rmsnorm_dispatch<bf16>(out_fmt, grid, (const bf16 *)in, copy_to, pt, g, out, D, eps, s);
  else
    rmsnorm_dispatch<float>(out_fmt, grid, (const float *)in, copy_to, pt, g, out, D, eps, s);
  return hipGetLastError();
}

// h[r, c] += parts[0][r, c] + ... + parts[np-1][r, c], in that order.
__global__ __launch_bounds__(256) void k_resid_add(float *__restrict__ h, Parts pt, size_t n4) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  f32x4 v = ((const f32x4 *)h)[i];
  f32x4 q[kMaxParts];
#pragma unroll
  for (int k = 0; k < kMaxParts; ++k)
    if (k < pt.np) q[k] = ((const f32x4 *)(pt.p + (size_t)k * pt.stride))[i];
#pragma unroll
  for (int k = 0; k < kMaxParts; ++k)
    if (k < pt.np)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += q[k][e];
  ((f32x4 *)h)[i] = v;
}

hipError_t launch_resid_add(float *h, const float *parts, int nparts, int rows, int D, hipStream_t s) {
  const size_t n = (size_t)rows * D;
  if (n == 0 || nparts <= 0) return hipSuccess;
  if (nparts > kMaxParts || D % 4) return hipErrorInvalidValue;
  const Parts pt{parts, nparts, n};
  hipLaunchKernelGGL(k_resid_add, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0, s, h, pt, n / 4);
  return hipGetLastError();
}

// Grid (token, item block). Items are the token's rotary pairs, head-major
// (pair j of q/k head h is item h*d/2 + j; a head's d/2 items sit in one
// wave, so the per-head sum of squares of the QK-norm is a butterfly over
// those lanes), followed by its v elements. Every value is first summed
// from the partial sums (in split order).
__global__ __launch_bounds__(256) void k_qkv_parts(float *__restrict__ qkv, Parts pt, int Hq, int Hkv,
                                                   QkvEpi qe) {
  const int tok = blockIdx.x, tid = threadIdx.x;
  const int d = qe.hd, half = d >> 1;
  const int nh = Hq + Hkv, nqkv = (Hq + 2 * Hkv) * d;
  float *row = qkv + (size_t)tok * nqkv;
  const float *prow = pt.p + (size_t)tok * nqkv;
  auto ld = [&](int c) -> float {
    float q[kMaxParts];
#pragma unroll
    for (int k = 0; k < kMaxParts; ++k)
      if (k < pt.np) q[k] = prow[(size_t)k * pt.stride + c];
    float v = q[0];
#pragma unroll
    for (int k = 1; k < kMaxParts; ++k)
      if (k < pt.np) v += q[k];
    return v;
  };
  const int it = blockIdx.y * 256 + tid;
  if (it < nh * half) {
    const int h = it / half, j = it % half;
    const int c0 = h * d + j;
    // every load first (the pair's partial sums, gains and rotary table entry),
    // so that one memory latency covers them all
    float qa[kMaxParts], qb[kMaxParts];
#pragma unroll
    for (int k = 0; k < kMaxParts; ++k)
      if (k < pt.np) {
        qa[k] = prow[(size_t)k * pt.stride + c0];
        qb[k] = prow[(size_t)k * pt.stride + c0 + half];
      }
    const float *gn = (h < Hq) ? qe.qn : qe.kn;
    const float ga = qe.qn ? gn[j] : 1.f, gb = qe.qn ? gn[j + half] : 1.f;
    const float c = qe.rcos[(size_t)tok * half + j], s = qe.rsin[(size_t)tok * half + j];
    asm volatile("" ::"v"(ga), "v"(gb), "v"(c), "v"(s) : "memory");   // keeps these loads up here
    float u = qa[0], w = qb[0];
#pragma unroll
    for (int k = 1; k < kMaxParts; ++k)
      if (k < pt.np) {
        u += qa[k];
        w += qb[k];
      }
    if (qe.qn) {
      float ss = u * u + w * w;
      for (int m = half >> 1; m >= 1; m >>= 1) ss = warp_sum_xor(ss, m);
      const float rs = rsqrtf(ss / (float)d + qe.eps);
      u = u * rs * ga;
      w = w * rs * gb;
    }
    row[c0] = u * c - w * s;
    row[c0 + half] = w * c + u * s;
  } else if (it < nh * half + Hkv * d) {
    const int c = nh * d + (it - nh * half);
    row[c] = ld(c);
  }
}

// The same into the attention operand layout (qe.qk / qe.vt): one block per
// token of the padded range [0, 32 ceil(T / 32)); tokens past T only write
// their V^T entries, as zeros.
__global__ __launch_bounds__(256) void k_qkv_parts_h(Parts pt, int T, int Hq, int Hkv, QkvEpi qe) {
  const int tok = blockIdx.x, tid = threadIdx.x;
  const int d = qe.hd, half = d >> 1;
  const int nh = Hq + Hkv, nqkv = (Hq + 2 * Hkv) * d;
  const bool live = tok < T;
  const float *prow = pt.p + (size_t)min(tok, T - 1) * nqkv;
  auto ld = [&](int c) -> float {
    float q[kMaxParts];
#pragma unroll
    for (int k = 0; k < kMaxParts; ++k)
      if (k < pt.np) q[k] = prow[(size_t)k * pt.stride + c];
    float v = q[0];
#pragma unroll
    for (int k = 1; k < kMaxParts; ++k)
      if (k < pt.np) v += q[k];
    return v;
  };
  const int it = blockIdx.y * 256 + tid;
  if (it < nh * half) {
    if (!live) return;                           // block-uniform
    const int h = it / half, j = it % half;
    const int c0 = h * d + j;
    // every load first (the pair's partial sums, gains and rotary table entry),
    // so that one memory latency covers them all
    float qa[kMaxParts], qb[kMaxParts];
#pragma unroll
    for (int k = 0; k < kMaxParts; ++k)
      if (k < pt.np) {
        qa[k] = prow[(size_t)k * pt.stride + c0];
        qb[k] = prow[(size_t)k * pt.stride + c0 + half];
      }
    const float *gn = (h < Hq) ? qe.qn : qe.kn;
    const float ga = qe.qn ? gn[j] : 1.f, gb = qe.qn ? gn[j + half] : 1.f;
    const float c = qe.rcos[(size_t)tok * half + j], s = qe.rsin[(size_t)tok * half + j];
    asm volatile("" ::"v"(ga), "v"(gb), "v"(c), "v"(s) : "memory");   // keeps these loads up here
    float u = qa[0], w = qb[0];
#pragma unroll
    for (int k = 1; k < kMaxParts; ++k)
      if (k < pt.np) {
        u += qa[k];
        w += qb[k];
      }
    if (qe.qn) {
      float ss = u * u + w * w;
      for (int m = half >> 1; m >= 1; m >>= 1) ss = warp_sum_xor(ss, m);
      const float rs = rsqrtf(ss / (float)d + qe.eps);
      u = u * rs * ga;
      w = w * rs * gb;
    }
    const float pre = h < Hq ? qe.q_pre : qe.k_pre;
    f16 *row = qe.qk + (size_t)tok * nh * d;
    row[c0] = (f16)((u * c - w * s) * pre);
    row[c0 + half] = (f16)((w * c + u * s) * pre);
  } else if (it < nh * half + Hkv * d) {
    const int dv = it - nh * half;
    const float v = live ? ld(nh * d + dv) * qe.v_pre : 0.f;
    // position of the token in its tile's fragment order
    const int t = tok & 31, i = 4 * (t >> 3) + (t & 3);
    const int pos = 16 * (i >> 3) + 8 * ((t >> 2) & 1) + (i & 7);
    qe.vt[(((size_t)(tok >> 5) * Hkv + dv / d) * d + dv % d) * 32 + pos] = (f16)v;
  }
}

hipError_t launch_qkv_parts(float *qkv, const float *parts, int nparts, int T, int Hq, int Hkv,
                            const QkvEpi &qe, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (!parts || nparts < 1 || nparts > kMaxParts) return hipErrorInvalidValue;
  const int d = qe.hd;
  const Parts pt{parts, nparts, (size_t)T * (Hq + 2 * Hkv) * d};
  const int items = (Hq + Hkv) * (d / 2) + Hkv * d;
  if (qe.qk) {
    if (!qe.vt || qe.hkv != Hkv) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_qkv_parts_h, dim3((T + 31) / 32 * 32, (items + 255) / 256), dim3(256), 0, s, pt, T, Hq,
                       Hkv, qe);
  } else {
    hipLaunchKernelGGL(k_qkv_parts, dim3(T, (items + 255) / 256), dim3(256), 0, s, qkv, pt, Hq, Hkv, qe);
  }
  return hipGetLastError();
}

// SwiGLU of summed gate/up partial sums. parts: np x [rows, 2F], gate and up
// columns interleaved in blocks of 16 (block b: gate 16b.., then up 16b..).
// out [rows, F] = out_scale * silu(gate) * up: float (OUT_FMT FMT_F32) or fp16.
template <int OUT_FMT>
__global__ __launch_bounds__(256) void k_swiglu_parts(Parts pt, int F, void *__restrict__ out,
                                                      float out_scale, size_t n) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;   // output element (r, f)
  if (i >= n) return;
  const size_t r = i / F;
  const int f = (int)(i % F);
  const size_t gc = r * 2 * F + 32 * (f >> 4) + (f & 15);
  float qg[kMaxParts], qu[kMaxParts];
#pragma unroll
  for (int k = 0; k < kMaxParts; ++k)
    if (k < pt.np) {
      qg[k] = pt.p[(size_t)k * pt.stride + gc];
      qu[k] = pt.p[(size_t)k * pt.stride + gc + 16];
    }
  float gt = qg[0], up = qu[0];
#pragma unroll
  for (int k = 1; k < kMaxParts; ++k)
    if (k < pt.np) {
      gt += qg[k];
      up += qu[k];
    }
  const float y = gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up * out_scale;   // silu(gate) * up
  if constexpr (OUT_FMT == FMT_F32) ((float *)out)[i] = y;
  else ((f16 *)out)[i] = (f16)y;
}

hipError_t launch_swiglu_parts(int out_fmt, const float *parts, int nparts, int rows, int F, void *out,
                               float out_scale, hipStream_t s) {
  const size_t n = (size_t)rows * F;
  if (n == 0) return hipSuccess;
  if (nparts < 1 || nparts > kMaxParts || F % 16) return hipErrorInvalidValue;
  const Parts pt{parts, nparts, (size_t)rows * 2 * F};
  dim3 grid((unsigned)((n + 255) / 256));
  if (out_fmt == FMT_F32)
    hipLaunchKernelGGL(k_swiglu_parts<FMT_F32>, grid, dim3(256), 0, s, pt, F, out, out_scale, n);
  else
    hipLaunchKernelGGL(k_swiglu_parts<FMT_F16>, grid, dim3(256), 0, s, pt, F, out, out_scale, n);
  return hipGetLastError();
}

// ---------------------------------------------------- rotary table
// cos / sin of the rotation angle of every (token, pair): pair j of token
// t turns by pos[axis(j)][t] * inv_freq[j]; the angle and its sincos are
// evaluated in float64 and rounded to fp32. Built once per forward and
// shared by the q and k heads of all layers.
__global__ __launch_bounds__(256) void k_rope_table(const int32_t *__restrict__ pos, int T_tokens,
                                                    int half, RopeParams rp, float *__restrict__ rcos,
                                                    float *__restrict__ rsin) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)T_tokens * half) return;
  const int tok = (int)(i / half), j = (int)(i % half);
  const double ang = (double)pos[(size_t)rp.axis[j] * T_tokens + tok] * rp.inv_freq[j];
  double sv, cv;
  sincos(ang, &sv, &cv);
  rcos[i] = (float)cv;
  rsin[i] = (float)sv;
}

hipError_t launch_rope_table(const int32_t *pos_thw, int T, int half, const RopeParams &rp, float *rcos,
                             float *rsin, hipStream_t s) {
  const size_t n = (size_t)T * half;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, pos_thw, T, half,
                     rp, rcos, rsin);
  return hipGetLastError();
}

// ------------------------------------------------------------ positions
constexpr int kPosSeqPerLaunch = 128;

struct PosArgs {
  int n_seq;
  int start[kPosSeqPerLaunch + 1];   // absolute token offsets
  int nb[kPosSeqPerLaunch];          // text tokens before the image
  int gt[kPosSeqPerLaunch], gh[kPosSeqPerLaunch], gw[kPosSeqPerLaunch];
};

__global__ __launch_bounds__(256) void k_positions(int32_t *__restrict__ pos, int T_tokens, PosArgs a) {
  const int tk = a.start[0] + blockIdx.x * 256 + threadIdx.x;
  if (tk >= a.start[a.n_seq]) return;
  int lo = 0, hi = a.n_seq - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (a.start[mid] <= tk) lo = mid; else hi = mid - 1;
  }
  const int i = tk - a.start[lo];
  const int nb = a.nb[lo], gt = a.gt[lo], gh = a.gh[lo], gw = a.gw[lo];
  const int plane = gh * gw, nimg = gt * plane;
  int t, h, w;
  if (i < nb) {
    t = h = w = i;
  } else if (i < nb + nimg) {
    const int k = i - nb;
    t = nb + k / plane;
    h = nb + (k / gw) % gh;
    w = nb + k % gw;
  } else {
    // one past the largest position used so far
    int mx = nb - 1;
    if (nimg > 0) mx = nb + max(gt - 1, max(gh - 1, gw - 1));
    t = h = w = mx + 1 + (i - nb - nimg);
  }
  pos[tk] = t;
  pos[(size_t)T_tokens + tk] = h;
  pos[2 * (size_t)T_tokens + tk] = w;
}

hipError_t launch_positions(const int32_t *layouts5, int batch, int32_t *pos_thw, int T,
                            hipStream_t s) {
  int tok = 0;
  for (int first = 0; first < batch; first += kPosSeqPerLaunch) {
    const int n = batch - first < kPosSeqPerLaunch ? batch - first : kPosSeqPerLaunch;
    PosArgs a;
    a.n_seq = n;
    a.start[0] = tok;
    for (int i = 0; i < n; ++i) {
      const int32_t *l = layouts5 + 5 * (first + i);
      a.nb[i] = l[0];
      a.gt[i] = l[1];
      a.gh[i] = l[2];
      a.gw[i] = l[3];
      tok += l[0] + l[1] * l[2] * l[3] + l[4];
      a.start[i + 1] = tok;
    }
    const int cnt = a.start[n] - a.start[0];
    if (cnt > 0) {
      hipLaunchKernelGGL(k_positions, dim3((cnt + 255) / 256), dim3(256), 0, s, pos_thw, T, a);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

// ------------------------------------------------------ weight repacking
template <typename T>
__global__ void k_to_f32(const T *__restrict__ src, float *__restrict__ dst, int n, float scale) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = to_f32(src[i]) * scale;
}

hipError_t launch_to_f32(int src_fmt, const void *src, float *dst, int n, float scale, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dim3 grid((n + 255) / 256);
  if (src_fmt == FMT_BF16)
    hipLaunchKernelGGL(k_to_f32<bf16>, grid, dim3(256), 0, s, (const bf16 *)src, dst, n, scale);
  else
    hipLaunchKernelGGL(k_to_f32<float>, grid, dim3(256), 0, s, (const float *)src, dst, n, scale);
  return hipGetLastError();
}

// One workgroup per row: the row's max |w| and L2 norm, folded into
// stats[0] / stats[1] with atomic max on the (non-negative) float bit
// patterns, whose integer order matches their value order.
template <typename T>
__global__ __launch_bounds__(256) void k_matrix_stats(const T *__restrict__ src, int cols,
                                                      float *__restrict__ stats) {
  __shared__ float rmax[4], rss[4];
  const T *row = src + (size_t)blockIdx.x * cols;
  float mx = 0.f, ss = 0.f;
  for (int c = threadIdx.x; c < cols; c += 256) {
    const float v = to_f32(row[c]);
    mx = fmaxf(mx, fabsf(v));
    ss += v * v;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    mx = warp_max_xor(mx, m);
    ss = warp_sum_xor(ss, m);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { rmax[w] = mx; rss[w] = ss; }
  __syncthreads();
  if (threadIdx.x == 0) {
    const float m4 = fmaxf(fmaxf(rmax[0], rmax[1]), fmaxf(rmax[2], rmax[3]));
    const float n4 = sqrtf(rss[0] + rss[1] + rss[2] + rss[3]);
    atomicMax((unsigned int *)&stats[0], __float_as_uint(m4));
    atomicMax((unsigned int *)&stats[1], __float_as_uint(n4));
  }
}

hipError_t launch_matrix_stats(int src_fmt, const void *src, int rows, int cols, float *stats,
                               hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (src_fmt == FMT_BF16)
    hipLaunchKernelGGL(k_matrix_stats<bf16>, dim3(rows), dim3(256), 0, s, (const bf16 *)src, cols, stats);
  else
    hipLaunchKernelGGL(k_matrix_stats<float>, dim3(rows), dim3(256), 0, s, (const float *)src, cols, stats);
  return hipGetLastError();
}

// One workgroup per source row: dst[map(r)] = convert(src[r] * scale).
template <typename TS, typename TD>
__global__ __launch_bounds__(256) void k_convert_rows(const TS *__restrict__ src, TD *__restrict__ dst,
                                                      int cols, float scale, int interleave, int up) {
  const int r = blockIdx.x;
  const int dr = interleave ? 32 * (r >> 4) + 16 * up + (r & 15) : r;
  const TS *s = src + (size_t)r * cols;
  TD *d = dst + (size_t)dr * cols;
  for (int c = threadIdx.x; c < cols; c += 256) d[c] = from_f32<TD>(to_f32(s[c]) * scale);
}

hipError_t launch_convert_rows(int src_fmt, const void *src, int dst_fmt, void *dst, int rows, int cols,
                               float scale, int interleave, int up, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (interleave && rows % 16) return hipErrorInvalidValue;
  dim3 grid(rows);
  if (src_fmt == FMT_BF16 && dst_fmt == FMT_F16)
    hipLaunchKernelGGL((k_convert_rows<bf16, f16>), grid, dim3(256), 0, s, (const bf16 *)src, (f16 *)dst,
                       cols, scale, interleave, up);
  else if (src_fmt == FMT_F32 && dst_fmt == FMT_F32)
    hipLaunchKernelGGL((k_convert_rows<float, float>), grid, dim3(256), 0, s, (const float *)src,
                       (float *)dst, cols, scale, interleave, up);
  else if (src_fmt == FMT_F32 && dst_fmt == FMT_BF16)
    hipLaunchKernelGGL((k_convert_rows<float, bf16>), grid, dim3(256), 0, s, (const float *)src,
                       (bf16 *)dst, cols, scale, interleave, up);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// OCP e4m3 code of x, |x| <= 448, rounded to nearest with ties to even.
// Below 2^-6 the codes are subnormal with quantum 2^-9; binade [2^E, 2^(E+1))
// above has quantum 2^(E-3). A significand that rounds up to 16 carries into
// the exponent field through the code arithmetic itself, and 2^-6 (count 8
// of the subnormal quantum) is the first normal code. Zero is +0.
__device__ __forceinline__ uint32_t e4m3_code(float x) {
  const float a = fabsf(x);
  uint32_t mag;
  if (a < 0.015625f) {
    mag = (uint32_t)rintf(a * 512.f);                                 // exact scaling, 0..8
  } else {
    const int E = (int)((__float_as_uint(a) >> 23) & 0xFF) - 127;     // 2^-6 <= a <= 448: normal
    mag = (uint32_t)((E + 7) * 8) + (uint32_t)rintf(ldexpf(a, 3 - E)) - 8u;   // count 8..16
  }
  return mag == 0 ? 0u : (mag | (x < 0.f ? 0x80u : 0u));
}

// One workgroup per source row: the row's max |x| fixes its scale 2^e
// (smallest e with max <= 448 * 2^e, frexp: max = f * 2^E2, f in [0.5, 1),
// 448 = 0.875 * 2^9), then every element is coded after the exact division.
template <typename TS>
__global__ __launch_bounds__(256) void k_quantize_e4m3_rows(const TS *__restrict__ src, int cols,
                                                            uint8_t *__restrict__ codes,
                                                            float *__restrict__ scales, int interleave,
                                                            int up) {
  __shared__ float rmax[4];
  const int r = blockIdx.x;
  const int dr = interleave ? 32 * (r >> 4) + 16 * up + (r & 15) : r;
  const TS *s = src + (size_t)r * cols;
  float mx = 0.f;
  for (int c = threadIdx.x; c < cols; c += 256) mx = fmaxf(mx, fabsf(to_f32(s[c])));
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) mx = warp_max_xor(mx, m);
  if ((threadIdx.x & 63) == 0) rmax[threadIdx.x >> 6] = mx;
  __syncthreads();
  const float amax = fmaxf(fmaxf(rmax[0], rmax[1]), fmaxf(rmax[2], rmax[3]));
  int e = 0;
  if (amax > 0.f) {
    int E2 = 0;
    const float f = frexpf(amax, &E2);
    e = f <= 0.875f ? E2 - 9 : E2 - 8;
  }
  uint8_t *d = codes + (size_t)dr * cols;
  for (int c = threadIdx.x; c < cols; c += 256) d[c] = (uint8_t)e4m3_code(ldexpf(to_f32(s[c]), -e));
  if (threadIdx.x == 0) scales[dr] = ldexpf(1.f, e);
}

hipError_t launch_quantize_e4m3_rows(int src_fmt, const void *src, int rows, int cols, uint8_t *codes,
                                     float *scales, int interleave, int up, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (interleave && rows % 16) return hipErrorInvalidValue;
  if (src_fmt == FMT_BF16)
    hipLaunchKernelGGL(k_quantize_e4m3_rows<bf16>, dim3(rows), dim3(256), 0, s, (const bf16 *)src, cols, codes,
                       scales, interleave, up);
  else if (src_fmt == FMT_F32)
    hipLaunchKernelGGL(k_quantize_e4m3_rows<float>, dim3(rows), dim3(256), 0, s, (const float *)src, cols,
                       codes, scales, interleave, up);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace mte
