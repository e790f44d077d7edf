// Projection GEMMs of the decoder layer on gfx950 matrix cores.
//
// C = A[M, K] * W[N, K]^T, A = activations (row-major, K contiguous),
// W = weights in nn.Linear layout (row-major, K contiguous).
//
// Precision modes:
//  MODE_F32: A and W fp32, v_mfma_f32_32x32x2_f32.
//  MODE_F16: A and W fp16, v_mfma_f32_32x32x16_f16, fp32 accumulation. The
//   weights are bf16 values held as fp16 times a power of two chosen per
//   matrix so that its largest magnitude lands in [2^14, 2^15): every bf16
//   value down to 2^-31 of that maximum converts exactly. Activations are
//   rounded once to fp16 (an 11-bit significand, against bf16's 8) after a
//   power-of-two pre-scale that a static bound keeps in fp16 range; the
//   epilogue multiplies the product by the inverse of both scales (`scale`,
//   exact). One MFMA per fragment at the same dense rate as bf16.
//  MODE_F8W: A fp16 as in MODE_F16; W OCP e4m3 codes (one byte per weight)
//   with one power-of-two scale per output row (`cs`). The codes are staged
//   through LDS at half the bytes of fp16 and widened to fp16 after the LDS
//   read (exact: every e4m3 value is an fp16 value), one k-step ahead of
//   the MFMAs that use them; the accumulators are multiplied by their
//   column's scale before the epilogue.
//
// Each workgroup (4 or 8 waves, WM x WN) owns a BM x BN output tile; each
// wave a (BM/WM) x (BN/WN) block of 32x32 MFMA tiles. Eight waves, or two
// four-wave workgroups per CU, put two waves on every SIMD, so one wave's
// LDS reads and waits overlap the other's MFMAs. K is walked in stages of 64
// or 128 bytes per row, staged through a ring of 2-16 LDS slots (one barrier
// per stage): the loads of the next P stages are in flight while the current
// one feeds the MFMAs. The deep rings serve small M (one frame), where a
// workgroup's whole K range is a handful of stages: all of them are then in
// flight at once and the kernel waits for memory once, not once per stage.
//
// LDS rows are 128 bytes = 8 chunks of 16 bytes; chunk c of row r is stored
// at slot c ^ ((r ^ (r >> 3)) & 7), so the 16-byte fragment reads of 8 or 16
// consecutive rows at one logical chunk hit distinct banks.
//
// Epilogues are fused: fp32 store with the per-head QK-norm and rotary
// embedding of the q and k heads (QKV projection; a wave's columns cover
// whole heads, so a head's sum of squares is a reduction over the wave's
// lanes and both members of each rotary pair sit in one lane), SwiGLU over
// gate/up rows interleaved in blocks of 16 (MLP up-projection: a 32-column
// MFMA tile holds 16 gate and the 16 matching up columns, paired by one
// lane exchange; written in the activation format) and accumulation into
// the fp32 residual stream (attention output projection and MLP
// down-projection). With K split over workgroups (small M), each
// split stores its partial sum instead, and the kernel that consumes the
// product adds the partials up in split order, so results do not depend on
// the order in which workgroups finish.
#pragma once

#include <cmath>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace mte {

struct GemmArgs {
  const char *A;
  const char *W;
  void *C;            // EPI_STORE / EPI_RESID / EPI_PARTIAL: float; EPI_SWIGLU / EPI_GELU: activation format
  size_t c_plane;     // EPI_PARTIAL: elements between the partial sums of two K splits
  int M, N, K, ldc;
  int k_chunk;        // K range of one split (gridDim.z splits)
  float scale;        // product multiplier (inverse operand pre-scales)
  float out_scale;    // EPI_SWIGLU / EPI_GELU output multiplier
  QkvEpi qe;          // EPI_QKV
  const float *cs;    // MODE_F8W: per-column (weight row) scales [N]
  const float *bias;  // [N] added to the product before the epilogue (unsplit launches), or null
  // Placement of tiles on the eight XCDs (workgroup i of a launch runs on XCD
  // i % 8): xa x xb x xc = 8 with xa | M tiles, xb | N tiles, xc | K splits;
  // XCD x serves one block of M tiles, one of N tiles and one of splits, so
  // it fetches only its share of A and W into its L2. xa = 0: workgroup
  // (x, y, z) serves N tile x, M tile y, split z.
  int xa, xb, xc;
};

// tanh-approximated GELU, 0.5 z (1 + tanh(u)) with u = sqrt(2/pi) (z + 0.044715 z^3),
// evaluated as z * sigmoid(2u) = z / (1 + exp(-2u)) (the same function): one
// exp and one hardware reciprocal (1 ulp) instead of a library tanh. Large
// negative z: exp overflows to inf and the result is 0.
__device__ __forceinline__ float gelu_tanh(float z) {
  const float m2u = -1.5957691216057308f * z * (1.f + 0.044715f * z * z);
  return z * __builtin_amdgcn_rcpf(1.f + __expf(m2u));
}
// silu(z) = z / (1 + exp(-z)), with the hardware reciprocal.
__device__ __forceinline__ float silu_f(float z) { return z * __builtin_amdgcn_rcpf(1.f + __expf(-z)); }

// Chunk swizzles for rows of 128 bytes (8 chunks) and 64 bytes (4 chunks):
// the 16-byte fragment reads (32 consecutive rows at one logical chunk, the
// upper half-wave at the next chunk) are free of LDS bank conflicts with
// these two (measured with SQ_LDS_BANK_CONFLICT on gfx950; e.g. the 64-byte
// variant c ^ ((r >> 1) & 3) is 2-way conflicted).
template <int CH>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (CH == 8) return c ^ ((r ^ (r >> 3)) & 7);
  else return c ^ ((r >> 2) & 3);
}

// Eight OCP e4m3 codes (k order, byte 0 first) -> eight fp16 values, exact
// (v_cvt_scalef32_pk_f16_fp8 with scale 1: e4m3's range [2^-9, 448] and its
// 3-bit significand fit fp16).
__device__ __forceinline__ f16x8 widen_e4m3(u32x2 w) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)w[0], 1.f, false);
  const h2 b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)w[0], 1.f, true);
  const h2 c = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)w[1], 1.f, false);
  const h2 d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)w[1], 1.f, true);
  return f16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// Cross-lane steps without the LDS unit (gfx950):
// swap16(a, b): v_permlane16_swap -- in each 32-lane half, the upper 16 lanes'
// a and the lower 16 lanes' b trade places, so that afterwards a lower lane
// holds (its a, its partner's a) and an upper lane (its partner's b, its b).
__device__ __forceinline__ void swap16(float &a, float &b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
// x + the same value of lane (l + n) mod 16 in its 16-lane row (DPP row_ror:n).
template <int n>
__device__ __forceinline__ float add_row_ror(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + n, 0xf, 0xf, false));
}
// Sum of x over the 32 lanes of each half-wave, in every lane of it.
__device__ __forceinline__ float sum_half_wave(float x) {
  x = add_row_ror<8>(x);
  x = add_row_ror<4>(x);
  x = add_row_ror<2>(x);
  x = add_row_ror<1>(x);            // every lane: its 16-lane row's sum
  float y = x;
  swap16(x, y);                     // (own, partner) or (partner, own)
  return x + y;
}

// Element at byte offset `off` of `base`: with a wave-uniform base and a 32-bit
// lane offset this is one global access with a scalar base address (no
// 64-bit address arithmetic per lane).
template <typename T>
__device__ __forceinline__ T &at(T *base, uint32_t off) { return *(T *)((char *)base + off); }

// Row of accumulator register r of a 32x32 MFMA tile, less the lane's
// 4 * (lane >> 5): acc_row(r, lane) = acc_row0(r) + 4 * (lane >> 5).
__host__ __device__ constexpr int acc_row0(int r) { return 8 * (r >> 2) + (r & 3); }

// EPI_QKV epilogue of one wave: rows mw.. (TM blocks of 32), columns cw..
// (TN blocks of 32 = whole heads of HD columns), mw and cw wave-uniform. For
// each row and q or k head: RMS-normalise (sum of squares over the head's
// HD/32 column blocks and the 32 lanes that hold the row) and rotate pair
// (c, c + HD/2), i.e. column blocks (jb, jb + HD/64) of one lane. Gains are
// read once; the rotary table values of a block of 32 rows are read before
// they are used. fp32 rows: a block wholly inside M is stored at a
// wave-uniform row address plus a 32-bit lane offset, without per-row tests.
// With q.qk the result goes out in the fp16 attention operand layout.
template <int HD, int TM, int TN>
__device__ __forceinline__ void qkv_epilogue(const f32x16 (&acc)[TM][TN], const GemmArgs &g, int cw,
                                             int mw, int lane) {
  constexpr int HJB = HD / 32;                    // column blocks per head
  constexpr int NH = TN / HJB;                    // heads of the wave
  static_assert(TN % HJB == 0, "whole heads per wave");
  const QkvEpi &q = g.qe;
  const int lrow = lane & 31, lgrp = lane >> 5;
  const int M = g.M;
  float *C = (float *)g.C;
  const uint32_t lofs = (uint32_t)(4 * lgrp * g.ldc + lrow) * 4u;   // bytes
  bool rot[NH], anyrot = false;
  float gsc[TN];
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const int cb = cw + h * HD;
    rot[h] = cb < q.rot_cols;                     // wave-uniform
    anyrot |= rot[h];
    const float *gn = cb < q.nq_cols ? q.qn : q.kn;
#pragma unroll
    for (int jj = 0; jj < HJB; ++jj) gsc[h * HJB + jj] = (rot[h] && gn) ? gn[jj * 32 + lrow] : 1.f;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = mw + i * 32;
    const bool full = mb + 32 <= M;               // wave-uniform
    // the rotary entries of a row depend on the pair index only: one set of
    // HJB / 2 blocks serves every head of the wave
    float tc[16][HJB / 2], ts[16][HJB / 2];
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int jj = 0; jj < HJB / 2; ++jj) {
        tc[r][jj] = 1.f;
        ts[r][jj] = 0.f;
      }
    // table row mb + acc_row(r, lane), clamped to M - 1 in a partial block
    if (anyrot) {
      if (full) {
        const uint32_t to = (uint32_t)(4 * lgrp * (HD / 2) + lrow) * 4u;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const size_t rb = (size_t)(mb + acc_row0(r)) * (HD / 2);
#pragma unroll
          for (int jj = 0; jj < HJB / 2; ++jj) {
            tc[r][jj] = at(q.rcos + rb, to + jj * 128u);
            ts[r][jj] = at(q.rsin + rb, to + jj * 128u);
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const size_t rb = (size_t)min(mb + acc_row(r, lane), M - 1) * (HD / 2);
#pragma unroll
          for (int jj = 0; jj < HJB / 2; ++jj) {
            tc[r][jj] = q.rcos[rb + jj * 32 + lrow];
            ts[r][jj] = q.rsin[rb + jj * 32 + lrow];
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float v[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) v[j] = acc[i][j][r] * g.scale;
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        if (!rot[h]) continue;
        if (q.qn) {
          float ss = 0.f;
#pragma unroll
          for (int jj = 0; jj < HJB; ++jj) ss += v[h * HJB + jj] * v[h * HJB + jj];
          ss = sum_half_wave(ss);
          const float rs = rsqrtf(ss / (float)HD + q.eps);
#pragma unroll
          for (int jj = 0; jj < HJB; ++jj) v[h * HJB + jj] = v[h * HJB + jj] * rs * gsc[h * HJB + jj];
        }
#pragma unroll
        for (int jj = 0; jj < HJB / 2; ++jj) {
          const int j = h * HJB + jj, jp = j + HJB / 2;
          const float u = v[j], w = v[jp];
          v[j] = u * tc[r][jj] - w * ts[r][jj];
          v[jp] = w * tc[r][jj] + u * ts[r][jj];
        }
      }
      if (q.qk) {
        // attention operand layout: q and k heads as fp16 rows (v below)
        const int m = mb + acc_row(r, lane);
        if (m < M) {
          f16 *qr = q.qk + (size_t)m * q.rot_cols + cw + lrow;
#pragma unroll
          for (int h = 0; h < NH; ++h) {
            if (!rot[h]) continue;
            const float pre = cw + h * HD < q.nq_cols ? q.q_pre : q.k_pre;
#pragma unroll
            for (int jj = 0; jj < HJB; ++jj) qr[(h * HJB + jj) * 32] = (f16)(v[h * HJB + jj] * pre);
          }
        }
      } else if (full) {
        float *p = C + (size_t)(mb + acc_row0(r)) * g.ldc + cw;
#pragma unroll
        for (int j = 0; j < TN; ++j) at(p, lofs + j * 128u) = v[j];
      } else {
        const int m = mb + acc_row(r, lane);
        if (m < M)
#pragma unroll
          for (int j = 0; j < TN; ++j) C[(size_t)m * g.ldc + cw + j * 32 + lrow] = v[j];
      }
    }
    if (q.qk && mb < M) {
      // v heads as V^T tiles: the block's 32 rows are one token tile (mb is a
      // multiple of 32), and a lane's 16 accumulator rows are exactly the
      // values of its column in the tile's fragment order: registers 0..7 go
      // to positions 8g.., registers 8..15 to 16 + 8g.. (g = lane / 32).
      // Rows past M are written as zeros; blocks wholly past M belong to no
      // tile of the batch and are skipped.
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        if (rot[h]) continue;
#pragma unroll
        for (int jj = 0; jj < HJB; ++jj) {
          const int j = h * HJB + jj;
          const int dv = cw + j * 32 + lrow - q.rot_cols;
          f16 *dst = q.vt + (((size_t)(mb >> 5) * q.hkv + dv / HD) * HD + dv % HD) * 32 + lgrp * 8;
          f16x8 lo, hi;
          const float sv = g.scale * q.v_pre;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            lo[e] = (f16)(mb + acc_row(e, lane) < M ? acc[i][j][e] * sv : 0.f);
            hi[e] = (f16)(mb + acc_row(8 + e, lane) < M ? acc[i][j][8 + e] * sv : 0.f);
          }
          *(f16x8 *)dst = lo;
          *(f16x8 *)(dst + 16) = hi;
        }
      }
    }
  }
}

// The main loop keeps P stages in an LDS ring filled by direct global->LDS
// loads, and double-buffers the MFMA operand fragments in registers. One
// barrier per stage, placed after the first MFMA of the stage's last k-step:
// before it each wave waits for its own loads of the next stage and for its
// own LDS reads (the last k-step's fragments are already in registers).
// After it, all waves' loads of stage kt+1 are in LDS and no wave reads slot
// kt % P again, so the loads of stage kt+P go into that slot, and the first
// fragments of stage kt+1 are read while the last MFMAs of stage kt run.
// Raw s_barrier (no fence) keeps the compiler from forcing vmcnt(0) at the
// barrier; the waits are explicit.
template <int MODE, int BM, int BN, int WM, int WN, int ROWB, int P, int EPI, int OCC>
__global__ __launch_bounds__(64 * WM * WN, OCC) __attribute__((amdgpu_waves_per_eu((OCC * WM * WN + 3) / 4, (OCC * WM * WN + 3) / 4))) void k_gemm(GemmArgs g) {
  typedef typename std::conditional<MODE == MODE_F32, float, f16>::type T;
  constexpr bool W8 = MODE == MODE_F8W;           // one-byte weights
  constexpr int KS = ROWB / (int)sizeof(T);       // k elements per stage
  constexpr int CH = ROWB / 16;                   // 16-byte chunks per A row per stage
  constexpr int CHW = W8 ? CH / 2 : CH;           // 16-byte chunks per W row per stage
  static_assert(!W8 || CHW == 4, "e4m3 weights: 64-byte W rows per stage");
  constexpr int WTM = BM / WM, WTN = BN / WN;     // wave tile
  constexpr int TM = WTM / 32, TN = WTN / 32;     // 32x32 MFMA tiles per wave
  constexpr int ACH = BM * CH, BCH = BN * CHW;    // chunks per stage (A / W)
  constexpr int NW = WM * WN;                     // waves per workgroup
  constexpr int NT = 64 * NW;                     // threads per workgroup
  // DMA rounds: each wave instruction fills one group of 64 chunks. A last,
  // partial round repeats the matrix's final group in the waves past it
  // (the same bytes to the same LDS slots), so every wave issues the same
  // number of loads and the vmcnt waits stay exact.
  static_assert(ACH % 64 == 0 && BCH % 64 == 0, "whole 64-chunk groups");
  constexpr int AG = ACH / 64, BG = BCH / 64;     // chunk groups per stage
  constexpr int AR = (AG + NW - 1) / NW, BR = (BG + NW - 1) / NW;   // DMA instructions per thread
  constexpr int LOADS = AR + BR;                  // per thread per stage
  constexpr int STAGE = ACH + BCH;                // u32x4 slots per stage
  static_assert(NW == 4 || NW == 6 || NW == 8, "4, 6 or 8 waves");
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
  static_assert(LOADS * (P - 1) < 64 && P >= 2 && P <= 16, "vmcnt range, ring depth");
  typedef typename Frag<T>::type frag_t;

  extern __shared__ u32x4 lds[];                  // [P][STAGE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int tn = blockIdx.x, tm = blockIdx.y, tz = blockIdx.z;
  if (g.xa) {
    // XCD of this workgroup and its index among that XCD's workgroups
    const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int xcd = lin & 7, j = lin >> 3;
    const int xbc = g.xb * g.xc;
    const int xi = xcd / xbc, xj = (xcd % xbc) / g.xc, xk = xcd % g.xc;
    const int sm = gridDim.y / g.xa, sn = gridDim.x / g.xb, ss = gridDim.z / g.xc;
    const int n = j % sn, t = j / sn;
    tn = xj * sn + n;
    tm = xi * sm + t % sm;
    tz = xk * ss + t / sm;
  }
  const int n0 = tn * BN, m0 = tm * BM;
  const int M = g.M;
  const size_t rowb = (size_t)g.K * sizeof(T);    // row pitch in bytes (A; W unless W8)
  const size_t kb0 = (size_t)tz * g.k_chunk * sizeof(T);
  const size_t rowbw = W8 ? (size_t)g.K : rowb;
  const size_t kb0w = W8 ? (size_t)tz * g.k_chunk : kb0;
  const int nk = g.k_chunk / KS;

  // DMA sources: instruction c of this thread fills LDS slot q = (c*NW + wave)*64 + lane
  // of its matrix (row q / CH, swizzled slot q % CH, logical chunk slot ^ f(row)).
  // As 32-bit byte offsets from g.A and g.W (the host keeps both matrices
  // under 4 GiB). The W rows of DMA instruction c are instruction 0's plus
  // c * BROWS when every round is whole and the step keeps the chunk swizzle
  // (a multiple of 64 rows for 8-chunk rows, 16 for 4-chunk rows): one offset
  // and a uniform stride then replace BR of them (registers the two-stage
  // 128-byte tiles need for their fragments).
  constexpr int BROWS = NW * 64 / CHW;
  constexpr bool BSTRIDE = BG % NW == 0 && BROWS % (CHW == 8 ? 64 : 16) == 0;
  uint32_t pa[AR], pb[BSTRIDE ? 1 : BR];
  const size_t bstep = (size_t)BROWS * rowbw;
#pragma unroll
  for (int c = 0; c < AR; ++c) {
    const int q = min(c * NW + wave, AG - 1) * 64 + lane, r = q / CH, ch = swz<CH>(r, q % CH);
    pa[c] = (uint32_t)((size_t)min(m0 + r, M - 1) * rowb + ch * 16);
  }
#pragma unroll
  for (int c = 0; c < (BSTRIDE ? 1 : BR); ++c) {
    const int q = min(c * NW + wave, BG - 1) * 64 + lane, r = q / CHW, ch = swz<CHW>(r, q % CHW);
    pb[c] = (uint32_t)((size_t)(n0 + r) * rowbw + ch * 16);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  const int uwave = __builtin_amdgcn_readfirstlane(wave);   // wave-uniform in an SGPR
  // DMA load x (0 <= x < LOADS) of K-stage `ks` into ring slot `slot`.
  auto dma_one = [&](int ks, int slot, int x) {
    const uint32_t st = lds0 + (uint32_t)(slot * STAGE) * 16u;
    const size_t ko = (size_t)ks * ROWB;
    if (x < AR) {
      dma16(g.A + kb0 + ko, pa[x], st + (uint32_t)(min(x * NW + uwave, AG - 1) * 64) * 16u);
    } else {
      const int c = x - AR;
      const char *wb = g.W + kb0w + (W8 ? ko / 2 : ko);
      if constexpr (BSTRIDE) dma16(wb + c * bstep, pb[0], st + (uint32_t)(ACH + min(c * NW + uwave, BG - 1) * 64) * 16u);
      else dma16(wb, pb[c], st + (uint32_t)(ACH + min(c * NW + uwave, BG - 1) * 64) * 16u);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  frag_t fa[2][TM], fb[2][TN];
  // W8: the raw codes of a W fragment (8 bytes per lane) are read into fw;
  // the first MFMA of the next k-step that uses them widens them into fb.
  typedef typename std::conditional<W8, u32x2, char>::type wraw_t;
  wraw_t fw[2][TN];
  const int lrow = lane & 31, lgrp = lane >> 5;
  // Fragment read x (0 <= x < NR) of k-step kk of the stage at `st` into
  // buffer b, in the order the MFMAs consume them: the W fragments, then the
  // A fragments.
  auto read_one = [&](const u32x4 *st, int kk, int b, int x) {
    const int ch = kk * 2 + lgrp;
    if (x < TN) {
      const int r = wn * WTN + x * 32 + lrow;
      if constexpr (W8) {
        // k-step kk of a W row is its chunk kk; lane group g takes bytes 8g..8g+7
        const char *sw = (const char *)(st + ACH);
        fw[b][x] = *(const u32x2 *)(sw + (r * CHW + swz<CHW>(r, kk)) * 16 + lgrp * 8);
      } else {
        fb[b][x] = __builtin_bit_cast(frag_t, st[ACH + r * CH + swz<CH>(r, ch)]);
      }
    } else {
      const int i = x - TN;
      const int r = wm * WTM + i * 32 + lrow;
      fa[b][i] = __builtin_bit_cast(frag_t, st[r * CH + swz<CH>(r, ch)]);
    }
  };
  auto mfma_one = [&](int b, int x) {
    const int j = x % TN, i = x / TN;
    if constexpr (W8) {
      if (i == 0) fb[b][j] = widen_e4m3(fw[b][j]);
    }
    mfma32(acc[i][j], fa[b][i], fb[b][j]);
  };
  constexpr int KK = CH / 2;                      // 16-k steps per stage (even)
  static_assert(KK % 2 == 0, "fragment buffer parity");
  constexpr int NM = TM * TN;                     // MFMAs per k-step
  constexpr int NR = TM + TN;                     // fragment reads per k-step
  // The loads of stage kt+P are issued in NPART parts: part 0 right after the
  // barrier of stage kt, parts 1.. in the k-steps of stage kt+1 before its
  // barrier. With P >= 3 every stage still has P-2 whole stages of loads in
  // flight behind it at the barrier that waits for it; P = 2 issues each
  // stage whole, after the barrier.
  constexpr int NPART = (P >= 3) ? KK : 1;
  constexpr int PART = (LOADS + NPART - 1) / NPART;

  // One k-step: the NM MFMAs on fragment buffer `cur`, with the side work
  // spread between them in issue order -- the NR fragment reads of the next
  // k-step (k-step rkk of the stage at rst, into buffer cur^1), then DMA
  // loads [d0, d1) of stage ks into slot `slot`. With `bar`, the barrier of
  // the stage (after this wave's loads of the next stage have landed) goes
  // after the first MFMA, ahead of all side work.
  // Each unit of side work is pinned behind its MFMA by a scheduling
  // barrier, so the matrix core keeps busy while it issues.
  auto kstep = [&](int cur, const u32x4 *rst, int rkk, int ks, int slot, int d0, int d1, bool bar) {
    const int nside = NR + (d1 - d0);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      mfma_one(cur, m);
      if (bar && m == 0) {
        wait_vm_lds0<(P - 2) * LOADS>();   // this wave's loads of the next stage landed, its reads done
        __builtin_amdgcn_s_barrier();      // ... everyone's: slot kt % P is free
        asm volatile("" ::: "memory");     // keep LDS reads of the next stage below it
      }
      const int s0 = (m * nside + NM - 1) / NM, s1 = ((m + 1) * nside + NM - 1) / NM;
#pragma unroll
      for (int x = s0; x < s1; ++x) {
        if (x < NR) read_one(rst, rkk, cur ^ 1, x);
        else dma_one(ks, slot, d0 + x - NR);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // The loop body is branch-free (a branch between LDS reads and their
  // use makes the waitcnt pass drain all outstanding reads): every iteration
  // issues its loads -- past the end, repeats of the last stage into slots
  // that are never read again -- so every wait is a fixed vmcnt.
  // Prologue: stages 0..P-2 whole and part 0 of stage P-1 (P = 2: stages
  // 0..P-1 whole), then stage 0 must have landed.
  constexpr int PRE_FULL = (NPART > 1) ? P - 1 : P;
  constexpr int PRE_PART = (NPART > 1) ? (PART < LOADS ? PART : LOADS) : 0;
#pragma unroll
  for (int s = 0; s < PRE_FULL; ++s)
#pragma unroll
    for (int x = 0; x < LOADS; ++x) dma_one(min(s, nk - 1), s, x);
#pragma unroll
  for (int x = 0; x < PRE_PART; ++x) dma_one(min(P - 1, nk - 1), P - 1, x);
  wait_vm<(PRE_FULL - 1) * LOADS + PRE_PART>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
#pragma unroll
  for (int x = 0; x < NR; ++x) read_one(lds, 0, 0, x);
  for (int kt = 0; kt < nk; ++kt) {
    const u32x4 *st = lds + (kt % P) * STAGE;
    const u32x4 *nx = lds + ((kt + 1) % P) * STAGE;
    const int ksa = min(kt + P - 1, nk - 1), sla = (kt + P - 1) % P;   // parts 1.. issued here
    const int ksb = min(kt + P, nk - 1), slb = kt % P;                  // part 0 issued here
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < KK) {
        const int q = kk + 1;                       // DMA part of this k-step
        const int d0 = (NPART > 1) ? min(q * PART, LOADS) : 0;
        const int d1 = (NPART > 1) ? min((q + 1) * PART, LOADS) : 0;
        kstep(cur, st, kk + 1, ksa, sla, d0, d1, false);
      } else {
        const int d1 = (NPART > 1) ? min(PART, LOADS) : LOADS;
        kstep(cur, nx, 0, ksb, slb, 0, d1, true);
      }
    }
  }
  wait_vm<0>();                          // no load may land after the workgroup ends
  if constexpr (W8) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float c = g.cs[n0 + wn * WTN + j * 32 + lrow];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] *= c;
    }
  }
  if (g.bias) {
    // bias / scale added to the accumulators: `scale` is a power of two, so
    // (acc + bias / scale) * scale rounds exactly like acc * scale + bias.
    const float ib = 1.f / g.scale;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float b = g.bias[n0 + wn * WTN + j * 32 + lrow] * ib;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += b;
    }
  }

  // Epilogue. The wave's rows are mw + 32 i + acc_row(r, lane), its columns
  // cw + 32 j + lrow (mw, cw wave-uniform). A 32-row block wholly inside M
  // (a wave-uniform test) is written without per-row tests, each row at a
  // wave-uniform address plus a 32-bit lane offset; only the last, partial
  // block tests rows.
  const int uwm = uwave / WN, uwn = uwave % WN;
  const int mw = m0 + uwm * WTM, cw = n0 + uwn * WTN;
  if constexpr (EPI == EPI_QKV) {
    // (the host only launches tiles whose waves cover whole heads)
    if (g.qe.hd == 128) {
      if constexpr (TN % 4 == 0) qkv_epilogue<128, TM, TN>(acc, g, cw, mw, lane);
    } else {
      if constexpr (TN % 2 == 0) qkv_epilogue<64, TM, TN>(acc, g, cw, mw, lane);
    }
    return;
  }
  typedef typename std::conditional<MODE == MODE_F32, float, f16>::type TO;   // activation outputs
  if constexpr (EPI == EPI_SWIGLU) {
    // Column block j (32 columns) of the interleaved product holds gate
    // (lanes l%32 < 16) and up (l%32 >= 16) of outputs f = 16*block + l%16.
    // Of each pair of accumulator rows (r, r+1) the gate lane finishes row r
    // and the up lane row r+1: one swap16 hands each the (gate, up) pair it
    // needs. With z = scale*g and u = scale*up,
    //   silu(z) * u * out_scale = (g * up) / (1 + 2^(g * (-scale*log2 e))) * (scale^2 * out_scale).
    const bool upl = lrow >= 16;
    const float c1 = -g.scale * 1.4426950408889634f;
    const float s2 = g.scale * g.scale * g.out_scale;
    TO *C = (TO *)g.C;
    const int fc = cw >> 1;                       // first output column of the wave
    const uint32_t lofs = (uint32_t)((4 * lgrp + (upl ? 1 : 0)) * g.ldc + (lrow & 15)) * (uint32_t)sizeof(TO);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int mb = mw + i * 32;
      const bool full = mb + 32 <= M;
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        float y[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          float ga = acc[i][j][r], up = acc[i][j][r + 1];
          swap16(ga, up);
          const float e = __builtin_amdgcn_exp2f(ga * c1);
          y[j] = (ga * up) * __builtin_amdgcn_rcpf(1.f + e) * s2;
        }
        if (full) {
          TO *p = C + (size_t)(mb + acc_row0(r)) * g.ldc + fc;
#pragma unroll
          for (int j = 0; j < TN; ++j) at(p, lofs + j * 16u * (uint32_t)sizeof(TO)) = (TO)y[j];
        } else {
          const int m = mb + acc_row(r + (upl ? 1 : 0), lane);
          if (m < M)
#pragma unroll
            for (int j = 0; j < TN; ++j) C[(size_t)m * g.ldc + fc + j * 16 + (lrow & 15)] = (TO)y[j];
        }
      }
    }
    return;
  }
  const uint32_t lofs = (uint32_t)(4 * lgrp * g.ldc + lrow);   // elements
  if constexpr (EPI == EPI_GELU) {
    // gelu_tanh(scale*a) * out_scale = a / (1 + 2^(c0 a (1 + k2 a^2))) * (scale * out_scale),
    // c0 = -2 sqrt(2/pi) log2(e) scale, k2 = 0.044715 scale^2.
    const float k2 = 0.044715f * g.scale * g.scale;
    const float c0 = -1.5957691216057308f * 1.4426950408889634f * g.scale;
    const float so = g.scale * g.out_scale;
    TO *C = (TO *)g.C;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int mb = mw + i * 32;
      const bool full = mb + 32 <= M;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float y[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const float a = acc[i][j][r];
          const float e = __builtin_amdgcn_exp2f(a * fmaf(a * a, k2, 1.f) * c0);
          y[j] = a * __builtin_amdgcn_rcpf(1.f + e) * so;
        }
        if (full) {
          TO *p = C + (size_t)(mb + acc_row0(r)) * g.ldc + cw;
#pragma unroll
          for (int j = 0; j < TN; ++j) at(p, (lofs + j * 32u) * (uint32_t)sizeof(TO)) = (TO)y[j];
        } else {
          const int m = mb + acc_row(r, lane);
          if (m < M)
#pragma unroll
            for (int j = 0; j < TN; ++j) C[(size_t)m * g.ldc + cw + j * 32 + lrow] = (TO)y[j];
        }
      }
    }
    return;
  }
  // EPI_STORE / EPI_PARTIAL: C = scale * acc; EPI_RESID: C += scale * acc (one
  // rounding: scale is a power of two), the block's old values all read
  // before the first store so that their latencies overlap.
  float *C = (float *)g.C + (EPI == EPI_PARTIAL ? (size_t)tz * g.c_plane : 0);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = mw + i * 32;
    const bool full = mb + 32 <= M;
    float old[16][TN];
    if constexpr (EPI == EPI_RESID) {
      if (full) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float *p = C + (size_t)(mb + acc_row0(r)) * g.ldc + cw;
#pragma unroll
          for (int j = 0; j < TN; ++j) old[r][j] = at(p, (lofs + j * 32u) * 4u);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = min(mb + acc_row(r, lane), M - 1);
#pragma unroll
          for (int j = 0; j < TN; ++j) old[r][j] = C[(size_t)m * g.ldc + cw + j * 32 + lrow];
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float y[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        y[j] = EPI == EPI_RESID ? fmaf(acc[i][j][r], g.scale, old[r][j]) : acc[i][j][r] * g.scale;
      if (full) {
        float *p = C + (size_t)(mb + acc_row0(r)) * g.ldc + cw;
#pragma unroll
        for (int j = 0; j < TN; ++j) at(p, (lofs + j * 32u) * 4u) = y[j];
      } else {
        const int m = mb + acc_row(r, lane);
        if (m < M)
#pragma unroll
          for (int j = 0; j < TN; ++j) C[(size_t)m * g.ldc + cw + j * 32 + lrow] = y[j];
      }
    }
  }
}

// A tile configuration is a compile-time instantiation of k_gemm.
struct TileCfg {
  int bm, bn, wm, wn, rowb, p, occ, f32;
};

template <int MODE, int BM, int BN, int WM, int WN, int ROWB, int P, int EPI, int OCC, int F32>
static hipError_t run(const GemmArgs &a, int splits, hipStream_t s) {
  if constexpr (EPI == EPI_QKV && (BN / WN) % 64 != 0) {
    return hipErrorInvalidValue;  // the QK-norm epilogue needs whole heads per wave
  } else if constexpr (MODE == MODE_F32 && !F32) {
    return hipErrorInvalidValue;  // fp32 operands are built for a few tiles only
  } else if constexpr (MODE == MODE_F8W && (ROWB != 128 || EPI == EPI_GELU)) {
    return hipErrorInvalidValue;  // e4m3 weights: tiles staging 128 bytes of A per row, decoder epilogues
  } else {
    constexpr int lds_bytes = P * (BM + (MODE == MODE_F8W ? BN / 2 : BN)) * ROWB;
    auto kern = k_gemm<MODE, BM, BN, WM, WN, ROWB, P, EPI, OCC>;
    static const hipError_t attr = hipFuncSetAttribute(
        (const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (attr != hipSuccess) return attr;
    dim3 grid(a.N / BN, (a.M + BM - 1) / BM, splits);
    hipLaunchKernelGGL(kern, grid, dim3(64 * WM * WN), lds_bytes, s, a);
    return hipGetLastError();
  }
}


// Tile table: id -> instantiation (bm, bn, wave layout wm x wn, bytes of K
// per row per stage, LDS ring stages, workgroups per CU, built for fp32
// operands too). The LDS ring (P * (bm + bn) * rowb bytes, bn / 2 for e4m3
// weights) must fit 160 KB / occ; the planner skips a tile whose ring does
// not fit the operand format. bm * rowb / 16 and bn * rowb / 16 must be
// multiples of 64 (whole 64-chunk DMA groups).
#define MTE_TILE_TABLE(X)                    \
  X(0, 256, 256, 2, 2, 64, 4, 1, 0)          \
  X(1, 256, 192, 2, 2, 64, 4, 1, 0)          \
  X(2, 192, 256, 2, 2, 64, 4, 1, 0)          \
  X(3, 192, 192, 2, 2, 64, 5, 1, 0)          \
  X(4, 192, 192, 2, 2, 128, 3, 1, 0)         \
  X(5, 256, 128, 2, 2, 128, 3, 1, 0)         \
  X(6, 256, 128, 2, 2, 64, 6, 1, 0)          \
  X(7, 128, 256, 2, 2, 64, 6, 1, 0)          \
  X(8, 192, 128, 2, 2, 128, 3, 1, 0)         \
  X(9, 128, 128, 2, 2, 128, 4, 1, 1)         \
  X(10, 128, 128, 2, 2, 64, 4, 2, 0)         \
  X(11, 256, 128, 4, 1, 64, 6, 1, 0)         \
  X(12, 128, 128, 4, 1, 128, 4, 1, 1)        \
  X(13, 128, 64, 4, 1, 64, 4, 2, 1)          \
  X(14, 96, 128, 1, 4, 128, 4, 1, 0)         \
  X(15, 64, 256, 1, 4, 128, 3, 1, 0)         \
  X(16, 64, 128, 2, 2, 64, 4, 2, 1)          \
  X(17, 32, 256, 1, 4, 128, 3, 1, 1)         \
  X(18, 192, 64, 2, 2, 128, 4, 1, 0)         \
  X(19, 96, 256, 1, 4, 128, 3, 1, 0)         \
  X(20, 192, 192, 2, 2, 64, 3, 2, 0)         \
  X(21, 256, 128, 2, 2, 64, 3, 2, 0)         \
  X(22, 128, 256, 2, 2, 64, 3, 2, 0)         \
  X(23, 128, 128, 4, 1, 64, 4, 2, 0)         \
  X(24, 256, 128, 4, 1, 64, 3, 2, 0)         \
  X(25, 192, 128, 2, 2, 64, 3, 2, 0)         \
  X(26, 256, 256, 2, 4, 64, 4, 1, 0)         \
  X(27, 256, 256, 4, 2, 64, 4, 1, 0)         \
  X(28, 256, 128, 4, 2, 64, 6, 1, 0)         \
  X(29, 128, 256, 2, 4, 64, 6, 1, 0)         \
  X(30, 128, 128, 2, 4, 128, 4, 1, 0)         \
  X(31, 384, 192, 4, 2, 64, 4, 1, 0)         \
  X(32, 192, 384, 2, 4, 64, 4, 1, 0)         \
  X(33, 192, 384, 2, 4, 128, 2, 1, 0)        \
  X(34, 256, 256, 2, 4, 128, 2, 1, 0)        \
  X(35, 192, 384, 2, 4, 64, 3, 1, 0)         \
  X(36, 128, 128, 4, 1, 128, 2, 2, 0)        \
  X(37, 192, 128, 2, 2, 128, 2, 1, 0)        \
  X(38, 256, 256, 4, 2, 128, 2, 1, 0)        \
  X(39, 96, 64, 3, 2, 64, 16, 1, 0)          \
  X(40, 96, 64, 3, 2, 64, 8, 2, 0)           \
  X(41, 96, 128, 3, 2, 64, 10, 1, 0)         \
  X(42, 96, 64, 3, 2, 128, 8, 1, 0)          \
  X(43, 128, 64, 4, 1, 64, 12, 1, 0)         \
  X(44, 96, 128, 3, 2, 128, 5, 1, 0)         \
  X(45, 96, 256, 3, 2, 64, 6, 1, 0)          \
  X(46, 192, 128, 6, 1, 128, 2, 1, 0)        \
  X(47, 192, 128, 6, 1, 128, 3, 1, 0)


template <int MODE, int EPI>
static hipError_t run_id(int id, const GemmArgs &a, int splits, hipStream_t s) {
  switch (id) {
#define MTE_TILE_CASE(idv, bm, bn, wm, wn, rowb, p, occ, f32) \
  case idv: return run<MODE, bm, bn, wm, wn, rowb, p, EPI, occ, f32>(a, splits, s);
    MTE_TILE_TABLE(MTE_TILE_CASE)
#undef MTE_TILE_CASE
  }
  return hipErrorInvalidValue;
}

template <int MODE>
static hipError_t launch_mode(int epi, int tile, int splits, const GemmArgs &a, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return run_id<MODE, EPI_STORE>(tile, a, splits, s);
    case EPI_SWIGLU: return run_id<MODE, EPI_SWIGLU>(tile, a, splits, s);
    case EPI_RESID: return run_id<MODE, EPI_RESID>(tile, a, splits, s);
    case EPI_QKV: return run_id<MODE, EPI_QKV>(tile, a, splits, s);
    case EPI_GELU: return run_id<MODE, EPI_GELU>(tile, a, splits, s);
    default: return run_id<MODE, EPI_PARTIAL>(tile, a, splits, s);
  }
}

}  // namespace mte
