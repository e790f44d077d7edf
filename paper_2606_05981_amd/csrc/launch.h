// Host-side launchers of the encoder kernels (internal to libmte).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mte {

// Arithmetic of the matrix-core steps.
enum Mode {
  MODE_F32 = 0,     // fp32 weights and activations, fp32 MFMA
  MODE_BF16X2 = 1,  // bf16 weights; activations as bf16 hi + lo planes, bf16 MFMA
};

// Storage formats of activation buffers.
enum Fmt {
  FMT_F32 = 0,
  FMT_BF16 = 1,
  FMT_BF16X2 = 2,   // two bf16 planes [rows, cols]: hi, and lo = bf16(x - hi) at +plane elements
};

enum Epilogue {
  EPI_STORE = 0,   // C (float) [m, n] = acc
  EPI_SWIGLU = 1,  // gate/up rows interleaved in blocks of 32: C[m, f] = silu(gate) * up,
                   // written as float (MODE_F32) or bf16 hi/lo planes (MODE_BF16X2)
  EPI_RESID = 2,   // C (float residual stream) [m, n] += acc
  EPI_PARTIAL = 3, // C (float) + split * c_plane [m, n] = acc: the partial sum of one K split
  EPI_QKV = 4,     // C (float) [m, n] = acc, q and k heads RMS-normalised per head and rotated
};

// Parameters of EPI_QKV: columns [0, nq_cols) are q heads, [nq_cols,
// rot_cols) k heads (hd columns each), the rest (v) is stored as is. Row m
// (token m) rotates pair (c, c + hd/2) of a head by the angle whose cos / sin
// are rcos / rsin [m * hd/2 + c]. qn / kn: per-head RMSNorm gains [hd], or
// both null (no QK-norm).
struct QkvEpi {
  const float *rcos, *rsin, *qn, *kn;
  int rot_cols, nq_cols, hd;
  float eps;
};

// C = A[M, K] * W[N, K]^T. MODE_F32: A, W float. MODE_BF16X2: A = A_hi + A_lo
// (bf16 planes), W bf16. ldc: C's row pitch in elements; c_plane: distance
// in elements between the hi and lo planes of a bf16x2 C.
// The planner may split K (small M only) when the partial sums fit the
// workspace ws (ws_elems floats; ws may be null): the product is then NOT
// finished -- *splits_out (> 1) partial sums [M, N] (row pitch N, M*N
// elements apart) are left in ws, in split order, for the consumer to add
// up and apply `epi` to (for EPI_SWIGLU: the raw interleaved gate/up
// columns). Otherwise *splits_out = 0 and C holds the result.
// qe: the EPI_QKV parameters (else ignored, may be null). With a K split,
// EPI_QKV's normalisation and rotation are left to the consumer as well.
hipError_t launch_gemm(int mode, int epi, const void *A, const void *A_lo, const void *W, void *C,
                       size_t c_plane, int M, int N, int K, int ldc, float *ws, size_t ws_elems,
                       int *splits_out, const QkvEpi *qe, hipStream_t s);

// The same with an explicit tile configuration (index into the GEMM tile
// table) and number of K splits (> 1 only with EPI_PARTIAL); used for
// tuning. Returns hipErrorInvalidValue if the tile does not fit the shape.
hipError_t launch_gemm_tile(int mode, int epi, int tile, int splits, const void *A, const void *A_lo,
                            const void *W, void *C, size_t c_plane, int M, int N, int K, int ldc,
                            const QkvEpi *qe, hipStream_t s);

// Per-row RMSNorm: out[r, :] = x[r, :] / sqrt(mean(x[r,:]^2) + eps) * g with
// x = in + parts[0] + ... + parts[nparts-1] (float [rows, D] partial sums,
// rows*D elements apart, added in that order; parts may be null).
// in: `in_fmt` (FMT_F32 or FMT_BF16) [rows, D]; when copy_to != nullptr x is
// also written to copy_to as float (copy_to may be in: the residual stream
// takes the partial sums this way). g: float [D]. out: `out_fmt`, lo plane
// at out + out_plane elements for FMT_BF16X2.
hipError_t launch_rmsnorm(int in_fmt, int out_fmt, const void *in, float *copy_to, const float *parts,
                          int nparts, const float *g, void *out, size_t out_plane, int rows, int D,
                          float eps, hipStream_t s);

// h[rows, D] += parts[0] + ... + parts[nparts-1] (float partial sums, rows*D
// elements apart, in that order). D a multiple of 4.
hipError_t launch_resid_add(float *h, const float *parts, int nparts, int rows, int D, hipStream_t s);

// out[r, f] = silu(gate) * up with gate and up summed from nparts partial
// sums [rows, 2F] of the interleaved gate/up projection (block b of 64
// columns: gate 32b..32b+31, then up 32b..32b+31). out: FMT_F32 float
// [rows, F], or FMT_BF16X2 bf16 hi / lo planes out_plane elements apart.
hipError_t launch_swiglu_parts(int out_fmt, const float *parts, int nparts, int rows, int F, void *out,
                               size_t out_plane, hipStream_t s);

struct RopeParams {
  double inv_freq[64];       // theta^(-2j/d) for pair j
  uint8_t axis[64];          // position axis (0 t, 1 h, 2 w) of pair j
};

// Rotary table of T tokens: rcos / rsin [T, half] = cos / sin of
// pos_thw[axis(j)][t] * inv_freq[j] (float64 angle and sincos, rounded).
hipError_t launch_rope_table(const int32_t *pos_thw, int T, int half, const RopeParams &rp, float *rcos,
                             float *rsin, hipStream_t s);

// QKV projection finished from nparts partial sums [T, (Hq+2Hkv)*d]
// (T*(Hq+2Hkv)*d elements apart, added in order) into qkv, with the q and k
// heads normalised and rotated as by EPI_QKV (qe; v copied).
hipError_t launch_qkv_parts(float *qkv, const float *parts, int nparts, int T, int Hq, int Hkv,
                            const QkvEpi &qe, hipStream_t s);

// Causal GQA attention over packed sequences. qkv: fp32 [T, (Hq+2Hkv)*d],
// q heads first, then k, then v (q and k already normalised and rotated).
// o: [T, Hq*d] as float (MODE_F32) or bf16 hi/lo planes o_plane elements
// apart (MODE_BF16X2). cu: host int32[batch+1] sequence offsets. Launches in
// chunks of <= 256 sequences.
hipError_t launch_attention(int mode, const float *qkv, void *o, size_t o_plane, const int32_t *cu,
                            int batch, int Hq, int Hkv, int d, hipStream_t s);

// Positions of packed sequences (see mte_build_positions).
hipError_t launch_positions(const int32_t *layouts5, int batch, int32_t *pos_thw, int T,
                            hipStream_t s);

// dst[i] = (float) src[i] for n elements of storage format src_fmt (FMT_F32 / FMT_BF16).
hipError_t launch_to_f32(int src_fmt, const void *src, float *dst, int n, hipStream_t s);

// Packs gate [F, D] and up [F, D] (element size esize bytes) into dst [2F, D]:
// block b of 64 rows holds gate rows 32b..32b+31 then up rows 32b..32b+31.
hipError_t launch_interleave_gate_up(int esize, const void *gate, const void *up, void *dst,
                                     int F, int D, hipStream_t s);

}  // namespace mte
