// Host-side launchers of the encoder kernels (internal to libmte).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mte {

typedef _Float16 f16;

// Arithmetic of the matrix-core steps.
enum Mode {
  MODE_F32 = 0,  // fp32 weights and activations, fp32 MFMA
  MODE_F16 = 1,  // projections: fp16 operands (weights = bf16 values as power-of-two
                 // scaled fp16, exact down to 2^-31 of the matrix maximum; activations
                 // rounded once to fp16), fp32 accumulate; attention (decoder and vision
                 // tower): q, k, v and P as fp16 (power-of-two pre-scales), fp32
                 // accumulate and softmax (launch_attention_h), output rounded to fp16
  MODE_F8W = 2,  // projections only: fp16 activations as MODE_F16, weights OCP e4m3 codes
                 // with a power-of-two scale per weight row, widened to fp16 for the MFMAs
};

// Storage formats of activation buffers.
enum Fmt {
  FMT_F32 = 0,
  FMT_BF16 = 1,
  FMT_F16 = 2,
};

enum Epilogue {
  EPI_STORE = 0,   // C (float) [m, n] = scale * acc
  EPI_SWIGLU = 1,  // gate/up rows interleaved in blocks of 16: C[m, f] = out_scale *
                   // silu(gate) * up, written as float (MODE_F32) or fp16 (MODE_F16)
  EPI_RESID = 2,   // C (float residual stream) [m, n] += scale * acc
  EPI_PARTIAL = 3, // C (float) + split * c_plane [m, n] = scale * acc: one K split's partial sum
  EPI_QKV = 4,     // C (float) [m, n] = scale * acc, q and k heads RMS-normalised per head and rotated
  EPI_GELU = 5,    // C [m, n] = out_scale * gelu_tanh(scale * acc), float (MODE_F32) or fp16
};

// Parameters of EPI_QKV: columns [0, nq_cols) are q heads, [nq_cols,
// rot_cols) k heads (hd columns each), the rest (v) is stored as is. Row m
// (token m) rotates pair (c, c + hd/2) of a head by the angle whose cos / sin
// are rcos / rsin [m * hd/2 + c]. qn / kn: per-head RMSNorm gains [hd], or
// both null (no QK-norm).
// With qk non-null the result is written in the operand layout of
// launch_attention_h instead of fp32 rows: q and k heads as fp16 rows
// qk [m, rot_cols] times q_pre / k_pre, and v as fp16 V^T tiles vt (see
// launch_attention_h) times v_pre, the rows of a 32-token tile past the last
// token written as zeros. q_pre, k_pre, v_pre: powers of two that keep the
// values in fp16 range.
struct QkvEpi {
  const float *rcos, *rsin, *qn, *kn;
  int rot_cols, nq_cols, hd;
  float eps;
  f16 *qk = nullptr;
  f16 *vt = nullptr;
  float q_pre = 1.f, k_pre = 1.f, v_pre = 1.f;
  int hkv = 0;
};

// C = A[M, K] * W[N, K]^T, A and W of the mode's operand type (float or
// fp16). The product is multiplied by `scale` (the inverse of the operands'
// power-of-two pre-scales; exact) before the epilogue; EPI_SWIGLU multiplies
// its fp16 output by `out_scale` (a power of two keeping it in fp16 range).
// ldc: C's row pitch in elements.
// The planner may split K (up to 2048 rows) when the partial sums fit the
// workspace ws (ws_elems floats; ws may be null): the product is then NOT
// finished -- *splits_out (> 1) scaled partial sums [M, N] (row pitch N,
// M*N elements apart) are left in ws, in split order, for the consumer to
// add up and apply `epi` to (for EPI_SWIGLU: the raw interleaved gate/up
// columns). Otherwise *splits_out = 0 and C holds the result.
// qe: the EPI_QKV parameters (else ignored, may be null). With a K split,
// EPI_QKV's normalisation and rotation are left to the consumer as well.
// MODE_F8W: W holds e4m3 codes [N, K] and col_scale [N] the scale of each
// weight row (column of the product), applied before `scale` and the
// epilogue; col_scale is ignored in the other modes.
// bias: optional float [N] added to the product (after col_scale and `scale`, before the
// epilogue); `scale` must then be a power of two, and the product is never K-split.
hipError_t launch_gemm(int mode, int epi, const void *A, const void *W, void *C, int M, int N, int K,
                       int ldc, float scale, float out_scale, float *ws, size_t ws_elems,
                       int *splits_out, const QkvEpi *qe, hipStream_t s,
                       const float *col_scale = nullptr, const float *bias = nullptr);

// The same with an explicit tile configuration (index into the GEMM tile
// table) and number of K splits (> 1 only with EPI_PARTIAL, partial sums
// c_plane elements apart); used for tuning. Returns hipErrorInvalidValue if
// the tile does not fit the shape. xcd: placement of the tiles on the eight
// XCDs, 100 xa + 10 xb + xc with xa x xb x xc = 8 groups of M tiles, N tiles
// and K splits (each XCD reads only its groups' operands); 0, or a placement
// that does not divide the grid: workgroup order by N tile.
hipError_t launch_gemm_tile(int mode, int epi, int tile, int splits, const void *A, const void *W,
                            void *C, size_t c_plane, int M, int N, int K, int ldc, float scale,
                            float out_scale, const QkvEpi *qe, hipStream_t s,
                            const float *col_scale = nullptr, const float *bias = nullptr, int xcd = 0);
int gemm_num_tiles();

// Per-row RMSNorm: out[r, :] = x[r, :] / sqrt(mean(x[r,:]^2) + eps) * g with
// x = in + parts[0] + ... + parts[nparts-1] (float [rows, D] partial sums,
// rows*D elements apart, added in that order; parts may be null).
// in: `in_fmt` (FMT_F32 or FMT_BF16) [rows, D]; when copy_to != nullptr x is
// also written to copy_to as float (copy_to may be in: the residual stream
// takes the partial sums this way). g: float [D] (a power-of-two pre-scale
// of the consuming GEMM's input is folded into it). out: `out_fmt`.
hipError_t launch_rmsnorm(int in_fmt, int out_fmt, const void *in, float *copy_to, const float *parts,
                          int nparts, const float *g, void *out, int rows, int D, float eps,
                          hipStream_t s);

// h[rows, D] += parts[0] + ... + parts[nparts-1] (float partial sums, rows*D
// elements apart, in that order). D a multiple of 4.
hipError_t launch_resid_add(float *h, const float *parts, int nparts, int rows, int D, hipStream_t s);

// out[r, f] = out_scale * silu(gate) * up with gate and up summed from nparts
// partial sums [rows, 2F] of the interleaved gate/up projection (block b of
// 32 columns: gate 16b..16b+15, then up 16b..16b+15). out: FMT_F32 float or
// FMT_F16 [rows, F].
hipError_t launch_swiglu_parts(int out_fmt, const float *parts, int nparts, int rows, int F, void *out,
                               float out_scale, hipStream_t s);

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
// heads normalised and rotated as by EPI_QKV (qe; v copied). With qe.qk
// non-null the output goes to qe.qk / qe.vt in the attention operand layout
// (qkv unused).
hipError_t launch_qkv_parts(float *qkv, const float *parts, int nparts, int T, int Hq, int Hkv,
                            const QkvEpi &qe, hipStream_t s);

// Causal GQA attention over packed sequences in fp32 (MODE_F32). qkv: fp32
// [T, (Hq+2Hkv)*d], q heads first, then k, then v (q and k already
// normalised and rotated). prefix: fp32 [P, (Hq+2Hkv)*d] rows of a shared
// prefix (same layout; its k and v columns are read) that every sequence
// attends to in full before its own keys, or P = 0. o: fp32 [T, Hq*d]. cu:
// host int32[batch+1] sequence offsets. Launches in chunks of <= 256
// sequences. causal = 0: bidirectional (every query attends to all keys of
// its own sequence).
hipError_t launch_attention(const float *qkv, const float *prefix, int P, float *o, const int32_t *cu, int batch,
                            int Hq, int Hkv, int d, hipStream_t s, int causal = 1);

// Causal (or bidirectional) GQA attention over packed sequences on fp16
// operands laid out for the matrix cores by the QKV projection's epilogue:
//  qk: fp16 [T, (Hq + Hkv) d] rows, q heads then k heads, q times 2^-aq and
//      k times 2^-ak (sc below undoes both);
//  vt: fp16 V^T tiles [ceil(T / 32)][Hkv][d][32]: tile t holds tokens
//      32t .. 32t+31, each d row's 32 values in the order the softmax
//      probabilities come out of the score MFMA (position 16f + 8g + e holds
//      token 8 (i / 4) + 4 g + i % 4 of the tile, i = 8 f + e), rows past T
//      zero; V already times the output's pre-scale.
//  prefix / pvt: the same two layouts for P rows of a shared prefix (its k
//      heads and V^T tiles are read), or P = 0.
// o: fp16 [T, Hq d]. sc = log2(e) / sqrt(d) * 2^(aq + ak). cu: host
// int32[batch+1] offsets. Launches in chunks of <= 256 sequences.
// Two kernels: workgroups of qbw 32-query blocks x the query heads of a kv
// head copy their key tiles (and the prefix's) into LDS, 64 KB per round,
// and compute from there (qbw = 0: the default chunk), when such a workgroup
// is 4 or 8 waves; otherwise one wave per (sequence, query head, 32 queries)
// streams the tiles from global memory, or ks waves (2 or 4) split its key
// tiles (ks = 0 picks by the number of work items). qbw < 0 or ks > 0
// selects the streaming kernel; qbw > 0 requires the staged one
// (hipErrorNotSupported if qbw blocks x Hq / Hkv heads is not 4 or 8 waves).
hipError_t launch_attention_h(const f16 *qk, const f16 *vt, const f16 *prefix, const f16 *pvt, int P, f16 *o,
                              float sc, const int32_t *cu, int batch, int T, int Hq, int Hkv, int d, int causal,
                              hipStream_t s, int ks = 0, int qbw = 0);

// Positions of packed sequences (see mte_build_positions).
hipError_t launch_positions(const int32_t *layouts5, int batch, int32_t *pos_thw, int T,
                            hipStream_t s);

// dst[i] = (float) src[i] * scale for n elements of storage format src_fmt (FMT_F32 / FMT_BF16).
hipError_t launch_to_f32(int src_fmt, const void *src, float *dst, int n, float scale, hipStream_t s);

// Statistics of a [rows, cols] matrix of format src_fmt (FMT_F32 / FMT_BF16),
// for the range analysis at encoder creation: stats[0] = max |w|,
// stats[1] = max over rows of the row's L2 norm (float, device). Each row's
// norm is accumulated in fp32; stats must be zeroed first.
hipError_t launch_matrix_stats(int src_fmt, const void *src, int rows, int cols, float *stats,
                               hipStream_t s);

// Converts rows [0, rows) of src (format src_fmt, cols columns) into
// dst_fmt (bf16 -> FMT_F16, f32 -> FMT_F32 or FMT_BF16) times `scale` (a power of two), writing
// source row r to destination row map(r): map(r) = r, or with `interleave`
// the gate/up packing (src = gate or up of F = rows rows: gate row f goes to
// 32*(f/16) + f%16, up row f to 32*(f/16) + 16 + f%16, `up` selecting which).
hipError_t launch_convert_rows(int src_fmt, const void *src, int dst_fmt, void *dst, int rows, int cols,
                               float scale, int interleave, int up, hipStream_t s);

// Vision tower. Patches of n images [n, C, H, W] (in_fmt FMT_F32 / FMT_BF16)
// -> out [n * (H/patch) * (W/patch), C*patch*patch] (out_fmt FMT_F32 / FMT_F16),
// patches of an image in merge-group order (groups of merge x merge patches
// row-major over the image, row-major inside a group), each patch's vector in
// (channel, row, column) order. H and W multiples of patch * merge.
hipError_t launch_patchify(int in_fmt, const void *pixels, int n, int C, int H, int W, int patch, int merge,
                           int out_fmt, void *out, hipStream_t s);
// pos [3, n * patches per image]: t = 0, h = patch row, w = patch column (same order).
hipError_t launch_patch_positions(int32_t *pos, int n, int H, int W, int patch, int merge, hipStream_t s);
// y[r] = (x[r] - mean) / sqrt(var + eps) * g + b per row of x (float [rows, D],
// D <= 4096); y in out_fmt (FMT_F32 / FMT_F16).
hipError_t launch_layernorm(const float *x, const float *g, const float *b, int out_fmt, void *y, int rows, int D,
                            float eps, hipStream_t s);

// dst row (r / group) * group_stride + r % group = src row r of a float
// [rows, cols] matrix (dst FMT_F32 or FMT_BF16); the other dst rows are untouched.
hipError_t launch_scatter_rows(const float *src, int dst_fmt, void *dst, int rows, int cols, int group,
                               int group_stride, hipStream_t s);

// OCP e4m3 quantisation of the rows of a [rows, cols] matrix (format src_fmt,
// FMT_F32 or FMT_BF16): row r gets the scale 2^e_r with e_r the smallest
// integer such that max_c |src[r, c]| <= 448 * 2^e_r (e_r = 0 for an
// all-zero row), and code(src[r, c] / 2^e_r) per element, rounded to
// nearest, ties to even (the division is exact), zero as +0. Source row r
// goes to destination row map(r) of codes (cols bytes per row) and scales,
// map as in launch_convert_rows (interleave / up).
hipError_t launch_quantize_e4m3_rows(int src_fmt, const void *src, int rows, int cols, uint8_t *codes,
                                     float *scales, int interleave, int up, hipStream_t s);

}  // namespace mte
