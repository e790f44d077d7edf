/*
 * mte_vision.h -- C ABI of the vision tower on MI355X (gfx950): images -> the
 * image-token embeddings the text encoder (mte.h) consumes.
 *
 * The operation. The paper's text encoder takes the source frame through the
 * Qwen3-VL vision tower, which turns the 256x256 source patch into the image
 * tokens the decoder attends to jointly with the instruction (Sec. I;
 * Sec. III-A, where the prompt template's image placeholder is filled by the
 * vision tower). The paper gives no architecture for it; this library builds
 * a plain pre-norm ViT with 2-D rotary positions and a 2x2 patch merger:
 *
 *   x_p   = patch_p W_patch^T + b_patch           (patch: C x patch x patch pixels)
 *   per block:  a = LN(x) g1 + b1;  q,k,v = a W_qkv^T + b_qkv
 *               q,k = RoPE2d(q,k; patch row, patch column)
 *               o = softmax(q k^T / sqrt(d)) v      (bidirectional, one image)
 *               x += o W_o^T + b_o
 *               m = LN(x) g2 + b2;  x += gelu(m W_fc1^T + b_fc1) W_fc2^T + b_fc2
 *   per group of merge x merge patches (row-major over the image):
 *               u = concat(LN(x_p) g_m + b_m over the group's patches)
 *               e = gelu(u W_m1^T + b_m1) W_m2^T + b_m2        (one image token)
 *
 * LN normalises by the mean and the biased variance (eps inside the square
 * root); gelu is the tanh form 0.5 z (1 + tanh(sqrt(2/pi)(z + 0.044715 z^3)));
 * RoPE2d rotates pair j (element j with j + d/2) of a head by
 * pos * rope_theta^(-2j/d), pos the patch row for j < d/4, the patch column
 * otherwise. Image tokens come out row-major over the merge groups, which is
 * the order of an image grid in mte_seq_layout.
 *
 * Conventions as in mte.h: device / host pointers, caller-owned buffers,
 * negative mte_status codes, host-side checks before any HIP call,
 * mte_vision_encode only enqueues work (no allocation, copy back or
 * synchronisation; graph-capturable), one vision encoder per stream at a time.
 */
#ifndef MTE_VISION_H
#define MTE_VISION_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "mte.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Shapes and capacity.
 *  depth blocks of width hidden = n_heads * head_dim (head_dim 64 or 128),
 *  MLP width ffn; patch x patch pixel patches of in_channels channels;
 *  merge x merge patches per image token; out_hidden = width of the image
 *  tokens (the text encoder's hidden size). hidden, ffn, out_hidden and
 *  in_channels * patch * patch must be multiples of 64, hidden <= 4096.
 *  dtype: weights and pixels (MTE_BF16: bf16 weights, fp16 matrix-core
 *  operands with fp32 accumulation, fp32 residual stream; pixels must lie
 *  in fp16's range; MTE_F32: fp32 throughout). out_dtype: the output.
 *  max_images / max_side: capacity (images per call, largest H or W). */
typedef struct {
  int32_t depth, hidden, n_heads, head_dim, ffn;
  int32_t patch, merge, in_channels, out_hidden;
  float ln_eps, rope_theta;
  int32_t dtype, out_dtype;
  int32_t max_images, max_side;
} mte_vision_config;

/* One block's weights, device pointers of config.dtype, nn.Linear layout
 * [out, in] row-major: ln1_g, ln1_b [hidden]; w_qkv [3*hidden, hidden] (q,
 * k, v rows, heads contiguous), b_qkv [3*hidden]; w_o [hidden, hidden],
 * b_o [hidden]; ln2_g, ln2_b [hidden]; w_fc1 [ffn, hidden], b_fc1 [ffn];
 * w_fc2 [hidden, ffn], b_fc2 [hidden]. */
typedef struct {
  const void *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o, *ln2_g, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} mte_vision_layer_weights;

/* patch_w [hidden, in_channels*patch*patch] (a Conv2d weight flattened in
 * (channel, row, column) order), patch_b [hidden]; layers: HOST array of
 * depth entries; merge_ln_g, merge_ln_b [hidden]; merge_w1 [mh, mh] with
 * mh = merge*merge*hidden (input = the group's patches concatenated in
 * group order), merge_b1 [mh]; merge_w2 [out_hidden, mh], merge_b2
 * [out_hidden]. */
typedef struct {
  const void *patch_w, *patch_b;
  const mte_vision_layer_weights *layers;
  const void *merge_ln_g, *merge_ln_b, *merge_w1, *merge_b1, *merge_w2, *merge_b2;
} mte_vision_weights;

typedef struct mte_vision mte_vision;

/* Host-only check: MTE_OK, MTE_E_INVALID (null, non-positive sizes,
 * hidden != n_heads*head_dim, bad enum) or MTE_E_UNSUPPORTED (head_dim not
 * 64/128, widths not multiples of 64, hidden > 4096, more than 2^24 patches,
 * or a projection operand -- patches x its K, or a weight matrix -- of 4 GiB
 * or more). */
int mte_vision_config_validate(const mte_vision_config *cfg);

/* Copies and repacks the weights (the caller may free its copies after
 * return), allocates the workspace for max_images images of max_side^2
 * pixels; may synchronise `stream`. Errors: those of validate, MTE_E_OOM,
 * MTE_E_HIP. */
int mte_vision_create(const mte_vision_config *cfg, const mte_vision_weights *w, hipStream_t stream,
                      mte_vision **out);

/* pixels: device [n_images, in_channels, height, width] of config.dtype.
 * out: device [n_images * (height/(patch*merge)) * (width/(patch*merge)),
 * out_hidden] of config.out_dtype, the image tokens of image 0, then 1, ...
 * height and width multiples of patch*merge, at most max_side; n_images in
 * [1, max_images]. Errors: MTE_E_INVALID (null, sizes), MTE_E_CAPACITY,
 * MTE_E_HIP. */
int mte_vision_encode(mte_vision *enc, const void *pixels, int32_t n_images, int32_t height, int32_t width,
                      void *out, hipStream_t stream);

/* The same with image i's tokens written to rows [i*image_stride,
 * i*image_stride + tokens per image) of out (image_stride >= tokens per
 * image; the rows in between are left untouched), so that the image tokens
 * land directly in a packed text-encoder input (mte_encode's embeds) whose
 * sequences each start with their image grid. Errors as mte_vision_encode,
 * and MTE_E_INVALID for a stride below the tokens per image. */
int mte_vision_encode_strided(mte_vision *enc, const void *pixels, int32_t n_images, int32_t height,
                              int32_t width, void *out, int32_t image_stride, hipStream_t stream);

/* Frees the encoder (synchronises its device); NULL is a no-op. */
void mte_vision_destroy(mte_vision *enc);

#ifdef __cplusplus
}
#endif

#endif /* MTE_VISION_H */
