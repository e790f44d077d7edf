/*
 * mte.h -- C ABI of the MI355X (gfx950) multimodal text-encoder prefill.
 *
 * The operation. The paper's text encoder is a Qwen3-VL decoder that jointly
 * attends to the merged image-patch tokens of a source frame and to the
 * instruction tokens (Sec. I; Sec. III-A). Buffered frames are encoded in one
 * batched call, each frame an independent sequence (Sec. III-B, "Asymmetric
 * batched dispatch"; Table "tab:batch"). Its rotary-position step is where the
 * reference stack stalls on a device-to-host read (Sec. III-B, "CUDA-stream
 * pipelining"); here positions are built and consumed on the device and the
 * host never reads device memory inside mte_encode / mte_build_positions.
 *
 * One call of mte_encode computes, for every packed sequence independently:
 *
 *   x = embeds
 *   per layer:  a = RMSNorm(x)*g_attn;  q,k,v = a Wq^T, a Wk^T, a Wv^T
 *               [qk_norm] q,k = RMSNorm_head(q)*g_q, RMSNorm_head(k)*g_k
 *               q,k = M-RoPE(q,k; (t,h,w) positions)
 *               o = causal GQA softmax(q k^T / sqrt(d)) v   (own sequence only)
 *               x += o Wo^T
 *               m = RMSNorm(x)*g_mlp;  x += (silu(m Wg^T) * m Wu^T) Wd^T
 *   out = RMSNorm(x)*g_final
 *
 * Conventions for every entry point:
 *  - "device" pointers are HIP device memory of the device current at
 *    mte_encoder_create; "host" pointers are ordinary host memory.
 *  - The caller owns every pointer it passes. The library owns the encoder,
 *    its repacked weight copies and its workspace.
 *  - Return values are mte_status codes (0 = success, negative = error).
 *    Argument and capacity checks run on the host before any HIP call, so an
 *    error return means nothing was enqueued. No entry point aborts.
 *  - mte_encode, mte_encode_layers and mte_build_positions only enqueue work
 *    on the given stream: no allocation, no device-to-host copy, no
 *    synchronisation. They can be captured into a HIP graph. Faults of the
 *    enqueued kernels surface at the caller's next synchronisation.
 *  - One encoder serves one stream at a time: its workspace is shared, so
 *    calls on one encoder that overlap in time race.
 */
#ifndef MTE_H
#define MTE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MTE_F32 = 0, MTE_BF16 = 1 } mte_dtype;

typedef enum {
  MTE_OK = 0,
  MTE_E_INVALID = -1,     /* null pointer, non-positive size, inconsistent argument */
  MTE_E_CAPACITY = -2,    /* batch / tokens / sequence length beyond the encoder's capacity */
  MTE_E_HIP = -3,         /* a HIP runtime call or kernel launch failed */
  MTE_E_OOM = -4,         /* device allocation failed in mte_encoder_create */
  MTE_E_UNSUPPORTED = -5  /* valid in principle but not built: head_dim, dtype, layout */
} mte_status;

typedef enum { MTE_MROPE_SECTIONS = 0, MTE_MROPE_INTERLEAVED = 1 } mte_mrope_layout;

/* How the encoder stores its projection weights (mte_config.weight_format).
 * MTE_WEIGHTS_DTYPE: in config.dtype. MTE_WEIGHTS_E4M3: as OCP fp8 e4m3 codes
 * with one power-of-two scale per weight row, quantised at creation by
 * mte_quantize_e4m3_rows: half the bytes of bf16 per forward, which is what
 * bounds a batch of one frame. The paper leaves FP8 execution on FP8-capable
 * hardware as an unverified direction (Sec. "Negative Results and Case
 * Studies", TensorRT FP16 paragraph). Only with dtype MTE_BF16. */
typedef enum { MTE_WEIGHTS_DTYPE = 0, MTE_WEIGHTS_E4M3 = 1 } mte_weight_format;

/* Model shape and workspace capacity.
 *  hidden = D, n_q_heads = Hq, n_kv_heads = Hkv (Hq % Hkv == 0; query head h
 *  reads kv head h / (Hq/Hkv)), head_dim = d in {64, 128}, ffn = F.
 *  rms_eps: every RMSNorm is x / sqrt(mean(x^2) + rms_eps) * gain.
 *  rope_theta: rotary pair j (element j with j + d/2) of a head turns by
 *  p * rope_theta^(-2j/d), p the token's position on the pair's axis.
 *  mrope_section[3]: number of rotary pairs driven by t, h, w; sum == d/2.
 *  mrope_layout: MTE_MROPE_SECTIONS assigns pairs [0,s_t) to t, then s_h to
 *  h, then s_w to w; MTE_MROPE_INTERLEAVED makes pair j h-driven if
 *  j%3==1 && j<3*s_h, w-driven if j%3==2 && j<3*s_w, t-driven otherwise.
 *  qk_norm: 1 applies a per-head RMSNorm (gain q_norm / k_norm) to q and k
 *  before the rotation.
 *  dtype: storage type of the weights and the embeddings (MTE_BF16: bf16
 *  storage, fp32 accumulation and an fp32 residual stream; MTE_F32: fp32
 *  throughout). With MTE_BF16 the projections run on fp16 matrix-core
 *  operands: each weight matrix is converted at creation to fp16 times a
 *  power of two that puts its largest magnitude in [2^14, 2^15), which holds
 *  every bf16 weight of magnitude at least 2^-31 of that maximum exactly
 *  (smaller ones round, with an absolute error below 2^-40 of the maximum);
 *  activations are rounded once to fp16 behind power-of-two pre-scales
 *  derived from static bounds. out_dtype: type of out_hidden.
 *  max_tokens / max_batch / max_seq: capacity the workspace is sized for.
 *  weight_format: mte_weight_format (MTE_WEIGHTS_E4M3 needs dtype MTE_BF16,
 *  else MTE_E_UNSUPPORTED). With e4m3 weights the encoder computes the same
 *  forward with every linear weight replaced by its dequantised value
 *  code * scale; activations, norms and attention are unchanged. */
typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn;
  float rms_eps, rope_theta;
  int32_t mrope_section[3];
  int32_t mrope_layout;
  int32_t qk_norm;
  int32_t dtype;
  int32_t out_dtype;
  int32_t max_tokens, max_batch, max_seq;
  int32_t weight_format;
} mte_config;

/* One layer's weights: device pointers of type config.dtype, linear weights
 * in nn.Linear layout [out_features, in_features], row-major:
 *  attn_norm [D], w_q [Hq*d, D], w_k [Hkv*d, D], w_v [Hkv*d, D],
 *  q_norm [d], k_norm [d] (ignored when qk_norm == 0; may then be NULL),
 *  w_o [D, Hq*d], mlp_norm [D], w_gate [F, D], w_up [F, D], w_down [D, F]. */
typedef struct {
  const void *attn_norm, *w_q, *w_k, *w_v, *q_norm, *k_norm, *w_o,
             *mlp_norm, *w_gate, *w_up, *w_down;
} mte_layer_weights;

/* layers: HOST array of n_layers entries; final_norm: device [D]. */
typedef struct {
  const mte_layer_weights *layers;
  const void *final_norm;
} mte_weights;

typedef struct mte_encoder mte_encoder;

/* Layout of one packed sequence: n_text_before text tokens, then an image
 * grid of grid_t x grid_h x grid_w merged-patch tokens (t-major, then rows,
 * then columns), then n_text_after text tokens. */
typedef struct {
  int32_t n_text_before, grid_t, grid_h, grid_w, n_text_after;
} mte_seq_layout;

/* Host-only check of a configuration. Returns MTE_OK, MTE_E_INVALID (null,
 * non-positive sizes, Hq % Hkv != 0, sections not summing to d/2, bad enum)
 * or MTE_E_UNSUPPORTED (head_dim not 64/128, D or F not multiples of 256,
 * capacities beyond the built limits: at most 2^24 - 1 tokens, and every
 * projection operand -- max_tokens x its K, or a weight matrix -- under 4 GiB).
 * Makes no HIP call. */
int mte_config_validate(const mte_config *cfg);

/* Host-only check of one batch against a configuration (the checks
 * mte_encode runs before enqueuing anything). seq_lens: HOST int32[batch],
 * each > 0. On success *total_tokens (if non-NULL) receives sum(seq_lens).
 * Errors: MTE_E_INVALID (null, batch <= 0, a length <= 0), MTE_E_CAPACITY
 * (batch > max_batch, a length > max_seq, total > max_tokens). */
int mte_check_batch(const mte_config *cfg, const int32_t *seq_lens, int32_t batch,
                    int32_t *total_tokens);

/* Creates an encoder on the current device: validates cfg, allocates the
 * workspace for cfg's capacities, copies the weights into library-owned,
 * repacked device buffers (fused QKV rows; gate/up rows interleaved) on
 * `stream`, and synchronises that stream once. The caller's weight buffers
 * may be freed when it returns. *out is set only on success.
 * Errors: MTE_E_INVALID, MTE_E_UNSUPPORTED, MTE_E_OOM, MTE_E_HIP. */
int mte_encoder_create(const mte_config *cfg, const mte_weights *weights,
                       hipStream_t stream, mte_encoder **out);

/* The batched prefill (the operation described at the top of this file).
 *  embeds:     device [T, D], config.dtype, T = sum(seq_lens); sequences are
 *              packed back to back in seq_lens order, no padding.
 *  pos_thw:    device int32 [3, T]: row 0 = t, row 1 = h, row 2 = w position
 *              of each token (0 <= pos < 2^24); e.g. from mte_build_positions.
 *              Not validated on the device.
 *  seq_lens:   HOST int32[batch]. It is read during the call only.
 *  out_hidden: device [T, D], config.out_dtype; must not overlap embeds.
 * Errors: MTE_E_INVALID, MTE_E_CAPACITY, MTE_E_HIP. */
int mte_encode(mte_encoder *enc, const void *embeds, const int32_t *pos_thw,
               const int32_t *seq_lens, int32_t batch, void *out_hidden,
               hipStream_t stream);

/* mte_encode for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same forward, arguments and errors as mte_encode, with the activations
 * held in the library's static device array of MTE_STATIC_SCRATCH_BYTES
 * (one per GPU, reserved when the library's device code is loaded on that
 * GPU and kept until the process ends) instead of the encoder's workspace.
 * It calls no hipMalloc / hipFree or other allocating routine and only
 * enqueues work on `stream`.
 * Capacity: at most MTE_STATIC_MAX_BATCH sequences, and the activations of
 * T = sum(seq_lens) tokens, T * (4 D + 4 (Hq + 2 Hkv) d + 4 d + e (D + Hq d
 * + F)) bytes with e = 2 for MTE_BF16 (4 for MTE_F32) plus 256-byte
 * alignment of seven regions, must fit MTE_STATIC_SCRATCH_BYTES (about 736
 * tokens of the 2048-wide bf16 model); the rest of the array holds K-split
 * partial sums. Beyond that: MTE_E_CAPACITY, checked before any HIP call.
 * The usual mte_encode limits (max_batch, max_seq, max_tokens) apply too.
 * Every call on one GPU shares that GPU's array, whichever encoder it
 * serves: calls that overlap in time on one GPU race. No part of the array
 * needs to start at zero (every value is written before it is read).
 * Results equal mte_encode's bit for bit whenever the batch's K-split
 * partial sums fit the array (then both take the same launch plan). */
#define MTE_STATIC_SCRATCH_BYTES (32u << 20)
#define MTE_STATIC_MAX_BATCH 1024
int mte_encode_static(mte_encoder *enc, const void *embeds, const int32_t *pos_thw,
                      const int32_t *seq_lens, int32_t batch, void *out_hidden,
                      hipStream_t stream);

/* Runs decoder layers [layer_begin, layer_end) on an fp32 residual stream
 * without the final norm: h_out = layers(h_in). h_in / h_out: device float
 * [T, D] (they may be the same buffer). Other arguments as mte_encode.
 * For per-layer comparisons and for splitting the stack across calls.
 * Errors: as mte_encode, plus MTE_E_INVALID for a bad layer range. */
int mte_encode_layers(mte_encoder *enc, const float *h_in, const int32_t *pos_thw,
                      const int32_t *seq_lens, int32_t batch, int32_t layer_begin,
                      int32_t layer_end, float *h_out, hipStream_t stream);

/* Builds the (t,h,w) positions of a packed batch on the device. This is the
 * step whose host round trip the paper's encoder pays inside its rotary-position
 * code and has to hide on a side stream (Sec. I; Sec. III-B, "CUDA-stream
 * pipelining"); here the positions follow from the host layout descriptors
 * alone and are written by one kernel, so no device value is ever read back.
 * Each sequence is one frame's source-image grid and its instruction, attended
 * jointly (Sec. I; Sec. III-A, "Notation and Setup").
 *  layouts: HOST [batch]; pos_thw: device int32 [3, T], T = sum of lengths.
 * Text before an image counts up t=h=w=i; image token k of a (gt,gh,gw) grid
 * after o text tokens gets (o + k/(gh*gw), o + (k/gw)%gh, o + k%gw); text
 * after the image starts one past the largest earlier position and counts up.
 * Errors: MTE_E_INVALID (null, batch <= 0, a negative count, an empty
 * sequence, a grid with some but not all extents zero, T >= 2^24),
 * MTE_E_HIP. */
int mte_build_positions(const mte_seq_layout *layouts, int32_t batch,
                        int32_t *pos_thw, hipStream_t stream);

/* Shared prefix (the paper's system prompt / chat template, identical for
 * every frame, Sec. V). Under causal attention a prefix's hidden states, keys
 * and values do not depend on what follows it, so they are computed once per
 * batch instead of once per sequence.
 *
 * mte_encoder_reserve_prefix allocates the per-layer key/value cache for
 * prefixes of up to max_prefix tokens (n_layers * max_prefix *
 * (Hq + 2 Hkv) * d floats; replaces an earlier reservation). It may
 * synchronise the device and allocate; call it next to mte_encoder_create.
 * Errors: MTE_E_INVALID (null, max_prefix <= 0 or beyond max_tokens /
 * max_seq), MTE_E_UNSUPPORTED (no layers), MTE_E_OOM. */
int mte_encoder_reserve_prefix(mte_encoder *enc, int32_t max_prefix);

/* Batched encode of sequences that all start with the same prefix_len-token
 * prefix. The result equals mte_encode of the full sequences
 * [prefix ++ own tokens of sequence b]: out_prefix receives the prefix's
 * rows (identical for every sequence, written once) and out_hidden the
 * sequences' own rows, packed as in mte_encode.
 *  prefix_embeds: device [prefix_len, D], config.dtype.
 *  prefix_pos:    device int32 [3, prefix_len], the prefix's (t,h,w) positions.
 *  embeds:        device [T, D], the sequences' own tokens, T = sum(seq_lens).
 *  pos_thw:       device int32 [3, T], their positions within the full
 *                 sequences (i.e. continuing after the prefix).
 *  seq_lens:      HOST int32[batch], own-token counts (without the prefix).
 *  out_prefix:    device [prefix_len, D], config.out_dtype.
 *  out_hidden:    device [T, D], config.out_dtype.
 * Only enqueues work on `stream`, like mte_encode; needs a prior
 * mte_encoder_reserve_prefix. Output buffers must not overlap the inputs or
 * each other. Errors: MTE_E_INVALID (null, no reservation, prefix_len <= 0,
 * overlap, bad seq_lens), MTE_E_CAPACITY (prefix_len > the reservation,
 * prefix_len + a sequence > max_seq, batch / tokens beyond capacity),
 * MTE_E_HIP. */
int mte_encode_prefixed(mte_encoder *enc, const void *prefix_embeds, const int32_t *prefix_pos,
                        int32_t prefix_len, const void *embeds, const int32_t *pos_thw,
                        const int32_t *seq_lens, int32_t batch, void *out_prefix, void *out_hidden,
                        hipStream_t stream);

/* Frees the encoder (synchronises the device first). NULL is a no-op. */
void mte_encoder_destroy(mte_encoder *enc);

/* OCP fp8 e4m3 quantisation of the rows of a matrix, the weight format of
 * MTE_WEIGHTS_E4M3 (e4m3: sign, 4 exponent bits of bias 7, 3 significand
 * bits; subnormals below 2^-6 in steps of 2^-9; largest finite 448; codes
 * 0x7F / 0xFF are NaN and never produced).
 *  src: device [rows, cols] of src_dtype (MTE_F32 or MTE_BF16), row-major.
 *  scales: device float[rows] out: scales[r] = 2^e_r with e_r the smallest
 *    integer such that max_c |src[r,c]| <= 448 * 2^e_r (1.0 for an all-zero
 *    row).
 *  codes: device uint8[rows, cols] out: the e4m3 code nearest to
 *    src[r,c] / 2^e_r (an exact division), ties to the even significand;
 *    a result of zero is coded +0 (0x00) whatever the sign.
 * The dequantised weight is decode(codes[r,c]) * scales[r]. Enqueues one
 * kernel on `stream`; no allocation, no synchronisation.
 * Errors: MTE_E_INVALID (null pointer, rows or cols <= 0, bad dtype),
 * MTE_E_HIP (launch failure). */
int mte_quantize_e4m3_rows(const void *src, int32_t src_dtype, int32_t rows, int32_t cols,
                           uint8_t *codes, float *scales, hipStream_t stream);

/* Static description of a status code. Never NULL. */
const char *mte_status_string(int status);

/* Kernel timing for roofline measurements (measurement hooks, no part of the
 * forward; they add nothing to a call while disabled). While enabled for a kernel class,
 * every launch of that class inside mte_encode / mte_encode_layers is
 * bracketed by HIP events on the launch stream (at most `capacity` pairs
 * are kept; `capacity` is allocated here, not in the encode calls).
 * kernel_class: 0 = QKV GEMM, 1 = attention, 2 = O-proj GEMM,
 * 3 = gate/up GEMM, 4 = down GEMM. mte_timing_read synchronises the recorded
 * events and returns the number of launches and their summed duration in
 * milliseconds, then clears the record. Errors: MTE_E_INVALID, MTE_E_HIP. */
int mte_timing_enable(mte_encoder *enc, int32_t kernel_class, int32_t capacity);
int mte_timing_read(mte_encoder *enc, int32_t *launches, double *total_ms);
int mte_timing_disable(mte_encoder *enc);

#ifdef __cplusplus
}
#endif
#endif /* MTE_H */
