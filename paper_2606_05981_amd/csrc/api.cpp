// C ABI of the encoder: argument validation, the sequence plan, weight
// repacking at creation and the per-call launch schedule. Nothing here reads
// device memory back during mte_encode / mte_encode_layers /
// mte_build_positions: the sequence plan is computed from the host lengths
// and handed to the kernels by value.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/mte.h"
#include "launch.h"

using namespace mte;

namespace {

constexpr int64_t kMaxTokens = (1 << 24) - 1;  // positions and offsets stay exact in fp32 / int32
constexpr int kNumClasses = 5;

struct LayerW {
  void *w_qkv, *w_o, *w_gu, *w_d;              // operand type (fp16, fp32 or e4m3 codes), repacked
  // e4m3 weights: the scale of every weight row (column of the product)
  const float *cs_qkv = nullptr, *cs_o = nullptr, *cs_gu = nullptr, *cs_d = nullptr;
  float *attn_norm, *mlp_norm, *q_norm, *k_norm;
  // Products are multiplied by s_* (the inverse of the weight's and the
  // activation's power-of-two pre-scales); the attention output and the
  // SwiGLU output are pre-scaled by o_pre / y_pre before rounding to fp16.
  float s_qkv = 1.f, s_o = 1.f, s_gu = 1.f, s_d = 1.f, o_pre = 1.f, y_pre = 1.f;
  // fp16 attention operands: q and k are stored times q_pre / k_pre (v times
  // o_pre); att_sc = log2(e) / sqrt(d) / (q_pre k_pre) turns their products
  // into scores in log2 units.
  float q_pre = 1.f, k_pre = 1.f, att_sc = 1.f;
};

size_t esize(int dtype) { return dtype == MTE_BF16 ? 2 : 4; }
int in_fmt(int dtype) { return dtype == MTE_BF16 ? FMT_BF16 : FMT_F32; }

// Exponent e with x in [2^(e-1), 2^e) (frexp), 0 for x <= 0.
int exp2_of(double x) {
  if (!(x > 0.0)) return 0;
  int e = 0;
  std::frexp(x, &e);
  return e;
}
// Weight pre-scale exponent: the largest magnitude lands in [2^14, 2^15),
// where every bf16 value down to 2^-31 of it converts to fp16 exactly.
int weight_shift(double maxabs) { return maxabs > 0.0 ? 15 - exp2_of(maxabs) : 0; }
// Activation pre-scale exponent (>= 0, applied as 2^-k): values bounded by
// `bound` stay within 2^15 after scaling, well inside fp16's range.
int act_shift(double bound) { return std::max(0, exp2_of(bound) - 15); }

// Bytes of the fp16 attention operands of T tokens (fp16 modes): q/k rows
// [T, (Hq + Hkv) d] (256-byte aligned), then V^T tiles [ceil(T / 32)][Hkv][d][32].
size_t qk_bytes(const mte_config &c, size_t T) {
  return ((T * (c.n_q_heads + c.n_kv_heads) * c.head_dim * 2) + 255) & ~(size_t)255;
}
size_t vt_bytes(const mte_config &c, size_t T) { return (T + 31) / 32 * 32 * c.n_kv_heads * c.head_dim * 2; }
// Bytes of the qkv region: fp32 rows [T, (Hq + 2 Hkv) d] (fp32 mode; also the
// bound used for the region in every mode), or the fp16 attention operands.
size_t qkv_bytes(const mte_config &c, size_t T) {
  const size_t rows = T * (c.n_q_heads + 2 * (size_t)c.n_kv_heads) * c.head_dim * 4;
  return c.dtype == MTE_F32 ? rows : std::max(rows, qk_bytes(c, T) + vt_bytes(c, T));
}

}  // namespace

// Workspace of mte_encode_static: a file-scope device array, one copy per
// GPU, never allocated or freed by the library. In host code `scratch` names
// a host-side stand-in, not device memory: its device address on each GPU
// comes from hipGetSymbolAddress (made with that GPU current) and only that
// address is handed to kernels.
__device__ __align__(256) unsigned char scratch[MTE_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `dev` (the current device), resolved once per
// device; nullptr if the runtime cannot provide it.
void *scratch_on(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch_ptr[dev] = p;
    else (void)hipGetLastError();   // clear the sticky error; the caller reports MTE_E_HIP
  }
  return g_scratch_ptr[dev];
}

}  // namespace

// The activations of one forward: fp32 residual stream h [T, D]; normalised
// GEMM input xn [T, D]; fp32 qkv [T, (Hq + 2 Hkv) d] (fp16 modes: the fp16
// q/k rows and V^T tiles the attention reads, in the same region); attention output
// [T, Hq d]; SwiGLU output [T, F]; partial sums of K-split projections (small
// batches: written by one GEMM, added up by the kernel that consumes its
// product); the rotary table of the batch [T, d/2] twice.
struct Work {
  float *h = nullptr;
  void *xn = nullptr;
  float *qkv = nullptr;
  f16 *qk = nullptr, *vt = nullptr;   // fp16 modes: the attention operands, inside the qkv region
  void *attn = nullptr;
  void *act = nullptr;
  float *ws = nullptr;
  size_t ws_elems = 0;
  float *rcos = nullptr, *rsin = nullptr;
};

struct mte_encoder {
  mte_config cfg;
  int device = 0;
  std::vector<LayerW> layers;
  void *wbuf = nullptr;      // all GEMM weights
  float *gbuf = nullptr;     // all norm gains (fp32)
  float *final_norm = nullptr;
  // Activations feeding the matrix cores are fp32 (MODE_F32) or fp16 (MODE_F16).
  int mode = MODE_F32;
  int gmode = MODE_F32;      // of the projection GEMMs: mode, or MODE_F8W for e4m3 weights
  int act_fmt = FMT_F32;
  Work w;                    // workspace for max_tokens, allocated at creation
  // Shared-prefix cache: per layer the prefix's packed q/k/v rows
  // [max_prefix, (Hq + 2 Hkv) d] (k and v are what later sequences read).
  char *pkv = nullptr;
  size_t pkv_stride = 0;     // bytes per layer
  int max_prefix = 0;
  RopeParams rope;
  // kernel timing
  int timing_class = -1;
  std::vector<hipEvent_t> ev;  // pairs: [2i] start, [2i+1] stop
  int ev_used = 0;
  int ev_cap = 0;
};

extern "C" {

const char *mte_status_string(int status) {
  switch (status) {
    case MTE_OK: return "ok";
    case MTE_E_INVALID: return "invalid argument";
    case MTE_E_CAPACITY: return "beyond the encoder's capacity";
    case MTE_E_HIP: return "HIP runtime error";
    case MTE_E_OOM: return "device out of memory";
    case MTE_E_UNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
  }
}

int mte_config_validate(const mte_config *c) {
  if (!c) return MTE_E_INVALID;
  if (c->n_layers < 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->ffn <= 0)
    return MTE_E_INVALID;
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f) || !std::isfinite(c->rms_eps) ||
      !std::isfinite(c->rope_theta))
    return MTE_E_INVALID;
  if (c->n_q_heads % c->n_kv_heads != 0) return MTE_E_INVALID;
  if (c->head_dim % 2 != 0) return MTE_E_INVALID;
  for (int i = 0; i < 3; ++i)
    if (c->mrope_section[i] < 0) return MTE_E_INVALID;
  if (c->mrope_section[0] + c->mrope_section[1] + c->mrope_section[2] != c->head_dim / 2)
    return MTE_E_INVALID;
  if (c->mrope_layout != MTE_MROPE_SECTIONS && c->mrope_layout != MTE_MROPE_INTERLEAVED)
    return MTE_E_INVALID;
  if (c->qk_norm != 0 && c->qk_norm != 1) return MTE_E_INVALID;
  if ((c->dtype != MTE_F32 && c->dtype != MTE_BF16) ||
      (c->out_dtype != MTE_F32 && c->out_dtype != MTE_BF16))
    return MTE_E_INVALID;
  if (c->max_tokens <= 0 || c->max_batch <= 0 || c->max_seq <= 0) return MTE_E_INVALID;
  if (c->weight_format != MTE_WEIGHTS_DTYPE && c->weight_format != MTE_WEIGHTS_E4M3) return MTE_E_INVALID;
  if (c->weight_format == MTE_WEIGHTS_E4M3 && c->dtype != MTE_BF16) return MTE_E_UNSUPPORTED;
  // Shapes the kernels are built for.
  if (c->head_dim != 64 && c->head_dim != 128) return MTE_E_UNSUPPORTED;
  const int rep = c->n_q_heads / c->n_kv_heads;
  if (!(rep == 1 || rep == 2 || rep % 4 == 0)) return MTE_E_UNSUPPORTED;
  if (c->hidden % 256 || c->ffn % 256 || (c->n_q_heads * c->head_dim) % 256 ||
      (c->n_kv_heads * c->head_dim) % 128)
    return MTE_E_UNSUPPORTED;
  if (c->max_tokens > kMaxTokens) return MTE_E_UNSUPPORTED;
  // the projection kernels address each operand with 32-bit byte offsets
  const int64_t es = c->dtype == MTE_F32 ? 4 : 2;
  const int64_t qd = (int64_t)c->n_q_heads * c->head_dim, qkv = qd + 2LL * c->n_kv_heads * c->head_dim;
  const int64_t kmax = std::max<int64_t>(std::max<int64_t>(c->hidden, c->ffn), qd);
  const int64_t nmax = std::max<int64_t>(std::max<int64_t>(2LL * c->ffn, qkv), c->hidden);
  if ((int64_t)c->max_tokens * kmax * es > 0xFFFFFFFFLL || nmax * kmax * es > 0xFFFFFFFFLL) return MTE_E_UNSUPPORTED;
  return MTE_OK;
}

int mte_check_batch(const mte_config *c, const int32_t *seq_lens, int32_t batch,
                    int32_t *total_tokens) {
  if (!c || !seq_lens || batch <= 0) return MTE_E_INVALID;
  int64_t tot = 0;
  bool over = batch > c->max_batch;
  for (int i = 0; i < batch; ++i) {
    if (seq_lens[i] <= 0) return MTE_E_INVALID;
    if (seq_lens[i] > c->max_seq) over = true;
    tot += seq_lens[i];
  }
  if (over || tot > c->max_tokens) return MTE_E_CAPACITY;
  if (total_tokens) *total_tokens = (int32_t)tot;
  return MTE_OK;
}

int mte_build_positions(const mte_seq_layout *layouts, int32_t batch, int32_t *pos_thw,
                        hipStream_t stream) {
  if (!layouts || !pos_thw || batch <= 0) return MTE_E_INVALID;
  int64_t T = 0;
  std::vector<int32_t> l5((size_t)batch * 5);
  for (int i = 0; i < batch; ++i) {
    const mte_seq_layout &s = layouts[i];
    if (s.n_text_before < 0 || s.n_text_after < 0 || s.grid_t < 0 || s.grid_h < 0 || s.grid_w < 0)
      return MTE_E_INVALID;
    const bool any = s.grid_t || s.grid_h || s.grid_w;
    const bool all = s.grid_t && s.grid_h && s.grid_w;
    if (any && !all) return MTE_E_INVALID;
    const int64_t nimg = (int64_t)s.grid_t * s.grid_h * s.grid_w;
    const int64_t len = (int64_t)s.n_text_before + nimg + s.n_text_after;
    if (len <= 0) return MTE_E_INVALID;
    T += len;
    if (T > kMaxTokens) return MTE_E_INVALID;
    int32_t *d = &l5[(size_t)i * 5];
    d[0] = s.n_text_before; d[1] = s.grid_t; d[2] = s.grid_h; d[3] = s.grid_w; d[4] = s.n_text_after;
  }
  return launch_positions(l5.data(), batch, pos_thw, (int)T, stream) == hipSuccess ? MTE_OK : MTE_E_HIP;
}

void mte_encoder_destroy(mte_encoder *e) {
  if (!e) return;
  int cur = 0;
  hipGetDevice(&cur);
  hipSetDevice(e->device);
  hipDeviceSynchronize();
  for (hipEvent_t ev : e->ev) hipEventDestroy(ev);
  hipFree(e->wbuf);
  hipFree(e->gbuf);
  hipFree(e->w.h);
  hipFree(e->w.xn);
  hipFree(e->w.qkv);
  hipFree(e->w.attn);
  hipFree(e->w.act);
  hipFree(e->w.ws);
  hipFree(e->w.rcos);
  hipFree(e->w.rsin);
  hipFree(e->pkv);
  hipSetDevice(cur);
  delete e;
}

int mte_encoder_create(const mte_config *cfg, const mte_weights *w, hipStream_t stream,
                       mte_encoder **out) {
  int st = mte_config_validate(cfg);
  if (st != MTE_OK) return st;
  if (!w || !out || (cfg->n_layers > 0 && !w->layers) || !w->final_norm) return MTE_E_INVALID;
  const mte_config &c = *cfg;
  for (int l = 0; l < c.n_layers; ++l) {
    const mte_layer_weights &L = w->layers[l];
    if (!L.attn_norm || !L.w_q || !L.w_k || !L.w_v || !L.w_o || !L.mlp_norm || !L.w_gate ||
        !L.w_up || !L.w_down)
      return MTE_E_INVALID;
    if (c.qk_norm && (!L.q_norm || !L.k_norm)) return MTE_E_INVALID;
  }
  mte_encoder *e = new (std::nothrow) mte_encoder();
  if (!e) return MTE_E_OOM;
  e->cfg = c;
  if (hipGetDevice(&e->device) != hipSuccess) { delete e; return MTE_E_HIP; }
  // set-up of mte_encode_static on this device (a failure here is reported by that call)
  scratch_on(e->device);

  const size_t es = esize(c.dtype);              // activations: fp16 or fp32
  const bool w8 = c.weight_format == MTE_WEIGHTS_E4M3;
  const size_t ws8 = w8 ? 1 : es;                // bytes per stored weight
  const size_t D = c.hidden, F = c.ffn, d = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads;
  const size_t nqkv = (Hq + 2 * Hkv) * d;
  const size_t b_qkv = nqkv * D * ws8, b_o = D * Hq * d * ws8, b_gu = 2 * F * D * ws8, b_d = D * F * ws8;
  // e4m3: the row scales of the four matrices follow their codes
  const size_t b_cs = w8 ? (nqkv + D + 2 * F + D) * sizeof(float) : 0;
  const size_t per_layer = b_qkv + b_o + b_gu + b_d + b_cs;
  const size_t g_per_layer = 2 * D + 2 * d;
  const size_t MT = c.max_tokens;

  auto fail = [&](int code) { mte_encoder_destroy(e); return code; };
  if (c.n_layers > 0 && hipMalloc(&e->wbuf, per_layer * c.n_layers) != hipSuccess) return fail(MTE_E_OOM);
  if (hipMalloc((void **)&e->gbuf, (g_per_layer * c.n_layers + D) * sizeof(float)) != hipSuccess)
    return fail(MTE_E_OOM);
  e->mode = c.dtype == MTE_BF16 ? MODE_F16 : MODE_F32;
  e->gmode = w8 ? MODE_F8W : e->mode;
  e->act_fmt = c.dtype == MTE_BF16 ? FMT_F16 : FMT_F32;
  Work &wk = e->w;
  if (hipMalloc((void **)&wk.h, MT * D * sizeof(float)) != hipSuccess ||
      hipMalloc(&wk.xn, MT * D * es) != hipSuccess ||
      hipMalloc((void **)&wk.qkv, qkv_bytes(c, MT)) != hipSuccess ||
      hipMalloc(&wk.attn, MT * Hq * d * es) != hipSuccess ||
      hipMalloc(&wk.act, MT * F * es) != hipSuccess)
    return fail(MTE_E_OOM);
  // K splits are planned for at most 8 splits of up to 256 rows, or 2 of up to 2048.
  wk.qk = (f16 *)wk.qkv;
  wk.vt = (f16 *)((char *)wk.qkv + qk_bytes(c, MT));
  wk.ws_elems = std::max(8 * std::min<size_t>(MT, 256), 2 * std::min<size_t>(MT, 2048)) *
                std::max(std::max(nqkv, 2 * F), D);
  if (hipMalloc((void **)&wk.ws, wk.ws_elems * sizeof(float)) != hipSuccess ||
      hipMalloc((void **)&wk.rcos, MT * (d / 2) * sizeof(float)) != hipSuccess ||
      hipMalloc((void **)&wk.rsin, MT * (d / 2) * sizeof(float)) != hipSuccess)
    return fail(MTE_E_OOM);

  const int sf = in_fmt(c.dtype);
  const bool f16 = c.dtype == MTE_BF16;
  e->layers.resize(c.n_layers);
  hipError_t he = hipSuccess;
  // Range analysis (bf16 weights only): per layer the max |w| of each
  // projection, the largest row norms of Wv, Wgate and Wup, and the largest
  // norm gains, from which the power-of-two pre-scales follow.
  enum { S_Q, S_K, S_V, S_O, S_G, S_U, S_D, S_AN, S_MN, S_QN, S_KN, S_N };
  std::vector<float> st_h;
  if (f16 && c.n_layers > 0) {
    float *st = nullptr;
    const size_t nst = (size_t)c.n_layers * S_N * 2;
    if (hipMalloc((void **)&st, nst * sizeof(float)) != hipSuccess) return fail(MTE_E_OOM);
    he = hipMemsetAsync(st, 0, nst * sizeof(float), stream);
    for (int l = 0; l < c.n_layers && he == hipSuccess; ++l) {
      const mte_layer_weights &L = w->layers[l];
      float *sl = st + (size_t)l * S_N * 2;
      const struct { const void *p; size_t rows, cols; } m[S_N] = {
          {L.w_q, Hq * d, D}, {L.w_k, Hkv * d, D}, {L.w_v, Hkv * d, D}, {L.w_o, D, Hq * d},
          {L.w_gate, F, D},   {L.w_up, F, D},      {L.w_down, D, F},    {L.attn_norm, 1, D},
          {L.mlp_norm, 1, D}, {L.q_norm, 1, d},    {L.k_norm, 1, d}};
      for (int k = 0; k < S_N && he == hipSuccess; ++k)
        if (m[k].p) he = launch_matrix_stats(sf, m[k].p, (int)m[k].rows, (int)m[k].cols, sl + 2 * k, stream);
    }
    st_h.resize(nst);
    if (he == hipSuccess) he = hipMemcpyAsync(st_h.data(), st, nst * sizeof(float), hipMemcpyDeviceToHost, stream);
    if (he == hipSuccess) he = hipStreamSynchronize(stream);
    hipFree(st);
    if (he != hipSuccess) return fail(MTE_E_HIP);
  }

  // Repack: fused [Wq; Wk; Wv], gate/up interleaved in blocks of 16 rows,
  // converted to the operand type with the weight pre-scales; fp32 norm
  // gains with the activation pre-scales folded in.
  const double sqrtD = std::sqrt((double)D);
  for (int l = 0; l < c.n_layers && he == hipSuccess; ++l) {
    const mte_layer_weights &L = w->layers[l];
    char *base = (char *)e->wbuf + per_layer * l;
    LayerW &o = e->layers[l];
    o.w_qkv = base;
    o.w_o = base + b_qkv;
    o.w_gu = base + b_qkv + b_o;
    o.w_d = base + b_qkv + b_o + b_gu;
    float *gb = e->gbuf + g_per_layer * l;
    o.attn_norm = gb;
    o.mlp_norm = gb + D;
    o.q_norm = gb + 2 * D;
    o.k_norm = gb + 2 * D + d;
    int w_qkv = 0, w_o = 0, w_gu = 0, w_d = 0, ka = 0, km = 0, ko = 0, ky = 0, kq = 0, kk = 0;
    if (f16) {
      const float *sl = &st_h[(size_t)l * S_N * 2];
      auto mx = [&](int k) { return (double)sl[2 * k]; };
      auto rn = [&](int k) { return (double)sl[2 * k + 1] * 1.001; };   // fp32 norm rounding margin
      w_qkv = weight_shift(std::max(mx(S_Q), std::max(mx(S_K), mx(S_V))));
      w_o = weight_shift(mx(S_O));
      w_gu = weight_shift(std::max(mx(S_G), mx(S_U)));
      w_d = weight_shift(mx(S_D));
      // |RMSNorm(x) * g|_2 <= sqrt(D) max|g|, so every element of the norm
      // output, of v (hence of the attention output, a convex combination
      // of v rows) and of gate / up is bounded by that times the row norm
      // of its weight; |silu(z)| <= |z|.
      const double ba = sqrtD * mx(S_AN), bm = sqrtD * mx(S_MN);
      // e4m3 codes are within 2^-4 relative of their weight (plus a
      // subnormal step 2^-10 of the row scale, far below 2^-4 of the row
      // norm): the row norms of the dequantised weights grow by at most 1/8.
      const double q8 = w8 ? 1.125 : 1.0;
      ka = act_shift(ba);
      km = act_shift(bm);
      ko = act_shift(ba * rn(S_V) * q8);
      ky = act_shift((bm * rn(S_G) * q8) * (bm * rn(S_U) * q8));
      // fp16 q and k of the attention: with QK-norm every element of a head
      // is at most its norm, sqrt(d) max|g_q| (resp. g_k), and the rotation
      // keeps each pair's norm; without it, the row norms of Wq / Wk times the
      // norm output's bound, times sqrt(2) for the rotation.
      const double sd = std::sqrt((double)d);
      kq = act_shift(c.qk_norm ? sd * mx(S_QN) : std::sqrt(2.0) * ba * rn(S_Q) * q8);
      kk = act_shift(c.qk_norm ? sd * mx(S_KN) : std::sqrt(2.0) * ba * rn(S_K) * q8);
      if (w8) w_qkv = w_o = w_gu = w_d = 0;    // codes are not pre-scaled; the row scales apply
    }
    o.s_qkv = std::ldexp(1.f, ka - w_qkv);
    o.s_o = std::ldexp(1.f, ko - w_o);
    o.s_gu = std::ldexp(1.f, km - w_gu);
    o.s_d = std::ldexp(1.f, ky - w_d);
    o.o_pre = std::ldexp(1.f, -ko);
    o.y_pre = std::ldexp(1.f, -ky);
    o.q_pre = std::ldexp(1.f, -kq);
    o.k_pre = std::ldexp(1.f, -kk);
    o.att_sc = (float)(1.4426950408889634 / std::sqrt((double)d) * std::ldexp(1.0, kq + kk));
    const int df = f16 ? FMT_F16 : FMT_F32;
    const size_t bq = Hq * d * D * es, bk = Hkv * d * D * es;
    const float sq = std::ldexp(1.f, w_qkv);
    if (w8) {
      float *cs = (float *)(base + b_qkv + b_o + b_gu + b_d);
      o.cs_qkv = cs;
      o.cs_o = cs + nqkv;
      o.cs_gu = cs + nqkv + D;
      o.cs_d = cs + nqkv + D + 2 * F;
      uint8_t *q = (uint8_t *)o.w_qkv;
      float *qs = (float *)o.cs_qkv;
      he = launch_quantize_e4m3_rows(sf, L.w_q, (int)(Hq * d), (int)D, q, qs, 0, 0, stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_k, (int)(Hkv * d), (int)D, q + Hq * d * D, qs + Hq * d, 0, 0,
                                       stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_v, (int)(Hkv * d), (int)D, q + (Hq + Hkv) * d * D,
                                       qs + (Hq + Hkv) * d, 0, 0, stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_o, (int)D, (int)(Hq * d), (uint8_t *)o.w_o, (float *)o.cs_o, 0,
                                       0, stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_gate, (int)F, (int)D, (uint8_t *)o.w_gu, (float *)o.cs_gu, 1,
                                       0, stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_up, (int)F, (int)D, (uint8_t *)o.w_gu, (float *)o.cs_gu, 1, 1,
                                       stream);
      if (he == hipSuccess)
        he = launch_quantize_e4m3_rows(sf, L.w_down, (int)D, (int)F, (uint8_t *)o.w_d, (float *)o.cs_d, 0, 0,
                                       stream);
    } else {
      he = launch_convert_rows(sf, L.w_q, df, o.w_qkv, (int)(Hq * d), (int)D, sq, 0, 0, stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_k, df, (char *)o.w_qkv + bq, (int)(Hkv * d), (int)D, sq, 0, 0, stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_v, df, (char *)o.w_qkv + bq + bk, (int)(Hkv * d), (int)D, sq, 0, 0,
                                 stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_o, df, o.w_o, (int)D, (int)(Hq * d), std::ldexp(1.f, w_o), 0, 0, stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_gate, df, o.w_gu, (int)F, (int)D, std::ldexp(1.f, w_gu), 1, 0, stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_up, df, o.w_gu, (int)F, (int)D, std::ldexp(1.f, w_gu), 1, 1, stream);
      if (he == hipSuccess)
        he = launch_convert_rows(sf, L.w_down, df, o.w_d, (int)D, (int)F, std::ldexp(1.f, w_d), 0, 0, stream);
    }
    if (he == hipSuccess) he = launch_to_f32(sf, L.attn_norm, o.attn_norm, (int)D, std::ldexp(1.f, -ka), stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.mlp_norm, o.mlp_norm, (int)D, std::ldexp(1.f, -km), stream);
    if (he == hipSuccess && c.qk_norm) he = launch_to_f32(sf, L.q_norm, o.q_norm, (int)d, 1.f, stream);
    if (he == hipSuccess && c.qk_norm) he = launch_to_f32(sf, L.k_norm, o.k_norm, (int)d, 1.f, stream);
  }
  e->final_norm = e->gbuf + g_per_layer * c.n_layers;
  if (he == hipSuccess) he = launch_to_f32(sf, w->final_norm, e->final_norm, (int)D, 1.f, stream);
  if (he == hipSuccess) he = hipStreamSynchronize(stream);
  if (he != hipSuccess) return fail(MTE_E_HIP);

  // Rotary tables: inverse frequencies in float64, pair -> axis.
  const int half = c.head_dim / 2;
  for (int j = 0; j < 64; ++j) {
    e->rope.inv_freq[j] = j < half ? std::pow((double)c.rope_theta, -2.0 * j / c.head_dim) : 0.0;
    int ax = 0;
    if (j < half) {
      if (c.mrope_layout == MTE_MROPE_SECTIONS) {
        ax = j < c.mrope_section[0] ? 0 : (j < c.mrope_section[0] + c.mrope_section[1] ? 1 : 2);
      } else {
        if (j % 3 == 1 && j < 3 * c.mrope_section[1]) ax = 1;
        else if (j % 3 == 2 && j < 3 * c.mrope_section[2]) ax = 2;
      }
    }
    e->rope.axis[j] = (uint8_t)ax;
  }
  *out = e;
  return MTE_OK;
}

}  // extern "C"

namespace {

struct Timer {
  mte_encoder *e;
  hipStream_t s;
  bool on;
  Timer(mte_encoder *e_, int cls, hipStream_t s_) : e(e_), s(s_) {
    on = e->timing_class == cls && e->ev_used < e->ev_cap;
    if (on) hipEventRecord(e->ev[2 * e->ev_used], s);
  }
  ~Timer() {
    if (on) {
      hipEventRecord(e->ev[2 * e->ev_used + 1], s);
      e->ev_used++;
    }
  }
};

// Shared-prefix mode of run_layers: `record` copies every layer's packed
// q/k/v rows (the prefix itself being encoded) into the cache; otherwise
// attention reads the cache's first P rows as keys / values before each
// sequence's own.
struct PrefixCtx {
  char *cache;       // [n_layers][layer stride]: one layer's q/k/v of the prefix
  size_t stride;     // bytes per layer
  int P;
  bool record;
};

// Runs layers [l0, l1) on the fp32 residual stream `h` (T rows).
hipError_t run_layers(mte_encoder *e, const Work &wk, float *h, const int32_t *cu, int batch, int T, int l0,
                      int l1, bool first_norm_done, int *pending, hipStream_t s,
                      const PrefixCtx *pre = nullptr) {
  const mte_config &c = e->cfg;
  const int D = c.hidden, d = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
  const int nqkv = (Hq + 2 * Hkv) * d;
  const int mode = e->mode, gm = e->gmode, af = e->act_fmt;
  float *ws = wk.ws;
  const size_t wn = wk.ws_elems;
  // `*pending` counts the partial sums of a K-split residual projection
  // still in ws, to be added into h by the next RMSNorm.
  int np = *pending;
  hipError_t err = hipSuccess;
#define MTE_TRY(x) do { err = (x); if (err != hipSuccess) return err; } while (0)
  for (int l = l0; l < l1; ++l) {
    const LayerW &W = e->layers[l];
    if (!(l == l0 && first_norm_done))
      MTE_TRY(launch_rmsnorm(FMT_F32, af, h, np ? h : nullptr, np ? ws : nullptr, np, W.attn_norm, wk.xn, T,
                             D, c.rms_eps, s));
    int sp = 0;
    QkvEpi qe{wk.rcos, wk.rsin, c.qk_norm ? W.q_norm : nullptr, c.qk_norm ? W.k_norm : nullptr,
              (Hq + Hkv) * d, Hq * d, d, c.rms_eps};
    const bool half = mode != MODE_F32;   // fp16 attention operands
    if (half) {
      qe.qk = wk.qk;
      qe.vt = wk.vt;
      qe.q_pre = W.q_pre;
      qe.k_pre = W.k_pre;
      qe.v_pre = W.o_pre;
      qe.hkv = Hkv;
    }
    {
      Timer t(e, 0, s);
      MTE_TRY(launch_gemm(gm, EPI_QKV, wk.xn, W.w_qkv, wk.qkv, T, nqkv, D, nqkv, W.s_qkv, 1.f, ws, wn,
                          &sp, &qe, s, W.cs_qkv));
    }
    if (sp) MTE_TRY(launch_qkv_parts(wk.qkv, ws, sp, T, Hq, Hkv, qe, s));
    {
      Timer t(e, 1, s);
      // the prefix cache of layer l: fp32 rows [max_prefix, nqkv], or the fp16
      // q/k rows [max_prefix, (Hq + Hkv) d] followed by V^T tiles
      char *lc = pre ? pre->cache + l * pre->stride : nullptr;
      const size_t cq = qk_bytes(c, e->max_prefix);
      if (pre && pre->record) {
        if (half) {
          MTE_TRY(hipMemcpyAsync(lc, wk.qk, (size_t)T * (Hq + Hkv) * d * sizeof(f16), hipMemcpyDeviceToDevice, s));
          MTE_TRY(hipMemcpyAsync(lc + cq, wk.vt, vt_bytes(c, T), hipMemcpyDeviceToDevice, s));
        } else {
          MTE_TRY(hipMemcpyAsync(lc, wk.qkv, (size_t)T * nqkv * sizeof(float), hipMemcpyDeviceToDevice, s));
        }
      }
      const bool use = pre && !pre->record;
      if (half)
        MTE_TRY(launch_attention_h(wk.qk, wk.vt, use ? (const f16 *)lc : nullptr,
                                   use ? (const f16 *)(lc + cq) : nullptr, use ? pre->P : 0, (f16 *)wk.attn,
                                   W.att_sc, cu, batch, T, Hq, Hkv, d, 1, s));
      else
        MTE_TRY(launch_attention(wk.qkv, use ? (const float *)lc : nullptr, use ? pre->P : 0, (float *)wk.attn,
                                 cu, batch, Hq, Hkv, d, s));
    }
    {
      Timer t(e, 2, s);
      MTE_TRY(launch_gemm(gm, EPI_RESID, wk.attn, W.w_o, h, T, D, Hq * d, D, W.s_o, 1.f, ws, wn, &np,
                          nullptr, s, W.cs_o));
    }
    MTE_TRY(launch_rmsnorm(FMT_F32, af, h, np ? h : nullptr, np ? ws : nullptr, np, W.mlp_norm, wk.xn, T, D,
                           c.rms_eps, s));
    {
      Timer t(e, 3, s);
      MTE_TRY(launch_gemm(gm, EPI_SWIGLU, wk.xn, W.w_gu, wk.act, T, 2 * F, D, F, W.s_gu, W.y_pre, ws, wn,
                          &sp, nullptr, s, W.cs_gu));
    }
    if (sp) MTE_TRY(launch_swiglu_parts(af, ws, sp, T, F, wk.act, W.y_pre, s));
    {
      Timer t(e, 4, s);
      MTE_TRY(launch_gemm(gm, EPI_RESID, wk.act, W.w_d, h, T, D, F, D, W.s_d, 1.f, ws, wn, &np, nullptr, s,
                          W.cs_d));
    }
  }
#undef MTE_TRY
  *pending = np;
  return err;
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) hipSetDevice(dev);
    else prev = -1;
  }
  ~DeviceGuard() {
    if (prev >= 0) hipSetDevice(prev);
  }
};

}  // namespace

extern "C" {

}  // extern "C"

namespace {

// The whole forward of mte_encode on workspace `wk`, after the host checks;
// cu: host [batch + 1] sequence offsets.
hipError_t encode_on(mte_encoder *e, const Work &wk, const void *embeds, const int32_t *pos_thw,
                     const int32_t *cu, int32_t batch, int32_t T, void *out_hidden, hipStream_t stream) {
  const mte_config &c = e->cfg;
  const int out_fmt = in_fmt(c.out_dtype);
  if (c.n_layers == 0)
    return launch_rmsnorm(in_fmt(c.dtype), out_fmt, embeds, nullptr, nullptr, 0, e->final_norm, out_hidden, T,
                          c.hidden, c.rms_eps, stream);
  hipError_t err = launch_rope_table(pos_thw, T, c.head_dim / 2, e->rope, wk.rcos, wk.rsin, stream);
  // Layer 0's attention norm also seeds the fp32 residual stream from the embeddings.
  if (err == hipSuccess)
    err = launch_rmsnorm(in_fmt(c.dtype), e->act_fmt, embeds, wk.h, nullptr, 0, e->layers[0].attn_norm, wk.xn,
                         T, c.hidden, c.rms_eps, stream);
  int np = 0;
  if (err == hipSuccess) err = run_layers(e, wk, wk.h, cu, batch, T, 0, c.n_layers, true, &np, stream);
  if (err == hipSuccess)
    err = launch_rmsnorm(FMT_F32, out_fmt, wk.h, nullptr, np ? wk.ws : nullptr, np, e->final_norm, out_hidden, T,
                         c.hidden, c.rms_eps, stream);
  return err;
}

// Host checks shared by mte_encode and its variants: pointers, the batch
// against the configuration, embeds / out_hidden disjoint.
int check_encode(const mte_encoder *e, const void *embeds, const int32_t *pos_thw, const int32_t *seq_lens,
                 int32_t batch, const void *out_hidden, int32_t *T) {
  if (!e || !embeds || !pos_thw || !out_hidden) return MTE_E_INVALID;
  int st = mte_check_batch(&e->cfg, seq_lens, batch, T);
  if (st != MTE_OK) return st;
  const mte_config &c = e->cfg;
  const size_t in_bytes = (size_t)*T * c.hidden * esize(c.dtype);
  const size_t out_bytes = (size_t)*T * c.hidden * esize(c.out_dtype);
  const char *ib = (const char *)embeds, *ob = (const char *)out_hidden;
  if (ib < ob + out_bytes && ob < ib + in_bytes) return MTE_E_INVALID;
  return MTE_OK;
}

}  // namespace

extern "C" {

int mte_encode(mte_encoder *e, const void *embeds, const int32_t *pos_thw, const int32_t *seq_lens,
               int32_t batch, void *out_hidden, hipStream_t stream) {
  int32_t T = 0;
  const int st = check_encode(e, embeds, pos_thw, seq_lens, batch, out_hidden, &T);
  if (st != MTE_OK) return st;
  std::vector<int32_t> cu(batch + 1, 0);
  for (int i = 0; i < batch; ++i) cu[i + 1] = cu[i] + seq_lens[i];
  DeviceGuard g(e->device);
  return encode_on(e, e->w, embeds, pos_thw, cu.data(), batch, T, out_hidden, stream) == hipSuccess ? MTE_OK
                                                                                                  : MTE_E_HIP;
}

int mte_encode_static(mte_encoder *e, const void *embeds, const int32_t *pos_thw, const int32_t *seq_lens,
                      int32_t batch, void *out_hidden, hipStream_t stream) {
  int32_t T = 0;
  const int st = check_encode(e, embeds, pos_thw, seq_lens, batch, out_hidden, &T);
  if (st != MTE_OK) return st;
  if (batch > MTE_STATIC_MAX_BATCH) return MTE_E_CAPACITY;
  const mte_config &c = e->cfg;
  const size_t es = esize(c.dtype), D = c.hidden, F = c.ffn, d = c.head_dim, Hq = c.n_q_heads;
  const size_t nqkv = (Hq + 2 * (size_t)c.n_kv_heads) * d;
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  // the activations of T tokens, each region 256-byte aligned; the rest holds K-split partials
  const size_t sizes[7] = {T * D * 4, T * D * es, qkv_bytes(c, T), T * Hq * d * es, T * F * es,
                           T * (d / 2) * 4, T * (d / 2) * 4};
  size_t used = 0;
  for (size_t b : sizes) used += up(b);
  if (used > (size_t)MTE_STATIC_SCRATCH_BYTES) return MTE_E_CAPACITY;
  int32_t cu[MTE_STATIC_MAX_BATCH + 1];
  cu[0] = 0;
  for (int i = 0; i < batch; ++i) cu[i + 1] = cu[i] + seq_lens[i];
  DeviceGuard g(e->device);
  unsigned char *base = (unsigned char *)scratch_on(e->device);
  if (!base) return MTE_E_HIP;
  unsigned char *ptr[7];
  size_t off = 0;
  for (int i = 0; i < 7; ++i) {
    ptr[i] = base + off;
    off += up(sizes[i]);
  }
  Work wk;
  wk.h = (float *)ptr[0];
  wk.xn = ptr[1];
  wk.qkv = (float *)ptr[2];
  wk.qk = (f16 *)ptr[2];
  wk.vt = (f16 *)(ptr[2] + qk_bytes(c, T));
  wk.attn = ptr[3];
  wk.act = ptr[4];
  wk.rcos = (float *)ptr[5];
  wk.rsin = (float *)ptr[6];
  // the encoder's own bound as well, so that a batch gets the same launch plan
  // (hence bit-identical results) as through mte_encode whenever its partial
  // sums fit here
  wk.ws = (float *)(base + off);
  wk.ws_elems = std::min(((size_t)MTE_STATIC_SCRATCH_BYTES - off) / sizeof(float), e->w.ws_elems);
  return encode_on(e, wk, embeds, pos_thw, cu, batch, T, out_hidden, stream) == hipSuccess ? MTE_OK : MTE_E_HIP;
}

int mte_encode_layers(mte_encoder *e, const float *h_in, const int32_t *pos_thw,
                      const int32_t *seq_lens, int32_t batch, int32_t layer_begin, int32_t layer_end,
                      float *h_out, hipStream_t stream) {
  if (!e || !h_in || !pos_thw || !h_out) return MTE_E_INVALID;
  int32_t T = 0;
  int st = mte_check_batch(&e->cfg, seq_lens, batch, &T);
  if (st != MTE_OK) return st;
  if (layer_begin < 0 || layer_end < layer_begin || layer_end > e->cfg.n_layers) return MTE_E_INVALID;
  const size_t bytes = (size_t)T * e->cfg.hidden * sizeof(float);
  const char *ib = (const char *)h_in, *ob = (const char *)h_out;
  if (ib != ob && ib < ob + bytes && ob < ib + bytes) return MTE_E_INVALID;
  std::vector<int32_t> cu(batch + 1, 0);
  for (int i = 0; i < batch; ++i) cu[i + 1] = cu[i] + seq_lens[i];
  DeviceGuard g(e->device);
  hipError_t err = hipSuccess;
  if (h_out != h_in) err = hipMemcpyAsync(h_out, h_in, bytes, hipMemcpyDeviceToDevice, stream);
  if (err == hipSuccess)
    err = launch_rope_table(pos_thw, T, e->cfg.head_dim / 2, e->rope, e->w.rcos, e->w.rsin, stream);
  int np = 0;
  if (err == hipSuccess)
    err = run_layers(e, e->w, h_out, cu.data(), batch, T, layer_begin, layer_end, false, &np, stream);
  if (err == hipSuccess && np) err = launch_resid_add(h_out, e->w.ws, np, T, e->cfg.hidden, stream);
  return err == hipSuccess ? MTE_OK : MTE_E_HIP;
}

int mte_encoder_reserve_prefix(mte_encoder *e, int32_t max_prefix) {
  if (!e || max_prefix <= 0 || max_prefix > e->cfg.max_tokens || max_prefix > e->cfg.max_seq)
    return MTE_E_INVALID;
  if (e->cfg.n_layers == 0) return MTE_E_UNSUPPORTED;
  DeviceGuard g(e->device);
  const mte_config &c = e->cfg;
  const size_t nqkv = (size_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  if (hipDeviceSynchronize() != hipSuccess) return MTE_E_HIP;
  hipFree(e->pkv);
  e->pkv = nullptr;
  e->max_prefix = 0;
  const size_t stride = c.dtype == MTE_F32 ? (size_t)max_prefix * nqkv * sizeof(float)
                                           : qk_bytes(c, max_prefix) + vt_bytes(c, max_prefix);
  if (hipMalloc((void **)&e->pkv, (size_t)c.n_layers * stride) != hipSuccess) return MTE_E_OOM;
  e->pkv_stride = stride;
  e->max_prefix = max_prefix;
  return MTE_OK;
}

int mte_encode_prefixed(mte_encoder *e, const void *prefix_embeds, const int32_t *prefix_pos,
                        int32_t prefix_len, const void *embeds, const int32_t *pos_thw,
                        const int32_t *seq_lens, int32_t batch, void *out_prefix, void *out_hidden,
                        hipStream_t stream) {
  if (!e || !prefix_embeds || !prefix_pos || !embeds || !pos_thw || !out_prefix || !out_hidden)
    return MTE_E_INVALID;
  const mte_config &c = e->cfg;
  if (c.n_layers == 0 || !e->pkv) return MTE_E_INVALID;     // mte_encoder_reserve_prefix first
  if (prefix_len <= 0) return MTE_E_INVALID;
  if (prefix_len > e->max_prefix) return MTE_E_CAPACITY;
  int32_t T = 0;
  int st = mte_check_batch(&c, seq_lens, batch, &T);
  if (st != MTE_OK) return st;
  for (int i = 0; i < batch; ++i)
    if ((int64_t)prefix_len + seq_lens[i] > c.max_seq) return MTE_E_CAPACITY;
  const size_t in_b = (size_t)T * c.hidden * esize(c.dtype), out_b = (size_t)T * c.hidden * esize(c.out_dtype);
  const size_t pin_b = (size_t)prefix_len * c.hidden * esize(c.dtype);
  const size_t pout_b = (size_t)prefix_len * c.hidden * esize(c.out_dtype);
  auto overlap = [](const void *a, size_t na, const void *b, size_t nb) {
    const char *x = (const char *)a, *y = (const char *)b;
    return x < y + nb && y < x + na;
  };
  if (overlap(embeds, in_b, out_hidden, out_b) || overlap(prefix_embeds, pin_b, out_hidden, out_b) ||
      overlap(embeds, in_b, out_prefix, pout_b) || overlap(prefix_embeds, pin_b, out_prefix, pout_b) ||
      overlap(out_prefix, pout_b, out_hidden, out_b))
    return MTE_E_INVALID;
  DeviceGuard g(e->device);
  const int out_fmt = in_fmt(c.out_dtype);
  hipError_t err = hipSuccess;
  // 1. The prefix, once: one sequence of prefix_len tokens, recording every
  //    layer's q/k/v rows.
  {
    std::vector<int32_t> cu{0, prefix_len};
    const PrefixCtx rec{e->pkv, e->pkv_stride, prefix_len, true};
    err = launch_rope_table(prefix_pos, prefix_len, c.head_dim / 2, e->rope, e->w.rcos, e->w.rsin, stream);
    if (err == hipSuccess)
      err = launch_rmsnorm(in_fmt(c.dtype), e->act_fmt, prefix_embeds, e->w.h, nullptr, 0, e->layers[0].attn_norm,
                           e->w.xn, prefix_len, c.hidden, c.rms_eps, stream);
    int np = 0;
    if (err == hipSuccess)
      err = run_layers(e, e->w, e->w.h, cu.data(), 1, prefix_len, 0, c.n_layers, true, &np, stream, &rec);
    if (err == hipSuccess)
      err = launch_rmsnorm(FMT_F32, out_fmt, e->w.h, nullptr, np ? e->w.ws : nullptr, np, e->final_norm, out_prefix,
                           prefix_len, c.hidden, c.rms_eps, stream);
  }
  // 2. The sequences' own tokens, attending to the cached prefix first.
  if (err == hipSuccess) {
    std::vector<int32_t> cu(batch + 1, 0);
    for (int i = 0; i < batch; ++i) cu[i + 1] = cu[i] + seq_lens[i];
    const PrefixCtx use{e->pkv, e->pkv_stride, prefix_len, false};
    err = launch_rope_table(pos_thw, T, c.head_dim / 2, e->rope, e->w.rcos, e->w.rsin, stream);
    if (err == hipSuccess)
      err = launch_rmsnorm(in_fmt(c.dtype), e->act_fmt, embeds, e->w.h, nullptr, 0, e->layers[0].attn_norm, e->w.xn,
                           T, c.hidden, c.rms_eps, stream);
    int np = 0;
    if (err == hipSuccess)
      err = run_layers(e, e->w, e->w.h, cu.data(), batch, T, 0, c.n_layers, true, &np, stream, &use);
    if (err == hipSuccess)
      err = launch_rmsnorm(FMT_F32, out_fmt, e->w.h, nullptr, np ? e->w.ws : nullptr, np, e->final_norm, out_hidden,
                           T, c.hidden, c.rms_eps, stream);
  }
  return err == hipSuccess ? MTE_OK : MTE_E_HIP;
}

int mte_timing_enable(mte_encoder *e, int32_t kernel_class, int32_t capacity) {
  if (!e || kernel_class < 0 || kernel_class >= kNumClasses || capacity <= 0) return MTE_E_INVALID;
  DeviceGuard g(e->device);
  while ((int)e->ev.size() < 2 * capacity) {
    hipEvent_t ev;
    if (hipEventCreate(&ev) != hipSuccess) return MTE_E_HIP;
    e->ev.push_back(ev);
  }
  e->ev_cap = capacity;
  e->ev_used = 0;
  e->timing_class = kernel_class;
  return MTE_OK;
}

int mte_timing_read(mte_encoder *e, int32_t *launches, double *total_ms) {
  if (!e || !launches || !total_ms) return MTE_E_INVALID;
  DeviceGuard g(e->device);
  double tot = 0.0;
  for (int i = 0; i < e->ev_used; ++i) {
    if (hipEventSynchronize(e->ev[2 * i + 1]) != hipSuccess) return MTE_E_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e->ev[2 * i], e->ev[2 * i + 1]) != hipSuccess) return MTE_E_HIP;
    tot += ms;
  }
  *launches = e->ev_used;
  *total_ms = tot;
  e->ev_used = 0;
  return MTE_OK;
}

int mte_quantize_e4m3_rows(const void *src, int32_t src_dtype, int32_t rows, int32_t cols, uint8_t *codes,
                           float *scales, hipStream_t stream) {
  if (!src || !codes || !scales || rows <= 0 || cols <= 0) return MTE_E_INVALID;
  if (src_dtype != MTE_F32 && src_dtype != MTE_BF16) return MTE_E_INVALID;
  return launch_quantize_e4m3_rows(in_fmt(src_dtype), src, rows, cols, codes, scales, 0, 0, stream) ==
                 hipSuccess
             ? MTE_OK
             : MTE_E_HIP;
}

int mte_timing_disable(mte_encoder *e) {
  if (!e) return MTE_E_INVALID;
  e->timing_class = -1;
  e->ev_used = 0;
  return MTE_OK;
}

}  // extern "C"
