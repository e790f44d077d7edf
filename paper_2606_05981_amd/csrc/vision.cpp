// C ABI of the vision tower (include/mte_vision.h): validation, weight
// repacking with the fp16 range analysis at creation, and the per-call
// launch schedule. Every step runs in the library's kernels: patch
// extraction, LayerNorm, the tiled GEMM (bias added in its epilogue; QKV with
// the 2-D rotary epilogue; GELU epilogue), bidirectional attention.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <new>
#include <vector>

#include "../../include/mte_vision.h"
#include "launch.h"

using namespace mte;

namespace {

int v_exp2_of(double x) {
  if (!(x > 0.0)) return 0;
  int e = 0;
  std::frexp(x, &e);
  return e;
}
// largest weight magnitude in [2^14, 2^15) after scaling (exact for bf16 values)
int v_weight_shift(double maxabs) { return maxabs > 0.0 ? 15 - v_exp2_of(maxabs) : 0; }
// activation pre-scale exponent keeping values bounded by `bound` within 2^15
int v_act_shift(double bound) { return std::max(0, v_exp2_of(bound) - 15); }

struct VLayer {
  void *w_qkv, *w_o, *w_fc1, *w_fc2;
  float *ln1_g, *ln1_b, *ln2_g, *ln2_b, *b_qkv, *b_o, *b_fc1, *b_fc2;
  float s_qkv = 1.f, s_o = 1.f, s_fc1 = 1.f, s_fc2 = 1.f, o_pre = 1.f, y_pre = 1.f;
  // fp16 attention operands (bf16 storage): q and k times q_pre / k_pre,
  // att_sc = log2(e) / sqrt(d) / (q_pre k_pre)
  float q_pre = 1.f, k_pre = 1.f, att_sc = 1.f;
};

size_t v_esize(int dtype) { return dtype == MTE_BF16 ? 2 : 4; }
int v_in_fmt(int dtype) { return dtype == MTE_BF16 ? FMT_BF16 : FMT_F32; }

}  // namespace

struct mte_vision {
  mte_vision_config cfg;
  int device = 0;
  int mode = MODE_F32, act_fmt = FMT_F32;
  std::vector<VLayer> layers;
  void *wbuf = nullptr;     // GEMM weights (operand type)
  float *fbuf = nullptr;    // gains and biases (fp32, pre-scales folded into the gains)
  void *w_patch = nullptr, *w_m1 = nullptr, *w_m2 = nullptr;
  float *b_patch = nullptr, *mln_g = nullptr, *mln_b = nullptr, *b_m1 = nullptr, *b_m2 = nullptr;
  float s_patch = 1.f, s_m1 = 1.f, s_m2 = 1.f, m_pre = 1.f;
  // workspace, for max_images * (max_side / patch)^2 patches
  void *patches = nullptr;  // [T, C p p] operand type
  float *h = nullptr;       // [T, D] residual stream
  void *xn = nullptr;       // [T, D] LayerNorm output (viewed [T/mm, mm D] for the merger)
  float *qkv = nullptr;     // [T, 3D] fp32 (fp32 storage), or fp16 q/k rows [T, 2D] then V^T tiles
  void *attn = nullptr;     // [T, D]
  void *act = nullptr;      // [T, F]
  void *mact = nullptr;     // [T/mm, mm D]
  float *mout = nullptr;    // [T/mm, out_hidden] (bf16 output only)
  int32_t *pos = nullptr;   // [3, T]
  float *rcos = nullptr, *rsin = nullptr;
  RopeParams rope;
};

extern "C" {

int mte_vision_config_validate(const mte_vision_config *c) {
  if (!c) return MTE_E_INVALID;
  if (c->depth < 0 || c->hidden <= 0 || c->n_heads <= 0 || c->head_dim <= 0 || c->ffn <= 0 || c->patch <= 0 ||
      c->merge <= 0 || c->in_channels <= 0 || c->out_hidden <= 0 || c->max_images <= 0 || c->max_side <= 0)
    return MTE_E_INVALID;
  if (c->hidden != c->n_heads * c->head_dim) return MTE_E_INVALID;
  if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps) || !(c->rope_theta > 0.f) || !std::isfinite(c->rope_theta))
    return MTE_E_INVALID;
  if ((c->dtype != MTE_F32 && c->dtype != MTE_BF16) || (c->out_dtype != MTE_F32 && c->out_dtype != MTE_BF16))
    return MTE_E_INVALID;
  if (c->head_dim != 64 && c->head_dim != 128) return MTE_E_UNSUPPORTED;
  const int64_t kp = (int64_t)c->in_channels * c->patch * c->patch;
  if (c->hidden % 64 || c->ffn % 64 || c->out_hidden % 64 || kp % 64 || c->hidden > 4096)
    return MTE_E_UNSUPPORTED;
  const int64_t side = (int64_t)c->patch * c->merge;
  if (c->max_side < side) return MTE_E_INVALID;
  const int64_t per = ((int64_t)c->max_side / c->patch) * ((int64_t)c->max_side / c->patch);
  if ((int64_t)c->max_images * per > (1 << 24)) return MTE_E_UNSUPPORTED;
  // the projection kernels address each operand with 32-bit byte offsets
  const int64_t es = c->dtype == MTE_F32 ? 4 : 2, mm = (int64_t)c->merge * c->merge;
  const int64_t kmax = std::max<int64_t>(std::max<int64_t>(kp, c->hidden), std::max<int64_t>(c->ffn, mm * c->hidden));
  const int64_t nmax = std::max<int64_t>(std::max<int64_t>(3LL * c->hidden, c->ffn), std::max<int64_t>(mm * c->hidden, c->out_hidden));
  if ((int64_t)c->max_images * per * kmax * es > 0xFFFFFFFFLL || nmax * kmax * es > 0xFFFFFFFFLL)
    return MTE_E_UNSUPPORTED;
  return MTE_OK;
}

void mte_vision_destroy(mte_vision *e) {
  if (!e) return;
  int cur = 0;
  hipGetDevice(&cur);
  hipSetDevice(e->device);
  hipDeviceSynchronize();
  for (void *p : {e->wbuf, (void *)e->fbuf, e->patches, (void *)e->h, e->xn, (void *)e->qkv, e->attn, e->act, e->mact,
                  (void *)e->mout, (void *)e->pos, (void *)e->rcos, (void *)e->rsin})
    hipFree(p);
  hipSetDevice(cur);
  delete e;
}

int mte_vision_create(const mte_vision_config *cfg, const mte_vision_weights *w, hipStream_t stream,
                      mte_vision **out) {
  int st = mte_vision_config_validate(cfg);
  if (st != MTE_OK) return st;
  if (!w || !out || !w->patch_w || !w->patch_b || (cfg->depth > 0 && !w->layers) || !w->merge_ln_g ||
      !w->merge_ln_b || !w->merge_w1 || !w->merge_b1 || !w->merge_w2 || !w->merge_b2)
    return MTE_E_INVALID;
  const mte_vision_config &c = *cfg;
  for (int l = 0; l < c.depth; ++l) {
    const mte_vision_layer_weights &L = w->layers[l];
    for (const void *p : {L.ln1_g, L.ln1_b, L.w_qkv, L.b_qkv, L.w_o, L.b_o, L.ln2_g, L.ln2_b, L.w_fc1, L.b_fc1,
                          L.w_fc2, L.b_fc2})
      if (!p) return MTE_E_INVALID;
  }
  mte_vision *e = new (std::nothrow) mte_vision();
  if (!e) return MTE_E_OOM;
  e->cfg = c;
  if (hipGetDevice(&e->device) != hipSuccess) { delete e; return MTE_E_HIP; }
  auto fail = [&](int code) { mte_vision_destroy(e); return code; };

  const bool f16 = c.dtype == MTE_BF16;
  e->mode = f16 ? MODE_F16 : MODE_F32;
  e->act_fmt = f16 ? FMT_F16 : FMT_F32;
  const size_t es = v_esize(c.dtype);
  const size_t D = c.hidden, F = c.ffn, mm = (size_t)c.merge * c.merge, MD = mm * D, DO = c.out_hidden;
  const size_t KP = (size_t)c.in_channels * c.patch * c.patch;
  // weights: per layer qkv, o, fc1, fc2; then patch, m1, m2
  const size_t wl = (3 * D * D + D * D + F * D + D * F) * es;
  const size_t wtot = wl * c.depth + (D * KP + MD * MD + DO * MD) * es;
  const size_t fl = 4 * D + 3 * D + D + F + D;   // ln1 g,b, ln2 g,b, b_qkv, b_o, b_fc1, b_fc2
  const size_t ftot = fl * c.depth + D + 2 * D + MD + DO;
  if (hipMalloc(&e->wbuf, wtot) != hipSuccess || hipMalloc((void **)&e->fbuf, ftot * sizeof(float)) != hipSuccess)
    return fail(MTE_E_OOM);
  const size_t per = (size_t)(c.max_side / c.patch) * (c.max_side / c.patch);
  const size_t T = (size_t)c.max_images * per;
  if (hipMalloc(&e->patches, T * KP * es) != hipSuccess || hipMalloc((void **)&e->h, T * D * 4) != hipSuccess ||
      hipMalloc(&e->xn, T * D * es) != hipSuccess || hipMalloc((void **)&e->qkv, std::max(T * 3 * D * 4, ((T * 2 * D * 2 + 255) & ~(size_t)255) + (T + 31) / 32 * 32 * D * 2)) != hipSuccess ||
      hipMalloc(&e->attn, T * D * es) != hipSuccess || hipMalloc(&e->act, T * F * es) != hipSuccess ||
      hipMalloc(&e->mact, T * D * es) != hipSuccess || hipMalloc((void **)&e->mout, (T / mm + 1) * DO * 4) != hipSuccess ||
      hipMalloc((void **)&e->pos, 3 * T * 4) != hipSuccess ||
      hipMalloc((void **)&e->rcos, T * (c.head_dim / 2) * 4) != hipSuccess ||
      hipMalloc((void **)&e->rsin, T * (c.head_dim / 2) * 4) != hipSuccess)
    return fail(MTE_E_OOM);

  const int sf = v_in_fmt(c.dtype);
  hipError_t he = hipSuccess;
  // Range analysis (bf16): max |.| of every matrix and vector, and the
  // largest row norms of Wv (rows 2D..3D of w_qkv), W_fc1 and W_m1.
  enum { Q_QKV, Q_V, Q_O, Q_FC1, Q_FC2, Q_G1, Q_B1, Q_G2, Q_B2, Q_BQKV, Q_BFC1, Q_Q, Q_K, Q_N };
  enum { G_PATCH, G_M1, G_M2, G_MG, G_MB, G_BM1, G_N };
  std::vector<float> sth;
  const size_t nst = 2 * ((size_t)c.depth * Q_N + G_N);
  if (f16) {
    float *stt = nullptr;
    if (hipMalloc((void **)&stt, nst * sizeof(float)) != hipSuccess) return fail(MTE_E_OOM);
    he = hipMemsetAsync(stt, 0, nst * sizeof(float), stream);
    const size_t eb = es;
    for (int l = 0; l < c.depth && he == hipSuccess; ++l) {
      const mte_vision_layer_weights &L = w->layers[l];
      float *sl = stt + 2 * (size_t)l * Q_N;
      const struct { const void *p; size_t rows, cols; } m[Q_N] = {
          {L.w_qkv, 3 * D, D}, {(const char *)L.w_qkv + 2 * D * D * eb, D, D}, {L.w_o, D, D}, {L.w_fc1, F, D},
          {L.w_fc2, D, F}, {L.ln1_g, 1, D}, {L.ln1_b, 1, D}, {L.ln2_g, 1, D}, {L.ln2_b, 1, D}, {L.b_qkv, 1, 3 * D},
          {L.b_fc1, 1, F}, {L.w_qkv, D, D}, {(const char *)L.w_qkv + D * D * eb, D, D}};
      for (int k = 0; k < Q_N && he == hipSuccess; ++k)
        he = launch_matrix_stats(sf, m[k].p, (int)m[k].rows, (int)m[k].cols, sl + 2 * k, stream);
    }
    float *sg = stt + 2 * (size_t)c.depth * Q_N;
    const struct { const void *p; size_t rows, cols; } g[G_N] = {
        {w->patch_w, D, KP}, {w->merge_w1, MD, MD}, {w->merge_w2, DO, MD},
        {w->merge_ln_g, 1, D}, {w->merge_ln_b, 1, D}, {w->merge_b1, 1, MD}};
    for (int k = 0; k < G_N && he == hipSuccess; ++k)
      he = launch_matrix_stats(sf, g[k].p, (int)g[k].rows, (int)g[k].cols, sg + 2 * k, stream);
    sth.resize(nst);
    if (he == hipSuccess) he = hipMemcpyAsync(sth.data(), stt, nst * sizeof(float), hipMemcpyDeviceToHost, stream);
    if (he == hipSuccess) he = hipStreamSynchronize(stream);
    hipFree(stt);
    if (he != hipSuccess) return fail(MTE_E_HIP);
  }
  // Bounds (bf16): |LN(x) g + b|_2 <= sqrt(D) (max|g| + max|b|) = N_ln bounds
  // every element of a norm output and, times a row norm plus the bias, every
  // element of v (so of the attention output), of the fc1 / merger-m1 input to
  // gelu (|gelu(z)| <= |z|); the merger input is four such vectors (norm
  // 2 N_ln for merge 2).
  const double sqD = std::sqrt((double)D), rnm = 1.001;   // fp32 norm rounding margin
  char *wb = (char *)e->wbuf;
  float *fb = e->fbuf;
  auto take_w = [&](size_t elems) { void *p = wb; wb += elems * es; return p; };
  auto take_f = [&](size_t n) { float *p = fb; fb += n; return p; };
  auto conv_w = [&](const void *src, void *dst, size_t rows, size_t cols, int shift) {
    return launch_convert_rows(sf, src, f16 ? FMT_F16 : FMT_F32, dst, (int)rows, (int)cols, std::ldexp(1.f, shift), 0,
                               0, stream);
  };
  e->layers.resize(c.depth);
  for (int l = 0; l < c.depth && he == hipSuccess; ++l) {
    const mte_vision_layer_weights &L = w->layers[l];
    VLayer &o = e->layers[l];
    o.w_qkv = take_w(3 * D * D);
    o.w_o = take_w(D * D);
    o.w_fc1 = take_w(F * D);
    o.w_fc2 = take_w(D * F);
    o.ln1_g = take_f(D); o.ln1_b = take_f(D); o.ln2_g = take_f(D); o.ln2_b = take_f(D);
    o.b_qkv = take_f(3 * D); o.b_o = take_f(D); o.b_fc1 = take_f(F); o.b_fc2 = take_f(D);
    int wq = 0, wo = 0, w1 = 0, w2 = 0, k1 = 0, k2 = 0, ko = 0, ky = 0, kq = 0, kk = 0;
    if (f16) {
      const float *s = &sth[2 * (size_t)l * Q_N];
      auto mx = [&](int k) { return (double)s[2 * k]; };
      auto rn = [&](int k) { return (double)s[2 * k + 1] * rnm; };
      wq = v_weight_shift(mx(Q_QKV));
      wo = v_weight_shift(mx(Q_O));
      w1 = v_weight_shift(mx(Q_FC1));
      w2 = v_weight_shift(mx(Q_FC2));
      const double n1 = sqD * (mx(Q_G1) + mx(Q_B1)), n2 = sqD * (mx(Q_G2) + mx(Q_B2));
      k1 = v_act_shift(n1);
      k2 = v_act_shift(n2);
      ko = v_act_shift(n1 * rn(Q_V) + mx(Q_BQKV));
      ky = v_act_shift(n2 * rn(Q_FC1) + mx(Q_BFC1));
      // q and k likewise, times sqrt(2) for the rotation of each pair
      kq = v_act_shift(std::sqrt(2.0) * (n1 * rn(Q_Q) + mx(Q_BQKV)));
      kk = v_act_shift(std::sqrt(2.0) * (n1 * rn(Q_K) + mx(Q_BQKV)));
    }
    o.s_qkv = std::ldexp(1.f, k1 - wq);
    o.s_o = std::ldexp(1.f, ko - wo);
    o.s_fc1 = std::ldexp(1.f, k2 - w1);
    o.s_fc2 = std::ldexp(1.f, ky - w2);
    o.o_pre = std::ldexp(1.f, -ko);
    o.y_pre = std::ldexp(1.f, -ky);
    o.q_pre = std::ldexp(1.f, -kq);
    o.k_pre = std::ldexp(1.f, -kk);
    o.att_sc = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim) * std::ldexp(1.0, kq + kk));
    he = conv_w(L.w_qkv, o.w_qkv, 3 * D, D, wq);
    if (he == hipSuccess) he = conv_w(L.w_o, o.w_o, D, D, wo);
    if (he == hipSuccess) he = conv_w(L.w_fc1, o.w_fc1, F, D, w1);
    if (he == hipSuccess) he = conv_w(L.w_fc2, o.w_fc2, D, F, w2);
    const float p1 = std::ldexp(1.f, -k1), p2 = std::ldexp(1.f, -k2);
    if (he == hipSuccess) he = launch_to_f32(sf, L.ln1_g, o.ln1_g, (int)D, p1, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.ln1_b, o.ln1_b, (int)D, p1, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.ln2_g, o.ln2_g, (int)D, p2, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.ln2_b, o.ln2_b, (int)D, p2, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.b_qkv, o.b_qkv, (int)(3 * D), 1.f, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.b_o, o.b_o, (int)D, 1.f, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.b_fc1, o.b_fc1, (int)F, 1.f, stream);
    if (he == hipSuccess) he = launch_to_f32(sf, L.b_fc2, o.b_fc2, (int)D, 1.f, stream);
  }
  e->w_patch = take_w(D * KP);
  e->w_m1 = take_w(MD * MD);
  e->w_m2 = take_w(DO * MD);
  e->b_patch = take_f(D);
  e->mln_g = take_f(D);
  e->mln_b = take_f(D);
  e->b_m1 = take_f(MD);
  e->b_m2 = take_f(DO);
  int wp = 0, wm1 = 0, wm2 = 0, kq = 0, km = 0;
  if (f16) {
    const float *s = &sth[2 * (size_t)c.depth * Q_N];
    auto mx = [&](int k) { return (double)s[2 * k]; };
    auto rn = [&](int k) { return (double)s[2 * k + 1] * rnm; };
    wp = v_weight_shift(mx(G_PATCH));
    wm1 = v_weight_shift(mx(G_M1));
    wm2 = v_weight_shift(mx(G_M2));
    const double nm = sqD * (mx(G_MG) + mx(G_MB));
    kq = v_act_shift(nm);
    km = v_act_shift(std::sqrt((double)mm) * nm * rn(G_M1) + mx(G_BM1));
  }
  e->s_patch = std::ldexp(1.f, -wp);
  e->s_m1 = std::ldexp(1.f, kq - wm1);
  e->s_m2 = std::ldexp(1.f, km - wm2);
  e->m_pre = std::ldexp(1.f, -km);
  if (he == hipSuccess) he = conv_w(w->patch_w, e->w_patch, D, KP, wp);
  if (he == hipSuccess) he = conv_w(w->merge_w1, e->w_m1, MD, MD, wm1);
  if (he == hipSuccess) he = conv_w(w->merge_w2, e->w_m2, DO, MD, wm2);
  const float pq = std::ldexp(1.f, -kq);
  if (he == hipSuccess) he = launch_to_f32(sf, w->patch_b, e->b_patch, (int)D, 1.f, stream);
  if (he == hipSuccess) he = launch_to_f32(sf, w->merge_ln_g, e->mln_g, (int)D, pq, stream);
  if (he == hipSuccess) he = launch_to_f32(sf, w->merge_ln_b, e->mln_b, (int)D, pq, stream);
  if (he == hipSuccess) he = launch_to_f32(sf, w->merge_b1, e->b_m1, (int)MD, 1.f, stream);
  if (he == hipSuccess) he = launch_to_f32(sf, w->merge_b2, e->b_m2, (int)DO, 1.f, stream);
  if (he == hipSuccess) he = hipStreamSynchronize(stream);
  if (he != hipSuccess) return fail(MTE_E_HIP);

  // 2-D rotary: pair j turns with the patch row (axis 1) for j < d/4, with
  // the patch column (axis 2) otherwise, at theta^(-2j/d).
  const int half = c.head_dim / 2;
  for (int j = 0; j < 64; ++j) {
    e->rope.inv_freq[j] = j < half ? std::pow((double)c.rope_theta, -2.0 * j / c.head_dim) : 0.0;
    e->rope.axis[j] = (uint8_t)(j < half / 2 ? 1 : 2);
  }
  *out = e;
  return MTE_OK;
}

int mte_vision_encode(mte_vision *e, const void *pixels, int32_t n, int32_t H, int32_t W, void *out,
                      hipStream_t s) {
  if (!e || H <= 0 || W <= 0) return MTE_E_INVALID;
  const int side = e->cfg.patch * e->cfg.merge;
  return mte_vision_encode_strided(e, pixels, n, H, W, out, (H / side) * (W / side), s);
}

int mte_vision_encode_strided(mte_vision *e, const void *pixels, int32_t n, int32_t H, int32_t W, void *out,
                              int32_t image_stride, hipStream_t s) {
  if (!e || !pixels || !out || n <= 0 || H <= 0 || W <= 0) return MTE_E_INVALID;
  const mte_vision_config &c = e->cfg;
  const int side = c.patch * c.merge;
  if (H % side || W % side) return MTE_E_INVALID;
  const int tpi = (H / side) * (W / side);
  if (image_stride < tpi || (int64_t)image_stride * n > (1 << 24)) return MTE_E_INVALID;
  if (n > c.max_images || H > c.max_side || W > c.max_side) return MTE_E_CAPACITY;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return MTE_E_HIP;
  if (cur != e->device && hipSetDevice(e->device) != hipSuccess) return MTE_E_HIP;
  const int D = c.hidden, F = c.ffn, hd = c.head_dim, nh = c.n_heads, mm = c.merge * c.merge;
  const int KP = c.in_channels * c.patch * c.patch, MD = mm * D, DO = c.out_hidden;
  const int per = (H / c.patch) * (W / c.patch);
  const int T = n * per, Tm = T / mm;
  const int mode = e->mode, af = e->act_fmt;
  std::vector<int32_t> cu(n + 1);
  for (int i = 0; i <= n; ++i) cu[i] = i * per;
  int sp = 0;
  hipError_t err = hipSuccess;
#define MTE_TRY(x) do { err = (x); if (err != hipSuccess) goto done; } while (0)
  MTE_TRY(launch_patchify(v_in_fmt(c.dtype), pixels, n, c.in_channels, H, W, c.patch, c.merge, af, e->patches, s));
  MTE_TRY(launch_patch_positions(e->pos, n, H, W, c.patch, c.merge, s));
  MTE_TRY(launch_rope_table(e->pos, T, hd / 2, e->rope, e->rcos, e->rsin, s));
  MTE_TRY(launch_gemm(mode, EPI_STORE, e->patches, e->w_patch, e->h, T, D, KP, D, e->s_patch, 1.f, nullptr, 0, &sp,
                      nullptr, s, nullptr, e->b_patch));
  for (int l = 0; l < c.depth; ++l) {
    const VLayer &L = e->layers[l];
    QkvEpi qe{e->rcos, e->rsin, nullptr, nullptr, 2 * D, D, hd, c.ln_eps};
    // bf16 storage: fp16 attention operands in the matrix-core layout (q/k
    // rows [T, 2D], then V^T tiles), in the qkv region
    const bool half = mode != MODE_F32;
    if (half) {
      qe.qk = (f16 *)e->qkv;
      qe.vt = (f16 *)((char *)e->qkv + (((size_t)T * 2 * D * 2 + 255) & ~(size_t)255));
      qe.q_pre = L.q_pre;
      qe.k_pre = L.k_pre;
      qe.v_pre = L.o_pre;
      qe.hkv = nh;
    }
    MTE_TRY(launch_layernorm(e->h, L.ln1_g, L.ln1_b, af, e->xn, T, D, c.ln_eps, s));
    MTE_TRY(launch_gemm(mode, EPI_QKV, e->xn, L.w_qkv, e->qkv, T, 3 * D, D, 3 * D, L.s_qkv, 1.f, nullptr, 0, &sp,
                        &qe, s, nullptr, L.b_qkv));
    if (half)
      MTE_TRY(launch_attention_h(qe.qk, qe.vt, nullptr, nullptr, 0, (f16 *)e->attn, L.att_sc, cu.data(), n, T, nh, nh,
                                 hd, 0, s));
    else
      MTE_TRY(launch_attention(e->qkv, nullptr, 0, (float *)e->attn, cu.data(), n, nh, nh, hd, s, 0));
    MTE_TRY(launch_gemm(mode, EPI_RESID, e->attn, L.w_o, e->h, T, D, D, D, L.s_o, 1.f, nullptr, 0, &sp, nullptr, s,
                        nullptr, L.b_o));
    MTE_TRY(launch_layernorm(e->h, L.ln2_g, L.ln2_b, af, e->xn, T, D, c.ln_eps, s));
    MTE_TRY(launch_gemm(mode, EPI_GELU, e->xn, L.w_fc1, e->act, T, F, D, F, L.s_fc1, L.y_pre, nullptr, 0, &sp,
                        nullptr, s, nullptr, L.b_fc1));
    MTE_TRY(launch_gemm(mode, EPI_RESID, e->act, L.w_fc2, e->h, T, D, F, D, L.s_fc2, 1.f, nullptr, 0, &sp, nullptr,
                        s, nullptr, L.b_fc2));
  }
  // merger: the norm output [T, D] read as [T/mm, mm*D] concatenates each
  // group's patches in group order
  MTE_TRY(launch_layernorm(e->h, e->mln_g, e->mln_b, af, e->xn, T, D, c.ln_eps, s));
  MTE_TRY(launch_gemm(mode, EPI_GELU, e->xn, e->w_m1, e->mact, Tm, MD, MD, MD, e->s_m1, e->m_pre, nullptr, 0, &sp,
                      nullptr, s, nullptr, e->b_m1));
  if (c.out_dtype == MTE_F32 && image_stride == tpi) {
    MTE_TRY(launch_gemm(mode, EPI_STORE, e->mact, e->w_m2, out, Tm, DO, MD, DO, e->s_m2, 1.f, nullptr, 0, &sp,
                        nullptr, s, nullptr, e->b_m2));
  } else {
    MTE_TRY(launch_gemm(mode, EPI_STORE, e->mact, e->w_m2, e->mout, Tm, DO, MD, DO, e->s_m2, 1.f, nullptr, 0, &sp,
                        nullptr, s, nullptr, e->b_m2));
    MTE_TRY(launch_scatter_rows(e->mout, c.out_dtype == MTE_F32 ? FMT_F32 : FMT_BF16, out, Tm, DO, tpi,
                                image_stride, s));
  }
#undef MTE_TRY
done:
  if (cur != e->device) hipSetDevice(cur);
  return err == hipSuccess ? MTE_OK : MTE_E_HIP;
}

}  // extern "C"
