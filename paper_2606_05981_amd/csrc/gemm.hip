// Planning and launch of the projection GEMMs (k_gemm, gemm_kernel.h): a
// tile configuration and K split per (M, N, K, epilogue), from a table of
// measured choices for the decoder's projections, else from the number of
// workgroups a tile yields and its measured steady-state rate.
#include "gemm_kernel.h"

namespace mte {

static const TileCfg kTiles[] = {
#define MTE_TILE_INFO(id, bm, bn, wm, wn, rowb, p, occ, f32) {bm, bn, wm, wn, rowb, p, occ, f32},
    MTE_TILE_TABLE(MTE_TILE_INFO)
#undef MTE_TILE_INFO
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

int gemm_num_tiles() { return kNumTiles; }

// Whether tile `id` can run an (N, K, epilogue, splits) product: N a multiple of
// its width, each K split a whole number of stages, fp32 operands only on the
// tiles built for them, e4m3 weights only on 128-byte stages. col_align: columns
// a wave must cover in whole units (heads for the QKV epilogue; gate/up pairs
// sit inside every 32-column block).
static bool tile_fits(int id, int N, int K, int esz, int epi, int splits, int col_align = 32,
                      bool w8 = false) {
  const TileCfg &t = kTiles[id];
  if (N % t.bn || (esz == 4 && !t.f32) || (w8 && t.rowb != 128)) return false;
  if (t.p * (t.bm + (w8 ? t.bn / 2 : t.bn)) * t.rowb * t.occ > 160 * 1024) return false;   // LDS ring
  const int ks = t.rowb / esz;
  if (K % splits || (K / splits) % ks) return false;
  if (epi == EPI_QKV && (t.bn / t.wn) % col_align) return false;
  return true;
}

// Steady-state throughput of each tile (TFLOP/s of an fp16 GEMM with
// M = 10240, measured on MI355X); the fallback planner's only calibration.
static const double kTileRate[kNumTiles] = {959, 944, 895, 850, 850, 884, 850, 850, 800, 819,
                                            640, 777, 860, 600, 700, 650, 550, 450, 600, 600,
                                            921, 850, 850, 714, 766, 800, 1026, 1018, 850, 728,
                                            803, 950, 950, 1150, 1106, 1084, 940, 1044, 1117,
                                            300, 300, 300, 300, 300, 300, 300, 800, 800};

// Measured choices (MI355X sweep of every tile, split count and XCD placement,
// weights rotated through 600 MB so that they stream from HBM; at 96 and 192 rows
// timed together with the kernel that consumes the product; the leading
// candidates then timed again round robin, three times each, since a sweep
// in fixed order drifts with the clock as the card warms) for the decoder's four
// projections (D 2048 / FFN 6144 / 16+8+8 heads of 128) at 96 ... 10240 rows. A K split is only
// kept where it still wins after the consumer's extra pass over the fp32
// partial sums (at 1536 rows two QKV partials cost 16 us to add up, more than
// the split saves; the 1536-row QKV product runs on six-wave 192x128 tiles,
// one workgroup per CU, in 34 us against 37.6 for 128x128 tiles, which put
// two workgroups on half of the CUs and one on the rest). Other row counts
// take the entry of the nearest row
// count (log scale) for the same N, K and epilogue. `epi` is the epilogue of
// the finished product; splits > 1 means the K splits write partial sums
// that the consuming kernel adds up.
struct TileChoice {
  int n, k, epi, m, tile, splits;
  int xcd = 0;   // placement on the XCDs as 100 xa + 10 xb + xc (see GemmArgs), 0: by N tile
};
static const TileChoice kChoices[] = {
    {4096, 2048, EPI_QKV, 96, 42, 4},     {2048, 2048, EPI_RESID, 96, 42, 4},
    {12288, 2048, EPI_SWIGLU, 96, 42, 1},  {2048, 6144, EPI_RESID, 96, 42, 8},
    {4096, 2048, EPI_QKV, 192, 12, 2},    {2048, 2048, EPI_RESID, 192, 13, 4},
    {12288, 2048, EPI_SWIGLU, 192, 12, 1}, {2048, 6144, EPI_RESID, 192, 14, 8},
    {4096, 2048, EPI_QKV, 768, 12, 1, 241},    {2048, 2048, EPI_RESID, 768, 12, 2, 222},
    {12288, 2048, EPI_SWIGLU, 768, 3, 1},  {2048, 6144, EPI_RESID, 768, 14, 2},
    {4096, 2048, EPI_QKV, 1536, 47, 1, 241},   {2048, 2048, EPI_RESID, 1536, 14, 1, 181},
    {12288, 2048, EPI_SWIGLU, 1536, 33, 1}, {2048, 6144, EPI_RESID, 1536, 8, 2},
    {4096, 2048, EPI_QKV, 3072, 38, 1},   {2048, 2048, EPI_RESID, 3072, 8, 1},
    {12288, 2048, EPI_SWIGLU, 3072, 33, 1}, {2048, 6144, EPI_RESID, 3072, 8, 1},
    {4096, 2048, EPI_QKV, 10240, 38, 1, 421},  {2048, 2048, EPI_RESID, 10240, 36, 1, 421},
    {12288, 2048, EPI_SWIGLU, 10240, 33, 1}, {2048, 6144, EPI_RESID, 10240, 12, 1, 421},
    // vision tower (width 1024, MLP 4096, 768-value patches, 2x2 merger to 2048):
    // 16 images of 256 patches, merger at 1024 rows
    {3072, 1024, EPI_QKV, 4096, 38, 1},   {1024, 1024, EPI_RESID, 4096, 12, 1, 421},
    {4096, 1024, EPI_GELU, 4096, 38, 1},  {1024, 4096, EPI_RESID, 4096, 12, 1, 421},
    {1024, 768, EPI_STORE, 4096, 12, 1},  {4096, 4096, EPI_GELU, 1024, 30, 1},
    {2048, 4096, EPI_STORE, 1024, 18, 1},
};
// The same for e4m3 weights (tiles staging 128 bytes of A per row).
static const TileChoice kChoicesW8[] = {
    {4096, 2048, EPI_QKV, 96, 17, 4},     {2048, 2048, EPI_RESID, 96, 17, 4},
    {12288, 2048, EPI_SWIGLU, 96, 14, 1},  {2048, 6144, EPI_RESID, 96, 17, 8},
    {4096, 2048, EPI_QKV, 192, 17, 2},    {2048, 2048, EPI_RESID, 192, 17, 4},
    {12288, 2048, EPI_SWIGLU, 192, 14, 1}, {2048, 6144, EPI_RESID, 192, 12, 8},
    {4096, 2048, EPI_QKV, 1536, 36, 1, 421},   {2048, 2048, EPI_RESID, 1536, 14, 1, 181},
    {12288, 2048, EPI_SWIGLU, 1536, 33, 1}, {2048, 6144, EPI_RESID, 1536, 8, 2},
};

// Fallback estimate: rounds of workgroups over the compute units x the time
// one full round takes at the tile's measured rate. Split-K is only
// considered up to 2048 rows (2 splits above 256), and only where the
// partial sums fit `ws_elems`.
static void plan_model(int M, int N, int K, int esz, int epi, int col_align, size_t ws_elems,
                       bool w8, int *tile, int *splits) {
  const int cus = 256;
  double best = 1e30;
  *tile = -1;
  *splits = 1;
  for (int id = 0; id < kNumTiles; ++id) {
    for (int sp = 1; sp <= 8; sp *= 2) {
      if (sp > 1 && (M > 2048 || (M > 256 && sp > 2) || (size_t)sp * M * N > ws_elems)) continue;
      if (!tile_fits(id, N, K, esz, sp > 1 ? EPI_PARTIAL : epi, sp, col_align, w8)) continue;
      const TileCfg &t = kTiles[id];
      const double tiles = (double)(N / t.bn) * ((M + t.bm - 1) / t.bm) * sp;
      const double slots = (double)cus * t.occ;
      const double rounds = std::ceil(tiles / slots);
      const double work = 2.0 * t.bm * t.bn * ((double)K / sp);
      const double cost = rounds * slots * work / kTileRate[id] * (sp > 1 ? 1.15 : 1.0);
      if (cost < best) {
        best = cost;
        *tile = id;
        *splits = sp;
      }
    }
  }
}

static void plan(int M, int N, int K, int esz, int epi, int col_align, size_t ws_elems, bool w8,
                 int *tile, int *splits, int *xcd) {
  *xcd = 0;
  const TileChoice *best = nullptr;
  double bd = 1e30;
  if (esz == 2) {
    const TileChoice *tab = w8 ? kChoicesW8 : kChoices;
    const size_t ntab = w8 ? sizeof(kChoicesW8) / sizeof(kChoicesW8[0]) : sizeof(kChoices) / sizeof(kChoices[0]);
    for (size_t ci = 0; ci < ntab; ++ci) {
      const TileChoice &c = tab[ci];
      if (c.n != N || c.k != K || c.epi != epi) continue;
      const double d = std::fabs(std::log((double)M / c.m));
      if (d < bd) { bd = d; best = &c; }
    }
  }
  if (best &&
      tile_fits(best->tile, N, K, esz, best->splits > 1 ? EPI_PARTIAL : epi, best->splits, col_align, w8) &&
      (best->splits == 1 ||
       ((M <= 256 || (M <= 2048 && best->splits == 2)) && (size_t)best->splits * M * N <= ws_elems))) {
    *tile = best->tile;
    *splits = best->splits;
    *xcd = best->xcd;
    return;
  }
  plan_model(M, N, K, esz, epi, col_align, ws_elems, w8, tile, splits);
}

hipError_t launch_mode_f8w(int epi, int tile, int splits, const GemmArgs &a, hipStream_t s);

// Decodes an XCD placement 100 xa + 10 xb + xc into a, or clears it when it
// does not fit the grid (xa x xb x xc != 8, or a factor not dividing its grid
// dimension): the placement only permutes tiles, so any grid stays correct.
static void set_xcd(GemmArgs &a, int code, int gm, int gn, int splits) {
  const int xa = code / 100, xb = (code / 10) % 10, xc = code % 10;
  a.xa = a.xb = a.xc = 0;
  if (code <= 0 || xa * xb * xc != 8 || gm % xa || gn % xb || splits % xc) return;
  a.xa = xa;
  a.xb = xb;
  a.xc = xc;
}

hipError_t launch_gemm_tile(int mode, int epi, int tile, int splits, const void *A, const void *W,
                            void *C, size_t c_plane, int M, int N, int K, int ldc, float scale,
                            float out_scale, const QkvEpi *qe, hipStream_t s, const float *col_scale,
                            const float *bias, int xcd) {
  if (M <= 0) return hipSuccess;
  const bool w8 = mode == MODE_F8W;
  if (bias && splits > 1) return hipErrorInvalidValue;
  const int esz = mode == MODE_F32 ? 4 : 2;
  if (epi == EPI_QKV && (!qe || (qe->hd != 64 && qe->hd != 128))) return hipErrorInvalidValue;
  if (w8 && !col_scale) return hipErrorInvalidValue;
  // the kernel addresses both operands with 32-bit byte offsets
  if ((size_t)M * K * esz > 0xFFFFFFFFull || (size_t)N * K * (w8 ? 1 : esz) > 0xFFFFFFFFull)
    return hipErrorInvalidValue;
  if (tile < 0 || tile >= kNumTiles || splits < 1 ||
      !tile_fits(tile, N, K, esz, epi, splits, epi == EPI_QKV ? qe->hd : 32, w8) ||
      (splits > 1 && epi != EPI_PARTIAL))
    return hipErrorInvalidValue;
  GemmArgs a{(const char *)A, (const char *)W, C, c_plane, M, N, K, ldc, K / splits, scale, out_scale,
             epi == EPI_QKV ? *qe : QkvEpi{}, w8 ? col_scale : nullptr, bias, 0, 0, 0};
  set_xcd(a, xcd, (M + kTiles[tile].bm - 1) / kTiles[tile].bm, N / kTiles[tile].bn, splits);
  if (w8) return launch_mode_f8w(epi, tile, splits, a, s);
  return mode == MODE_F16 ? launch_mode<MODE_F16>(epi, tile, splits, a, s)
                          : launch_mode<MODE_F32>(epi, tile, splits, a, s);
}

hipError_t launch_gemm(int mode, int epi, const void *A, const void *W, void *C, int M, int N, int K,
                       int ldc, float scale, float out_scale, float *ws, size_t ws_elems,
                       int *splits_out, const QkvEpi *qe, hipStream_t s, const float *col_scale,
                       const float *bias) {
  *splits_out = 0;
  if (M <= 0) return hipSuccess;
  if (epi == EPI_QKV && !qe) return hipErrorInvalidValue;
  int tile, splits, xcd;
  plan(M, N, K, mode == MODE_F32 ? 4 : 2, epi, epi == EPI_QKV ? qe->hd : 32, (ws && !bias) ? ws_elems : 0,
       mode == MODE_F8W, &tile, &splits, &xcd);
  if (tile < 0) return hipErrorInvalidValue;
  if (splits > 1) {
    *splits_out = splits;
    return launch_gemm_tile(mode, EPI_PARTIAL, tile, splits, A, W, ws, (size_t)M * N, M, N, K, N, scale,
                            1.f, nullptr, s, col_scale, nullptr, xcd);
  }
  return launch_gemm_tile(mode, epi, tile, 1, A, W, C, 0, M, N, K, ldc, scale, out_scale, qe, s, col_scale,
                          bias, xcd);
}

}  // namespace mte