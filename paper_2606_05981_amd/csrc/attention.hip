// Causal grouped-query attention over packed, ragged sequences (prefill).
//
// For every sequence, query head h and token i:
//   o[i, h] = sum_{j <= i} softmax_j(q_i . k_j / sqrt(d)) v_j,
// with k, v taken from kv head h / (Hq / Hkv) and j ranging over the same
// sequence only (q and k arrive normalised and rotated).
//
// Three kernels. With bf16 storage (decoder and vision tower) q, k and v
// arrive as fp16 operands that the QKV projection already wrote in the
// matrix-core layout: k_attn_s stages a workgroup's key range in LDS (in
// rounds when it is long), k_attn_h streams it from global memory for shapes
// the staged kernel's 4- or 8-wave workgroups do not cover (both at the end
// of this file). k_attn below serves fp32 storage, on the fp32 matrix cores:
//
// One workgroup (4 waves) serves one kv head, one tile of query rows of one
// sequence and the query heads of that kv head assigned to it; every wave
// owns 32 query rows of one query head. Key/value tiles of 32 tokens are
// staged in LDS once and shared by all four waves (K row-major, V
// transposed, its keys permuted so that every MFMA operand fragment is one
// 16-byte LDS read). Per wave and kv tile:
//   S^T = K Q^T   (32x32 MFMA; lane l ends up owning query l%32)
//   online softmax in fp32 over the lane's 16 scores plus one cross-lane
//   exchange (lane ^ 32)
//   O^T += V^T P^T  (32x32 MFMA; again query l%32 per lane, so the
//   rescaling of O by the running-max correction is a per-lane scalar).
// q, k, v arrive as fp32 rows of the packed QKV projection; o is written in
// fp32. The sequence table (offsets, first tile of each sequence) is passed
// by value in the kernel arguments, so nothing is read back to the host.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace mte {

constexpr int kMaxSeqPerLaunch = 256;

struct AttnArgs {
  const float *qkv;   // [T, ld_qkv] fp32
  const float *pre;   // [P, ld_qkv] fp32: keys / values of a shared prefix every sequence sees, or null
  int P;              // prefix length (0: none)
  float *o;
  int ld_qkv;      // floats per token row of qkv
  int Hq, Hkv, rep;
  int wph;         // waves per query head (query rows per workgroup = 32 * wph)
  int hpb;         // query heads per workgroup
  int head_blocks;
  int n_seq;
  int causal;      // 0: every query sees all keys of its sequence (and the prefix)
  int cu[kMaxSeqPerLaunch + 1];     // absolute token offsets
  int tile0[kMaxSeqPerLaunch + 1];  // first workgroup tile of each sequence
};

template <int NCH>
__device__ __forceinline__ int kswz(int r, int c) {
  if constexpr (NCH >= 16) return c ^ (r & 15);
  else return c ^ ((r ^ (r >> 3)) & 7);
}


// Position of key k (0..31) of a tile in a row of the transposed V stage:
// the P fragment f of lane group g holds the probabilities of keys
// 8*(i/4) + 4g + i%4 for i = EPF*f .. EPF*f + EPF-1 (the S accumulator
// layout), so those keys are stored contiguously at (2f + g) * EPF.
template <int EPF>
__device__ __forceinline__ int vt_pos(int k) {
  const int a = k >> 3, g = (k >> 2) & 1, c = k & 3;
  const int i = 4 * a + c;
  return (2 * (i / EPF) + g) * EPF + (i % EPF);
}

// NB: key/value tiles staged at once. NB = 1 keeps a ring of one tile with
// the next one in flight in registers (any length); NB > 1 loads all of a
// workgroup's tiles up front (sequences of at most NB * 32 tokens), so the
// whole key/value range costs one global-load latency and one barrier.
template <int HD, int NB>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  constexpr int KV = 32;
  constexpr int EC = 4;                          // fp32 elements per 16-byte chunk
  constexpr int NCH = HD / EC;                   // chunks per head row
  constexpr int EPF = Frag<float>::kElems;       // values per P / V fragment
  constexpr int NFP = 16 / EPF;                  // P fragments per 32-kv tile
  constexpr int VTP = KV + 4;                    // V^T row pitch: 16-byte aligned, conflict-free
  constexpr int ND = HD / 32;                    // 32-wide d blocks
  typedef f32x4 frag_t;

  constexpr int K_BYTES = KV * NCH * 16;
  constexpr int V_BYTES = HD * VTP * 4;
  constexpr int ST_BYTES = K_BYTES + V_BYTES;             // one staged tile
  constexpr int SMEM = NB * ST_BYTES;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  // tile b: K [KV * NCH] at smem + b * ST_BYTES, V^T [HD * VTP] after it
  auto sK_of = [&](int b) { return (u32x4 *)(smem + b * ST_BYTES); };
  auto sVt_of = [&](int b) { return (float *)(smem + b * ST_BYTES + K_BYTES); };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 31, lgrp = lane >> 5;

  // Which sequence / query tile / heads this workgroup serves.
  const int tile = blockIdx.x;
  int lo = 0, hi = a.n_seq - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (a.tile0[mid] <= tile) lo = mid; else hi = mid - 1;
  }
  const int seq = lo;
  const int s0 = a.cu[seq], L = a.cu[seq + 1] - s0;
  const int QT = 32 * a.wph;
  const int q0 = (tile - a.tile0[seq]) * QT;
  const int g = blockIdx.y / a.head_blocks, hb = blockIdx.y % a.head_blocks;
  const int head = g * a.rep + hb * a.hpb + wave / a.wph;
  const int P = a.P;                               // keys of the shared prefix
  const int q_last = min(q0 + QT, L) - 1;          // last valid query row of the workgroup
  // With every key tile staged at once and two waves per head, a head's
  // second 32-row block past the end of the sequence would leave its wave
  // idle: that wave instead takes the upper part of the first block's key
  // tiles, and the two partial softmax states are merged through LDS before
  // the output (a causal 96-token frame: 2 + 1 tiles instead of 3 on one wave).
  const int n_first = a.causal ? ((P + min(q0 + 31, L - 1)) / KV + 1) : ((P + L - 1) / KV + 1);
  const bool pair_split = NB > 1 && a.wph == 2 && q0 < L && q0 + 32 >= L && n_first >= 2;   // workgroup-uniform
  const bool helper = pair_split && (wave & 1);
  const int kb_split = n_first - n_first / 2;      // the helper's first key tile
  const int qw = q0 + (wave % a.wph) * 32 - (helper ? 32 : 0);   // first query row of this wave
  const int wave_last = min(qw + 31, L - 1);       // last valid query row of this wave
  const size_t ld = (size_t)a.ld_qkv;
  const size_t base = (size_t)s0 * ld;             // element offset of the sequence's first row
  const int k_off = (a.Hq + g) * HD;
  const int v_off = (a.Hq + a.Hkv + g) * HD;

  // Q fragments of this wave's 32 rows (B operand of S^T = K Q^T); rows
  // past the sequence read its last row (their outputs are not stored).
  // Loaded after the first key/value tiles' loads are issued, so that the
  // two global-load round trips overlap.
  frag_t qf[NCH / 2];
  auto load_q = [&]() {
    const int qi = min(qw + lrow, L - 1);
#pragma unroll
    for (int kk = 0; kk < NCH / 2; ++kk)
      qf[kk] = *(const f32x4 *)(a.qkv + base + (size_t)qi * ld + head * HD + (kk * 2 + lgrp) * EC);
  };
  // Scores are kept in log2 units: s * log2(e) / sqrt(d).
  const float sc = 1.4426950408889634f * rsqrtf((float)HD);

  f32x16 oacc[ND];
#pragma unroll
  for (int n = 0; n < ND; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[n][r] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;
  const int my_q = qw + lrow;

  // Keys are numbered over [0, P + L): the shared prefix's first, then the
  // sequence's own; own query i sits at key index P + i.
  const int n_blocks = (q_last < 0) ? 0 : a.causal ? ((P + q_last) / KV + 1) : ((P + L - 1) / KV + 1);
  auto key_row = [&](int kv) -> const float * {
    kv = min(kv, P + L - 1);
    return kv < P ? a.pre + (size_t)kv * ld : a.qkv + base + (size_t)(kv - P) * ld;
  };
  // Staging of one key/value tile through registers, one tile ahead:
  //  K: thread chunk (row r, chunk c) of EC consecutive d -> sK[r][c] (swizzled);
  //  V: thread (column d, row group v) reads EC rows of column d (lanes
  //     take consecutive d, so each load is one coalesced row segment) and
  //     writes them into row d of V^T at their permuted key positions.
  // Rows past the sequence read its last row: their scores are masked, so
  // they add exact zeros.
  constexpr int KCH = KV * NCH / 256;             // K chunks per thread
  constexpr int VCH = HD * (KV / EC) / 256;       // V column groups per thread
  static_assert(KCH * 256 == KV * NCH && VCH * 256 == HD * (KV / EC), "staging split");
  float kx[NB][KCH][EC], vx[NB][VCH][EC];
  // This thread's element offsets inside a tile of KV consecutive rows of
  // pitch ld: K chunk t (row idx / NCH, chunk idx % NCH), V column group t
  // (rows v*EC.., column d). 32-bit: a tile spans at most KV * ld elements.
  const int ldi = a.ld_qkv;
  int koff[KCH], voff[VCH];
#pragma unroll
  for (int t = 0; t < KCH; ++t) {
    const int idx = tid + t * 256;
    koff[t] = (idx / NCH) * ldi + k_off + (idx % NCH) * EC;
  }
#pragma unroll
  for (int t = 0; t < VCH; ++t) {
    const int idx = tid + t * 256;
    voff[t] = (idx / HD) * EC * ldi + v_off + idx % HD;
  }
  // Global loads of the tile at kv0 into register slot b. A tile wholly
  // inside the sequence's own keys or wholly inside the prefix is one block
  // of rows at a workgroup-uniform base; the tile that straddles the prefix
  // boundary or the end of the sequence goes row by row (clamped rows read
  // the sequence's last key, whose scores are masked).
  auto gload = [&](int b, int kv0) {
    const bool own = kv0 >= P && kv0 + KV <= P + L;
    const bool pre = kv0 + KV <= P;
    if (own || pre) {
      const float *tb = own ? a.qkv + base + (size_t)(kv0 - P) * ld : a.pre + (size_t)kv0 * ld;
#pragma unroll
      for (int t = 0; t < KCH; ++t)
#pragma unroll
        for (int e = 0; e < EC; e += 4) {
          const f32x4 v = *(const f32x4 *)(tb + koff[t] + e);
          kx[b][t][e] = v[0]; kx[b][t][e + 1] = v[1]; kx[b][t][e + 2] = v[2]; kx[b][t][e + 3] = v[3];
        }
#pragma unroll
      for (int t = 0; t < VCH; ++t)
#pragma unroll
        for (int e = 0; e < EC; ++e) vx[b][t][e] = tb[voff[t] + e * ldi];
      return;
    }
#pragma unroll
    for (int t = 0; t < KCH; ++t) {
      const int idx = tid + t * 256, c = idx % NCH;
      const float *kr = key_row(kv0 + idx / NCH);
#pragma unroll
      for (int e = 0; e < EC; e += 4) {
        const f32x4 v = *(const f32x4 *)(kr + k_off + c * EC + e);
        kx[b][t][e] = v[0]; kx[b][t][e + 1] = v[1]; kx[b][t][e + 2] = v[2]; kx[b][t][e + 3] = v[3];
      }
    }
#pragma unroll
    for (int t = 0; t < VCH; ++t) {
      const int idx = tid + t * 256, d = idx % HD, v = idx / HD;
#pragma unroll
      for (int e = 0; e < EC; ++e)
        vx[b][t][e] = key_row(kv0 + v * EC + e)[v_off + d];
    }
  };
  // Register slot b -> LDS tile sKb / sVtb.
  auto lstore = [&](int b, u32x4 *sKb, float *sVtb) {
#pragma unroll
    for (int t = 0; t < KCH; ++t) {
      const int idx = tid + t * 256, r = idx / NCH, c = idx % NCH;
      u32x4 w;
      __builtin_memcpy(&w, kx[b][t], 16);
      sKb[r * NCH + kswz<NCH>(r, c)] = w;
    }
#pragma unroll
    for (int t = 0; t < VCH; ++t) {
      const int idx = tid + t * 256, d = idx % HD, v = idx / HD;
      // keys v*EC .. v*EC+3 land in a run of 4 consecutive positions
      u32x4 w;
      __builtin_memcpy(&w, vx[b][t], 16);
      *(u32x4 *)(sVtb + d * VTP + vt_pos<EPF>(v * EC)) = w;
    }
  };
  // One key/value tile for this wave: scores, online softmax, O update.
  auto compute = [&](int kv0, const u32x4 *sK, const float *sVt) {
    if (!(qw < L && kv0 <= (a.causal ? P + wave_last : P + L - 1))) return;
    // Two accumulators (by k parity) so consecutive MFMAs do not wait on
    // each other's results.
    f32x16 sacc[2];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[u][r] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NCH / 2; ++kk) {
      const int slot = lrow * NCH + kswz<NCH>(lrow, kk * 2 + lgrp);
      mfma32(sacc[kk & 1], __builtin_bit_cast(frag_t, sK[slot]), qf[kk]);
    }
    f32x16 s = sacc[0] + sacc[1];
    float mb = -INFINITY;
    // a tile every query of the wave sees in full needs no mask
    const bool full = kv0 + KV <= P + L && (!a.causal || kv0 + KV - 1 <= P + qw);
    if (full) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] *= sc;
        mb = fmaxf(mb, s[r]);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kv = kv0 + acc_row(r, lane);
        s[r] = ((!a.causal || kv <= P + my_q) && kv < P + L) ? s[r] * sc : -INFINITY;
        mb = fmaxf(mb, s[r]);
      }
    }
    mb = warp_max_xor(mb, 32);
    const float m_new = fmaxf(m_i, mb);
    // no key of the query seen yet (a helper's range can start past it):
    // exponentiate against 0 so that every term is an exact 0, not NaN
    const float m_ref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m_i - m_ref);
    m_i = m_new;
    float p[16];
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = exp2f(s[r] - m_ref);
      ps += p[r];
    }
    l_i = l_i * alpha + ps;
    // the running max moved for some query of the wave: rescale O
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;
    }
    // P fragments: element e of fragment f is P value i = EPF*f + e.
    // Consecutive MFMAs go to the ND different output blocks.
#pragma unroll
    for (int f = 0; f < NFP; ++f) {
      const frag_t pf = {p[EPF * f], p[EPF * f + 1], p[EPF * f + 2], p[EPF * f + 3]};
      frag_t vf[ND];
#pragma unroll
      for (int n = 0; n < ND; ++n) vf[n] = *(const frag_t *)(sVt + (n * 32 + lrow) * VTP + (2 * f + lgrp) * EPF);
#pragma unroll
      for (int n = 0; n < ND; ++n) mfma32(oacc[n], vf[n], pf);
    }
  };
  if constexpr (NB == 1) {
    if (n_blocks > 0) gload(0, 0);
    load_q();
    for (int kb = 0; kb < n_blocks; ++kb) {
      const int kv0 = kb * KV;
      lstore(0, sK_of(0), sVt_of(0));
      __syncthreads();
      if (kb + 1 < n_blocks) gload(0, kv0 + KV);
      compute(kv0, sK_of(0), sVt_of(0));
      __syncthreads();
    }
  } else {
    // n_blocks <= NB (the host launches this variant for short sequences only)
#pragma unroll
    for (int b = 0; b < NB; ++b)
      if (b < n_blocks) gload(b, b * KV);
    __builtin_amdgcn_sched_barrier(0);   // every tile's loads in flight before the first LDS write
    load_q();
#pragma unroll
    for (int b = 0; b < NB; ++b)
      if (b < n_blocks) lstore(b, sK_of(b), sVt_of(b));
    __syncthreads();
    const int kb_lo = helper ? kb_split : 0;
    const int kb_hi = (pair_split && !helper) ? kb_split : n_blocks;
    for (int kb = kb_lo; kb < kb_hi; ++kb) compute(kb * KV, sK_of(kb), sVt_of(kb));
    if (pair_split) {
      // Every wave is done with the staged tiles; the helper's state (m, l,
      // the O^T accumulators) goes over them in lane order, one slab per
      // head, and its partner rescales both parts to the common max.
      constexpr int MS = 2 + ND * 16;
      static_assert(2 * MS * 64 * 4 <= SMEM, "merge slabs fit the stage buffers");
      __syncthreads();
      float *mx = (float *)smem + (size_t)(wave >> 1) * MS * 64 + lane;
      if (helper) {
        mx[0] = m_i;
        mx[64] = l_i;
#pragma unroll
        for (int n = 0; n < ND; ++n)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx[(2 + n * 16 + r) * 64] = oacc[n][r];
      }
      __syncthreads();
      if (!helper) {
        const float mb = mx[0], lb = mx[64];
        const float m = fmaxf(m_i, mb);           // finite: the partner saw key 0
        const float fa = exp2f(m_i - m), fb = exp2f(mb - m);
        l_i = l_i * fa + lb * fb;
        m_i = m;
#pragma unroll
        for (int n = 0; n < ND; ++n)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[n][r] = oacc[n][r] * fa + mx[(2 + n * 16 + r) * 64] * fb;
      }
    }
  }

  // Output. oacc[n] holds rows d = 32 n + acc_row(r, lane) of O^T for the
  // lane's query: accumulator registers 4c..4c+3 are four consecutive d, so
  // each lane writes them as one 16-byte store into its query's row, and the
  // two lane groups fill 32 contiguous bytes.
  const float inv = 1.f / (l_i + __shfl_xor(l_i, 32, kWave));
  if (my_q < L && !helper) {
    const size_t orow = ((size_t)(s0 + my_q) * a.Hq + head) * HD + 4 * lgrp;
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        f32x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = oacc[n][4 * c + e] * inv;
        *(f32x4 *)(a.o + orow + n * 32 + 8 * c) = y;
      }
  }
}

hipError_t launch_attention(const float *qkv, const float *prefix, int P, float *o, const int32_t *cu, int batch,
                            int Hq, int Hkv, int d, hipStream_t s, int causal) {
  const int rep = Hq / Hkv;
  if (P < 0 || (P > 0 && !prefix) || (d != 64 && d != 128) || Hq % Hkv) return hipErrorInvalidValue;
  AttnArgs a;
  a.causal = causal ? 1 : 0;
  a.qkv = qkv;
  a.pre = prefix;
  a.P = P;
  a.ld_qkv = (Hq + 2 * Hkv) * d;
  a.o = o;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.rep = rep;
  if (rep >= 4) { a.wph = 1; a.hpb = 4; a.head_blocks = rep / 4; }
  else { a.wph = 4 / rep; a.hpb = rep; a.head_blocks = 1; }
  const int QT = 32 * a.wph;
  for (int first = 0; first < batch; first += kMaxSeqPerLaunch) {
    const int n = batch - first < kMaxSeqPerLaunch ? batch - first : kMaxSeqPerLaunch;
    a.n_seq = n;
    int tiles = 0, max_len = 0;
    for (int i = 0; i < n; ++i) {
      a.cu[i] = cu[first + i];
      a.tile0[i] = tiles;
      const int L = cu[first + i + 1] - cu[first + i];
      tiles += (L + QT - 1) / QT;
      max_len = L > max_len ? L : max_len;
    }
    a.cu[n] = cu[first + n];
    a.tile0[n] = tiles;
    if (tiles == 0) continue;
    dim3 grid(tiles, Hkv * a.head_blocks);
    // Sequences of at most 128 tokens: every workgroup stages all of its
    // (at most 4) key/value tiles at once.
    const bool all = P + max_len <= 4 * 32;
    if (d == 128 && all) hipLaunchKernelGGL((k_attn<128, 4>), grid, dim3(256), 0, s, a);
    else if (d == 128) hipLaunchKernelGGL((k_attn<128, 1>), grid, dim3(256), 0, s, a);
    else if (all) hipLaunchKernelGGL((k_attn<64, 4>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn<64, 1>), grid, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ------------------------------------------------------------------
// Attention on fp16 operands in the matrix-core layout (launch_attention_h).
//
// Every wave owns one (sequence, query head, block of 32 queries) and works
// alone: no LDS, no barriers. Its q fragments stay in registers; per key
// tile of 32 tokens it reads the k fragments straight from the k rows (each
// lane one 16-byte piece of one key row) and the V^T fragments from the
// pre-arranged tiles (one 16-byte piece per lane and output block), forms
// S^T = K Q^T on eight fp16 MFMAs (lane l owns query l % 32 and 16 of the
// keys), the online softmax in fp32 with one cross-lane exchange, and
// O^T += V^T P^T on two fp16 MFMAs per 32 output columns. Key tiles are the
// batch's global 32-token tiles, so a sequence that starts inside a tile
// masks the tile's leading keys; keys of other sequences and zero-padded
// rows past the batch enter with probability exactly 0. The next tile's k
// fragments are loaded while the current tile is computed. Masks are
// selects on the key index, exponentials the hardware base-2 exponential
// (v_exp_f32; the arguments are <= 0, exp2(-inf) = 0).
// With KS > 1 (few work items, e.g. one frame) a workgroup of KS waves
// serves one item: wave w takes key tiles w, w + KS, ..., and wave 0 merges
// the partial softmax states (running max, sum, O) of the others from LDS,
// so an item's chain of dependent tile steps is KS times shorter.
// A wave's output for its lanes' queries: registers 4c..4c+3 of oacc[n] are
// d = 32 n + 8 c + 4 g + 0..3 of the lane's query (g = lane / 32). For each
// pair (2p, 2p+1) one v_permlane32_swap gives lane g = 0 the d 16p + 0..7 and
// lane g = 1 the d 16p + 8..15 of block n, so each lane stores 16 contiguous
// bytes (half the stores of 8-byte pieces, each to another row). `row`: the
// query's first output value plus 8 g; every lane of the wave takes part,
// lanes with `valid` false store nothing.
template <int HD>
__device__ __forceinline__ void store_o(const f32x16 (&oacc)[HD / 32], float inv, f16 *row, bool valid) {
#pragma unroll
  for (int n = 0; n < HD / 32; ++n)
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      f16x4 lo, hi;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = (f16)(oacc[n][8 * p + e] * inv);
        hi[e] = (f16)(oacc[n][8 * p + 4 + e] * inv);
      }
      u32x2 x = __builtin_bit_cast(u32x2, lo), y = __builtin_bit_cast(u32x2, hi);
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        // the upper 32 lanes' x and the lower 32 lanes' y trade places
        const auto r = __builtin_amdgcn_permlane32_swap(x[w], y[w], false, false);
        x[w] = r[0];
        y[w] = r[1];
      }
      if (valid) *(u32x4 *)(row + n * 32 + 16 * p) = u32x4{x[0], x[1], y[0], y[1]};
    }
}

struct AttnHArgs {
  const f16 *qk;      // [T, ldq]
  const f16 *vt;      // [ceil(T / 32)][Hkv][HD][32]
  const f16 *pqk;     // shared prefix rows [P, ldq], or null
  const f16 *pvt;     // shared prefix V^T tiles [ceil(P / 32)][Hkv][HD][32]
  f16 *o;             // [T, Hq HD]
  float sc;           // log2(e) / sqrt(d), times the inverse q and k pre-scales
  int ldq;            // halfs per qk row, (Hq + Hkv) HD
  int T, P;
  int Hq, Hkv, rep;
  int n_seq, causal;
  int n_items;        // waves of work in this launch
  int cu[kMaxSeqPerLaunch + 1];    // absolute token offsets
  int blk0[kMaxSeqPerLaunch + 1];  // first 32-query block of each sequence
};

template <int HD, int WPB, int KS, int MT>
__global__ __launch_bounds__(64 * WPB * KS) void k_attn_h(AttnHArgs a) {
  static_assert(KS == 1 || WPB == 1, "key split: one item per workgroup");
  constexpr int ND = HD / 32;   // 32-wide output blocks
  constexpr int NK = HD / 16;   // 16-deep MFMA steps of q . k
  const int lane = threadIdx.x & 63, lrow = lane & 31, lgrp = lane >> 5;
  const int kw = KS > 1 ? (int)(threadIdx.x >> 6) : 0;   // key-split wave
  const int w = KS > 1 ? (int)blockIdx.x : (int)(blockIdx.x * WPB + (threadIdx.x >> 6));
  // KS = 1: wave-uniform exit, nothing below synchronises waves; KS > 1: the
  // whole workgroup exits together (one item per workgroup)
  if (w >= a.n_items) return;
  const int bi = w / a.Hq, head = w % a.Hq, kvh = head / a.rep;
  int lo = 0, hi = a.n_seq - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.blk0[mid] <= bi) lo = mid; else hi = mid - 1;
  }
  const int s0 = a.cu[lo], L = a.cu[lo + 1] - s0;
  const int q0 = (bi - a.blk0[lo]) * 32;           // first query of the wave (within the sequence)
  const int my_q = q0 + lrow;
  const int q_last = min(q0 + 31, L - 1);
  const int P = a.P;
  const int koff = (a.Hq + kvh) * HD + lgrp * 8;   // this lane's 8 d of a key row

  f16x8 qf[NK];
  {
    const f16 *qr = a.qk + (size_t)(s0 + min(my_q, L - 1)) * a.ldq + head * HD + lgrp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = *(const f16x8 *)(qr + kk * 16);
  }
  f32x16 oacc[ND];
#pragma unroll
  for (int n = 0; n < ND; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[n][r] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;

  // Key tiles: the prefix's tiles 0 .. np-1, then the batch's global tiles
  // t_lo .. t_hi holding the sequence's visible keys.
  const int np = (P + 31) >> 5;
  const int kend = a.causal ? q_last : L - 1;      // last own key any query of the wave sees
  const int t_lo = s0 >> 5, t_hi = (s0 + kend) >> 5;
  const int nt = np + (t_hi - t_lo + 1);
  auto kload = [&](int u, f16x8 (&kf)[NK]) {
    const f16 *src;
    int row;
    if (u < np) { src = a.pqk; row = min(u * 32 + lrow, P - 1); }
    else { src = a.qk; row = min((t_lo + u - np) * 32 + lrow, a.T - 1); }
    const f16 *kr = src + (size_t)row * a.ldq + koff;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) kf[kk] = *(const f16x8 *)(kr + kk * 16);
  };
  auto vload = [&](int u, f16x8 (&vf)[ND][2]) {
    const bool pre = u < np;
    const int t = pre ? u : t_lo + u - np;
    const f16 *vb = (pre ? a.pvt : a.vt) + (((size_t)t * a.Hkv + kvh) * HD + lrow) * 32 + lgrp * 8;
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int f = 0; f < 2; ++f) vf[n][f] = *(const f16x8 *)(vb + (size_t)n * 32 * 32 + f * 16);
  };
  // k fragments of the wave's first tile now, of each next tile while the
  // current one is computed; V^T fragments at the start of their tile (they
  // are needed only after the softmax)
  f16x8 kf[NK], kn[NK];
  if (kw < nt) kload(kw, kf);
  // key-tile index u -> (prefix tile?, tile of its source, rows the lane's
  // query sees there)
  auto tile_of = [&](int u, int &t, int &k_lo, int &k_hi) {
    const bool pre = u < np;
    t = pre ? u : t_lo + u - np;
    k_lo = pre ? 0 : s0;
    k_hi = pre ? P - 1 : (a.causal ? s0 + min(my_q, L - 1) : s0 + L - 1);
  };
  if constexpr (MT > 0) {
    // Two passes over at most MT tiles per wave: all scores first (kept in
    // registers), one max, then the probabilities and O; no rescaling of O.
    f32x16 sv[MT];
    float mb = -INFINITY;
#pragma unroll
    for (int x = 0; x < MT; ++x) {
      const int u = kw + x * KS;
      if (u < nt) {                                  // wave-uniform
        int t, k_lo, k_hi;
        tile_of(u, t, k_lo, k_hi);
        f32x16 sacc[2];
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[y][r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) mfma32(sacc[kk & 1], kf[kk], qf[kk]);
        if (u + KS < nt) kload(u + KS, kn);
        const int kb = t * 32 + 4 * lgrp;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int k = kb + 8 * (r >> 2) + (r & 3);
          const float v = sacc[0][r] + sacc[1][r];
          sv[x][r] = ((k >= k_lo) & (k <= k_hi)) ? v * a.sc : -INFINITY;
          mb = fmaxf(mb, sv[x][r]);
        }
        if (u + KS < nt) {
#pragma unroll
          for (int kk = 0; kk < NK; ++kk) kf[kk] = kn[kk];
        }
      }
    }
    mb = warp_max_xor(mb, 32);
    m_i = mb;
    const float m_ref = mb == -INFINITY ? 0.f : mb;  // a key-split wave may own no tile
    f16x8 vf[ND][2], vn[ND][2];
    if (kw < nt) vload(kw, vf);
#pragma unroll
    for (int x = 0; x < MT; ++x) {
      const int u = kw + x * KS;
      if (u < nt) {
        if (u + KS < nt) vload(u + KS, vn);
        f16x8 pf[2];
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv = __builtin_amdgcn_exp2f(sv[x][8 * f + e] - m_ref);
            l_i += pv;
            pf[f][e] = (f16)pv;
          }
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
          for (int n = 0; n < ND; ++n) mfma32(oacc[n], vf[n][f], pf[f]);
        if (u + KS < nt) {
#pragma unroll
          for (int n = 0; n < ND; ++n)
#pragma unroll
            for (int f = 0; f < 2; ++f) vf[n][f] = vn[n][f];
        }
      }
    }
  } else
  for (int u = kw; u < nt; u += KS) {
    const bool pre = u < np;
    const int t = pre ? u : t_lo + u - np;
    f16x8 vf[ND][2];
    vload(u, vf);
    f32x16 sacc[2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[x][r] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) mfma32(sacc[kk & 1], kf[kk], qf[kk]);
    if (u + KS < nt) kload(u + KS, kn);
    f32x16 s = sacc[0] + sacc[1];
    // key of register r: row 32 t + acc_row(r, lane) of its source; the lane
    // sees rows [k_lo, k_hi] of this source (branch-free selects)
    const int k_lo = pre ? 0 : s0;
    const int k_hi = pre ? P - 1 : (a.causal ? s0 + min(my_q, L - 1) : s0 + L - 1);
    const int kb = t * 32 + 4 * lgrp;
    float mb = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int k = kb + 8 * (r >> 2) + (r & 3);
      s[r] = ((k >= k_lo) & (k <= k_hi)) ? s[r] * a.sc : -INFINITY;
      mb = fmaxf(mb, s[r]);
    }
    mb = warp_max_xor(mb, 32);
    const float m_new = fmaxf(m_i, mb);
    const float m_ref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_i - m_ref);
    m_i = m_new;
    float p[16], ps = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = __builtin_amdgcn_exp2f(s[r] - m_ref);
      ps += p[r];
    }
    l_i = l_i * alpha + ps;
    // the running max moved for some query: rescale O (not on the wave's
    // first tile, where O is still zero)
    if (u != kw && __any(alpha != 1.f)) {
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;
    }
    f16x8 pf[2];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[f][e] = (f16)p[8 * f + e];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int n = 0; n < ND; ++n) mfma32(oacc[n], vf[n][f], pf[f]);
    if (u + KS < nt) {
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) kf[kk] = kn[kk];
    }
  }
  if constexpr (KS > 1) {
    // waves 1.. hand (m, l, O^T) to wave 0, lane-contiguous (no bank conflicts)
    constexpr int NV = 2 + ND * 16;
    __shared__ float red[KS - 1][NV][64];
    if (kw > 0) {
      red[kw - 1][0][lane] = m_i;
      red[kw - 1][1][lane] = l_i;
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[kw - 1][2 + n * 16 + r][lane] = oacc[n][r];
    }
    __syncthreads();
    if (kw > 0) return;
    float mx = m_i;
#pragma unroll
    for (int v = 0; v < KS - 1; ++v) mx = fmaxf(mx, red[v][0][lane]);
    const float mr = mx == -INFINITY ? 0.f : mx;   // wave 0 always saw key 0, so mx is finite
    const float f0 = __builtin_amdgcn_exp2f(m_i - mr);
    l_i *= f0;
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[n][r] *= f0;
#pragma unroll
    for (int v = 0; v < KS - 1; ++v) {
      const float fv = __builtin_amdgcn_exp2f(red[v][0][lane] - mr);
      l_i += fv * red[v][1][lane];
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] += fv * red[v][2 + n * 16 + r][lane];
    }
  }
  const float inv = 1.f / (l_i + __shfl_xor(l_i, 32, kWave));
  store_o<HD>(oacc, inv, a.o + ((size_t)(s0 + min(my_q, L - 1)) * a.Hq + head) * HD + 8 * lgrp, my_q < L);
}

// Staged variant of k_attn_h for key ranges that fit in LDS. A workgroup
// serves one kv head and a chunk of `qbw` 32-query blocks of one sequence,
// one wave per (query head of the group, query block). All waves first copy
// every key tile the chunk sees (its k rows and V^T rows for this kv head)
// from global memory straight into LDS (global_load_lds, 16 bytes a lane,
// all copies in flight at once), wait for them once, and then compute from
// LDS only: the chain of dependent global loads of the register-streaming
// kernel becomes one load latency per round. A round fills the LDS cap (64
// KB: two workgroups a CU), 4 tiles of head size 128 or 8 of 64; within it
// the softmax is two-pass (every tile's scores in registers, one maximum,
// then the probabilities and O, code specialised per tile count; masks only
// in the tiles that need them), and longer ranges carry the running maximum,
// sum and O from round to round. The arithmetic of k_attn_h (fp16 operands,
// fp32 scores and softmax in base 2, masks as selects) on the same global
// 32-token key tiles, but for the scale: one fma before exp2 here, a multiply
// and a subtract there (one rounding apart).
// LDS per tile: k rows [32][HD] then V^T rows [HD][32], 16-byte chunks
// placed by an XOR of the row so that the 16 lanes of a quarter-wave that
// read one chunk column of 16 rows hit 16 distinct 16-byte bank groups.
struct AttnSArgs {
  const f16 *qk, *vt, *pqk, *pvt;
  f16 *o;
  float sc;
  int ldq, T, P;
  int Hq, Hkv, rep;
  int causal;
  int qbw;             // 32-query blocks per workgroup
  int cu[kMaxSeqPerLaunch + 1];   // absolute token offsets
};

// slot of 16-byte chunk c of k row r (HD / 8 chunks a row), and of chunk c
// of V^T row r (4 chunks a row); each is its own inverse
template <int HD>
__device__ __forceinline__ int kslot(int r, int c) {
  if constexpr (HD == 128) return c ^ (r & 15);
  else return c ^ ((r >> 1) & 7);
}
__device__ __forceinline__ int vslot(int r, int c) { return c ^ ((r >> 2) & 3); }

constexpr int kAttnSCap = 64 * 1024;   // LDS bytes per workgroup: two workgroups a CU

// Where a wave's staged tiles come from and which keys its lane's query sees.
struct STile {
  const char *lb;      // LDS base
  int np, t_lo, P, s0, kq_hi;
  int kw_hi;           // the smallest kq_hi of the wave's lanes (wave-uniform)
  float sc;
  int lgrp;
};

// The N tiles of one wave in one staged round (LDS slots 0 .. N-1 hold key
// tiles ub .. ub+N-1 of its range), in three passes: the raw scores q.k of
// every tile (one MFMA chain per tile, all kept in registers; straight-line
// code, so the loads and MFMAs of different tiles overlap), then the mask --
// only in a tile that some query of the wave does not see whole, a
// wave-uniform test -- and one maximum per query, then the probabilities
// 2^(sc s - m) (one fma per score: sc > 0 scales the maximum exactly as it
// scales each score) and O. Across rounds the running maximum m_i (scaled),
// sum l_i and O carry over (rescaled when the maximum moves); a range of one
// round is plain two-pass.
template <int HD, int N>
__device__ __forceinline__ void s_tiles(const STile &st, int ub, const uint32_t (&ka)[HD / 16],
                                        const uint32_t (&va)[HD / 32][2], const f16x8 (&qf)[HD / 16],
                                        f32x16 (&oacc)[HD / 32], float &m_i, float &l_i) {
  constexpr int ND = HD / 32, NK = HD / 16, TB = 128 * HD;
  f32x16 sv[N];
#pragma unroll
  for (int x = 0; x < N; ++x) {
    const char *tb = st.lb + x * TB;
    f16x8 kf[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) kf[kk] = *(const f16x8 *)(tb + ka[kk]);
#pragma unroll
    for (int r = 0; r < 16; ++r) sv[x][r] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) mfma32(sv[x], kf[kk], qf[kk]);
  }
  float mb = -INFINITY;
#pragma unroll
  for (int x = 0; x < N; ++x) {
    const int u = ub + x;
    const bool pre = u < st.np;
    const int kt0 = pre ? u * 32 : (st.t_lo + u - st.np) * 32;   // the tile's first key
    const int k_lo = pre ? 0 : st.s0;
    if (kt0 < k_lo || kt0 + 31 > (pre ? st.P - 1 : st.kw_hi)) {    // wave-uniform
      const int k_hi = pre ? st.P - 1 : st.kq_hi;
      const int kb = kt0 + 4 * st.lgrp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int k = kb + 8 * (r >> 2) + (r & 3);
        sv[x][r] = ((k >= k_lo) & (k <= k_hi)) ? sv[x][r] : -INFINITY;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) mb = fmaxf(mb, sv[x][r]);
  }
  mb = warp_max_xor(mb, 32) * st.sc;
  // a query with no visible key yet (impossible in a range's first round,
  // which holds a key every query sees) exponentiates against 0: exact zeros
  const float m_new = fmaxf(m_i, mb);
  const float m_ref = m_new == -INFINITY ? 0.f : m_new;
  if (ub > 0) {                                // wave-uniform: rounds after the first
    const float alpha = __builtin_amdgcn_exp2f(m_i - m_ref);
    l_i *= alpha;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;
    }
  }
  m_i = m_new;
#pragma unroll
  for (int x = 0; x < N; ++x) {
    const char *tb = st.lb + x * TB;
    f16x8 vf[ND][2];
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int f = 0; f < 2; ++f) vf[n][f] = *(const f16x8 *)(tb + va[n][f]);
    f16x8 pf[2];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sv[x][8 * f + e], st.sc, -m_ref));
        l_i += p;
        pf[f][e] = (f16)p;
      }
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int n = 0; n < ND; ++n) mfma32(oacc[n], vf[n][f], pf[f]);
  }
}

// Grid: x = (chunk of the sequence, kv head), y = sequence; workgroups past a
// sequence's last chunk leave at once. NWV waves (4 or 8), each copying a
// fixed block of GPT / NWV copies of every tile: all k rows or all V^T rows,
// the same per-lane offsets for every tile. Registers are held to two waves
// per SIMD (two 4-wave workgroups, or one 8-wave workgroup, per CU). MR:
// the launch has ranges longer than one round (without it the round loop is
// compiled out, which leaves the one-round kernel fewer registers).
template <int HD, int NWV, bool MR>
__global__ __launch_bounds__(64 * NWV) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_attn_s(AttnSArgs a) {
  constexpr int ND = HD / 32, NK = HD / 16, NCH = HD / 8;
  constexpr int MT = kAttnSCap / (128 * HD);   // tiles that fit the LDS cap
  constexpr int KB = 64 * HD;                  // bytes of k rows (and of V^T rows) per tile
  constexpr int TB = 2 * KB;                   // bytes per staged tile
  constexpr int GPT = TB / 1024;               // 64-lane copies per tile
  extern __shared__ u32x4 lds[];
  const int lane = threadIdx.x & 63, lrow = lane & 31, lgrp = lane >> 5;
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int chunk = (int)blockIdx.x / a.Hkv, kvh = (int)blockIdx.x % a.Hkv;
  const int s0 = a.cu[blockIdx.y], L = a.cu[blockIdx.y + 1] - s0;
  const int qc0 = chunk * a.qbw * 32;          // first query of the chunk
  if (qc0 >= L) return;                        // the whole workgroup, before any barrier
  const int P = a.P, np = (P + 31) >> 5;
  const int t_lo = s0 >> 5;
  // key tiles of the chunk: the prefix's, then the batch tiles up to the last
  // key its last query sees
  const int kend_c = a.causal ? min(qc0 + a.qbw * 32, L) - 1 : L - 1;
  const int nt = np + ((s0 + kend_c) >> 5) - t_lo + 1;

  // this wave's query head and 32 queries
  const int head = kvh * a.rep + wv % a.rep;
  const int q0 = qc0 + (wv / a.rep) * 32;
  const bool live = q0 < L;                    // wave-uniform
  const int my_q = q0 + lrow;
  f16x8 qf[NK];
  if (live) {
    const f16 *qr = a.qk + (size_t)(s0 + min(my_q, L - 1)) * a.ldq + head * HD + lgrp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = *(const f16x8 *)(qr + kk * 16);
  }
  // Copy g of a tile (0 <= g < GPT) fills its 1 KB group g: groups below
  // GPT / 2 hold k rows (lane l: row 64 g / NCH + l / NCH, chunk slot l % NCH),
  // the rest V^T rows (lane l: row 16 g' + l / 4, chunk slot l % 4).
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  const uint32_t kcol = (uint32_t)((a.Hq + kvh) * HD) * 2u;
  const uint32_t ldq2 = (uint32_t)a.ldq * 2u;
  auto kcopy = [&](int u, int slot, int g) {
    const bool pre = u < np;
    const int rb = pre ? u * 32 : (t_lo + u - np) * 32;
    const int r = g * (64 / NCH) + lane / NCH;
    const int row = min(rb + r, pre ? P - 1 : a.T - 1);
    dma16(pre ? a.pqk : a.qk, (uint32_t)row * ldq2 + kcol + (uint32_t)kslot<HD>(r, lane % NCH) * 16u,
          lds0 + (uint32_t)(slot * TB + g * 1024));
  };
  // V^T: the chunk slot of lane l is the same for every group
  const uint32_t voff = (uint32_t)((lane >> 2) * 64 + (((lane & 3) ^ ((lane >> 4) & 3)) * 16));
  auto vcopy = [&](int u, int slot, int g) {
    const bool pre = u < np;
    const int t = pre ? u : t_lo + u - np;
    const char *vb = (const char *)(pre ? a.pvt : a.vt) + ((size_t)(t * a.Hkv + kvh) * HD) * 64 + g * 1024;
    dma16(vb, voff, lds0 + (uint32_t)(slot * TB + KB + g * 1024));
  };
  constexpr int CPW = GPT / NWV;               // copies per wave and tile
  static_assert((NWV == 4 || NWV == 8) && GPT % NWV == 0 && (GPT / 2) % CPW == 0,
                "a wave's block is all k or all V^T");
  static_assert(MT * CPW + NK < 64, "vmcnt range: every copy and q load in flight at once");
  const int c0 = wv * CPW;
  // this wave's block of the copies of key tiles [ub, ue) into slots 0 ..
  auto copies = [&](int ub, int ue) {
    if (c0 < GPT / 2) {
      for (int u = ub; u < ue; ++u)
#pragma unroll
        for (int i = 0; i < CPW; ++i) kcopy(u, u - ub, c0 + i);
    } else {
      for (int u = ub; u < ue; ++u)
#pragma unroll
        for (int i = 0; i < CPW; ++i) vcopy(u, u - ub, c0 - GPT / 2 + i);
    }
  };
  // Rounds of at most MT tiles (one round when the range fits the cap). The
  // first round's copies go out before anything else; its fragment offsets
  // are computed while they land.
  const int nrounds = (nt + MT - 1) / MT;      // workgroup-uniform
  copies(0, min(nt, MT));

  const char *lb = (const char *)lds;
  uint32_t ka[NK], va[ND][2];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) ka[kk] = (uint32_t)(lrow * NCH + kslot<HD>(lrow, 2 * kk + lgrp)) * 16u;
#pragma unroll
  for (int n = 0; n < ND; ++n)
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int r = n * 32 + lrow;
      va[n][f] = (uint32_t)KB + (uint32_t)(r * 4 + vslot(r, 2 * f + lgrp)) * 16u;
    }
  // tiles this wave sees, and the keys its lane's query sees in each source
  const int kend = a.causal ? min(q0 + 31, L - 1) : L - 1;
  const int ntw = np + ((s0 + kend) >> 5) - t_lo + 1;
  const int kq_hi = a.causal ? s0 + min(my_q, L - 1) : s0 + L - 1;
  const int kw_hi = a.causal ? s0 + min(q0, L - 1) : s0 + L - 1;
  const STile st{lb, np, t_lo, P, s0, kq_hi, kw_hi, a.sc, lgrp};
  f32x16 oacc[ND];
#pragma unroll
  for (int n = 0; n < ND; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[n][r] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;
  // the round's tiles of this wave's own range, in straight-line code per
  // count (waves with no queries, or whose range ended, skip)
#define MTE_S_ROUND(UB_, UE_)                                                        \
  switch (live ? min(ntw, (UE_)) - (UB_) : 0) {                                     \
    case 1: s_tiles<HD, 1>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break;           \
    case 2: if constexpr (MT >= 2) s_tiles<HD, 2>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 3: if constexpr (MT >= 3) s_tiles<HD, 3>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 4: if constexpr (MT >= 4) s_tiles<HD, 4>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 5: if constexpr (MT >= 5) s_tiles<HD, 5>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 6: if constexpr (MT >= 6) s_tiles<HD, 6>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 7: if constexpr (MT >= 7) s_tiles<HD, 7>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    case 8: if constexpr (MT >= 8) s_tiles<HD, 8>(st, (UB_), ka, va, qf, oacc, m_i, l_i); break; \
    default: break;                                                                 \
  }
  wait_vm<0>();
  __syncthreads();
  MTE_S_ROUND(0, min(nt, MT))
  // further rounds: every wave is done with the slots before they are refilled
  if constexpr (MR) {
    for (int rd = 1; rd < nrounds; ++rd) {
      const int ub = rd * MT, ue = min(nt, ub + MT);
      __syncthreads();
      copies(ub, ue);
      wait_vm<0>();
      __syncthreads();
      MTE_S_ROUND(ub, ue)
    }
  }
#undef MTE_S_ROUND
  if (!live) return;
  const float inv = 1.f / (l_i + __shfl_xor(l_i, 32, kWave));
  store_o<HD>(oacc, inv, a.o + ((size_t)(s0 + min(my_q, L - 1)) * a.Hq + head) * HD + 8 * lgrp, my_q < L);
}

// Launches k_attn_s (hipErrorNotSupported, launching nothing, when a
// workgroup would not have 4 or 8 waves).
static hipError_t launch_attention_s(const AttnSArgs &base, const int32_t *cu, int batch, int d, int qbw,
                                     hipStream_t s) {
  constexpr int kCap = kAttnSCap;
  if (qbw < 1) return hipErrorInvalidValue;
  if (base.rep * qbw != 4 && base.rep * qbw != 8) return hipErrorNotSupported;   // 4 or 8 waves
  const int tb = 128 * d;
  const int np = (base.P + 31) / 32;
  AttnSArgs a = base;
  a.qbw = qbw;
  const int nwv = a.rep * qbw;
  for (int first = 0; first < batch; first += kMaxSeqPerLaunch) {
    const int n = batch - first < kMaxSeqPerLaunch ? batch - first : kMaxSeqPerLaunch;
    int nch_max = 0, nt_max = 0;
    for (int i = 0; i < n; ++i) {
      const int s0 = cu[first + i], L = cu[first + i + 1] - s0;
      a.cu[i] = s0;
      nch_max = std::max(nch_max, (L + 32 * qbw - 1) / (32 * qbw));
      if (L > 0) nt_max = std::max(nt_max, np + ((s0 + L - 1) >> 5) - (s0 >> 5) + 1);
    }
    a.cu[n] = cu[first + n];
    if (nch_max == 0) continue;
    const int lds = std::min(nt_max * tb, kCap);   // one round's tiles
    dim3 grid(nch_max * a.Hkv, n), blk(64 * nwv);
#define MTE_ATTN_S(HD_, NWV_, MR_)                                                                 \
    {                                                                                              \
      auto kern = k_attn_s<HD_, NWV_, MR_>;                                                        \
      static const hipError_t attr =                                                               \
          hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kCap); \
      if (attr != hipSuccess) return attr;                                                         \
      hipLaunchKernelGGL(kern, grid, blk, lds, s, a);                                              \
    }
    const bool mr = nt_max * tb > kCap;         // some range needs more than one round
    if (d == 128 && nwv == 4) { if (mr) MTE_ATTN_S(128, 4, true) else MTE_ATTN_S(128, 4, false) }
    else if (d == 128) { if (mr) MTE_ATTN_S(128, 8, true) else MTE_ATTN_S(128, 8, false) }
    else if (nwv == 4) { if (mr) MTE_ATTN_S(64, 4, true) else MTE_ATTN_S(64, 4, false) }
    else { if (mr) MTE_ATTN_S(64, 8, true) else MTE_ATTN_S(64, 8, false) }
#undef MTE_ATTN_S
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attention_h(const f16 *qk, const f16 *vt, const f16 *prefix, const f16 *pvt, int P, f16 *o,
                              float sc, const int32_t *cu, int batch, int T, int Hq, int Hkv, int d, int causal,
                              hipStream_t s, int ks, int qbw) {
  constexpr int WPB = 2;      // work items (waves) per workgroup without key split
  if (P < 0 || (P > 0 && (!prefix || !pvt)) || (d != 64 && d != 128) || Hq % Hkv || !qk || !vt || !o)
    return hipErrorInvalidValue;
  // the staged kernel addresses k rows and V^T tiles by 32-bit byte offsets
  const bool small = (uint64_t)std::max(T, P) * (uint64_t)(Hq + Hkv) * d * 2 < (1ull << 32);
  if (qbw >= 0 && ks == 0 && small) {
    AttnSArgs b;
    b.qk = qk;
    b.vt = vt;
    b.pqk = prefix;
    b.pvt = pvt;
    b.o = o;
    b.sc = sc;
    b.ldq = (Hq + Hkv) * d;
    b.T = T;
    b.P = P;
    b.Hq = Hq;
    b.Hkv = Hkv;
    b.rep = Hq / Hkv;
    b.causal = causal ? 1 : 0;
    // Default chunk: 2 query blocks of both query heads per kv head (4 waves)
    // for causal attention with two query heads per kv head, 8 query blocks
    // of one head (8 waves) for the bidirectional vision tower. Measured in
    // isolation, 16 x 96 tokens: 10.1 / 8.0 / 9.1 us with 1 / 2 / 3 blocks
    // (10.3 streaming), 16 x 128: 12.5 / 10.0 / 11.0 with 1 / 2 / 4 (12.9);
    // one frame 6.8 (6.7 streaming, two-wave key split); 16 images of 256
    // patches: 25.0 / 14.0 / 12.9 us with 2 / 4 / 8 blocks (19.5 streaming).
    const int q = qbw > 0 ? qbw : std::max(1, (causal ? 4 : 8) / b.rep);
    const hipError_t e = launch_attention_s(b, cu, batch, d, q, s);
    if (e != hipErrorNotSupported || qbw > 0) return e;
  }
  AttnHArgs a;
  a.qk = qk;
  a.vt = vt;
  a.pqk = prefix;
  a.pvt = pvt;
  a.o = o;
  a.sc = sc;
  a.ldq = (Hq + Hkv) * d;
  a.T = T;
  a.P = P;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.rep = Hq / Hkv;
  a.causal = causal ? 1 : 0;
  for (int first = 0; first < batch; first += kMaxSeqPerLaunch) {
    const int n = batch - first < kMaxSeqPerLaunch ? batch - first : kMaxSeqPerLaunch;
    a.n_seq = n;
    int blocks = 0;
    for (int i = 0; i < n; ++i) {
      a.cu[i] = cu[first + i];
      a.blk0[i] = blocks;
      blocks += (cu[first + i + 1] - cu[first + i] + 31) / 32;
    }
    a.cu[n] = cu[first + n];
    a.blk0[n] = blocks;
    a.n_items = blocks * Hq;
    if (a.n_items == 0) continue;
    // key tiles of the longest item: the prefix's, then the batch tiles the
    // sequence touches (it may start inside a tile)
    int nt_max = 0;
    for (int i = 0; i < n; ++i) {
      const int s0 = cu[first + i], e0 = cu[first + i + 1] - 1;
      nt_max = std::max(nt_max, (P + 31) / 32 + (e0 >> 5) - (s0 >> 5) + 1);
    }
    // Few items (one or two frames) leave most of the chip idle and each
    // item's tile steps in series: split every item's key tiles over 2 waves
    // (measured: one 96-token frame 7.3 us with 1 wave per item, 6.7 with 2,
    // 6.9 with 4; 16 frames 10.3 us with 1 or 2, 14.0 with 4).
    const int k = ks > 0 ? ks : (a.n_items < 256 ? 2 : 1);
    // at most 4 tiles per wave: the two-pass variant
    const bool two = (nt_max + k - 1) / k <= 4;
#define MTE_ATTN_H(KS_, WPB_)                                                                          \
    {                                                                                                  \
      dim3 grid_((a.n_items + WPB_ - 1) / WPB_), blk_(64 * WPB_ * KS_);                                \
      if (d == 128 && two) hipLaunchKernelGGL((k_attn_h<128, WPB_, KS_, 4>), grid_, blk_, 0, s, a);    \
      else if (d == 128) hipLaunchKernelGGL((k_attn_h<128, WPB_, KS_, 0>), grid_, blk_, 0, s, a);      \
      else if (two) hipLaunchKernelGGL((k_attn_h<64, WPB_, KS_, 4>), grid_, blk_, 0, s, a);            \
      else hipLaunchKernelGGL((k_attn_h<64, WPB_, KS_, 0>), grid_, blk_, 0, s, a);                     \
    }
    if (k == 4) MTE_ATTN_H(4, 1)
    else if (k == 2) MTE_ATTN_H(2, 1)
    else MTE_ATTN_H(1, WPB)
#undef MTE_ATTN_H
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mte
