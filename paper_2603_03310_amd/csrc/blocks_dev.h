// Device bodies of the block scoring and selection stages, shared by the
// per-stage kernels (blocks.hip, prologue.hip) and the fused step kernels
// (step.hip).
//
// Block entropic contribution (Section 3.2 of the paper): I_b is the
// attention-weighted surprisal of block b's tokens.  Weights come from the
// current query against each block's mean key (one summary per block and KV
// head), surprisal is -ln of the same weight, and scores are averaged over
// query heads:
//   z_bh = scale <q_h, kbar_b,g>,   L_h = ln sum_b n_b e^{z_bh}
//   I_b  = (1/H_q) sum_h e^{z_bh + ln n_b - L_h} (L_h - z_bh)
// The kept set is {b : I_b >= theta} with theta the k-th largest score and k
// the entropy-driven budget with its floor and minimum (Sections 3.2, 3.3, 5).
#pragma once

#include "ent_internal.h"

#include <math.h>

namespace ent {
namespace {

template <typename T>
__device__ __forceinline__ float load_elem(const T* p);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// ---------------------------------------------------------------------------
// Scoring.  Both scoring kernels write the block logits
//   z_bh = scale <q_h, kbar_b,g(h)>     zbuf [B, MAXB, H_q]
// and, per chunk of blocks and head, the log-sum-exp partial (max, sum) of
// l_bh = z_bh + ln n_b over the chunk's blocks.
//
// bf16 queries (MFMA).  A wave takes a tile of 16 blocks and one KV head.
// For each KV head g the tile's logits are one small contraction
//   Z[16 blocks x 16] = Kbar_g[16 x d] . Q_g^T[d x 16]   (columns: the G query
// heads of g, zero-padded), on v_mfma_f32_16x16x32_bf16.  The fp32 summaries
// are split exactly into three bf16 parts (hi + mid + lo), so three MFMAs per
// k-step give the fp32 dot product of exact bf16 products.  Both operands
// come straight from global memory (the queries are cache-resident).
//
// fp32 queries (VALU).  A workgroup of 4 waves takes 16 blocks, 4 per wave;
// a block's summary is read as NP passes of 256 floats, one float4 per lane
// per pass; each lane forms G partial dot products over its 4 dims and a
// halving butterfly reduces them over the d/4 lanes of its KV head.
// ---------------------------------------------------------------------------
constexpr int kScoreThreads = 256;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kMfmaChunk = 16;                 // blocks per MFMA scoring workgroup
constexpr int kValuChunk = 16;                 // blocks per VALU scoring workgroup
constexpr int kValuPerWave = kValuChunk / kScoreWaves;
static_assert(kValuChunk == kMfmaChunk, "both scoring paths write partials per 16-block tile");

typedef float sf32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

// Per-head log-sum-exp partial of l = z + ln n over the chunk's nblk blocks
// (z tile in LDS, row stride Hq).
__device__ __forceinline__ void chunk_lse(const float* zt, int nblk, int Hq, int j_lo, int nb,
                                          int N, float* lp_chunk) {
  const float ln_last = logf(static_cast<float>(N - kBlock * (nb - 1)));
  const float ln_full = logf(static_cast<float>(kBlock));
  for (int h = threadIdx.x; h < Hq; h += blockDim.x) {
    float m = -INFINITY;
    for (int i = 0; i < nblk; ++i) {
      const float lnn = (j_lo + i == nb - 1) ? ln_last : ln_full;
      m = fmaxf(m, zt[i * Hq + h] + lnn);
    }
    float s = 0.f;
    for (int i = 0; i < nblk; ++i) {
      const float lnn = (j_lo + i == nb - 1) ? ln_last : ln_full;
      s += expf(zt[i * Hq + h] + lnn - m);
    }
    lp_chunk[h * 2 + 0] = m;
    lp_chunk[h * 2 + 1] = s;
  }
}

// One scoring item: a tile of kMfmaChunk = 16 blocks of sequence b (tile
// ch) and one KV head g, by one wave: the summaries (16 blocks x d fp32),
// loaded by the prologue's score_job, are reduced with score_head_compute.
constexpr int kScoreSlots = 8;          // float4 slots per lane (d <= 128)

// Table entry of tile row r16 (lane & 15), read before the context length
// is known (-1 past the row); score_tile_check validates it once nb is.
__device__ __forceinline__ int score_tile_entry(const int* __restrict__ tables, int b, int ch,
                                                int MAXB) {
  const int j = ch * kMfmaChunk + (threadIdx.x & 15);
  return j < MAXB ? tables[static_cast<long long>(b) * MAXB + j] : -1;
}

// Physical block of tile row r16 from its table entry, validated; 0 for rows
// past the sequence's nb blocks.
__device__ __forceinline__ int score_tile_check(int p, int ch, int nb, int P, unsigned* flags) {
  const int j = ch * kMfmaChunk + (threadIdx.x & 15);
  if (j >= nb) return 0;
  if (p < 0 || p >= P) {
    raise_flag(flags, ENT_DEV_BAD_TABLE);
    p = 0;
  }
  return p;
}


typedef float sf32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 sbf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 sbf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));

// Exact three-way split x = hi + mid + lo of 8 floats into bf16 parts, each
// part rounded to nearest from the remainder of the previous ones: the
// remainders are exact in fp32 (they are differences of nearby floats) and
// the last one has at most 8 significant bits, so lo is exact in bf16.
__device__ __forceinline__ void split3(const float4& x0, const float4& x1, sbf16x8_t& hi,
                                       sbf16x8_t& mid, sbf16x8_t& lo) {
  const sf32x2_t v[4] = {{x0.x, x0.y}, {x0.z, x0.w}, {x1.x, x1.y}, {x1.z, x1.w}};
  sbf16x2_t h[4], m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = __builtin_convertvector(v[i], sbf16x2_t);
    const sf32x2_t r = v[i] - __builtin_convertvector(h[i], sf32x2_t);
    m[i] = __builtin_convertvector(r, sbf16x2_t);
    const sf32x2_t r2 = r - __builtin_convertvector(m[i], sf32x2_t);
    l[i] = __builtin_convertvector(r2, sbf16x2_t);
  }
  hi = sbf16x8_t{h[0].x, h[0].y, h[1].x, h[1].y, h[2].x, h[2].y, h[3].x, h[3].y};
  mid = sbf16x8_t{m[0].x, m[0].y, m[1].x, m[1].y, m[2].x, m[2].y, m[3].x, m[3].y};
  lo = sbf16x8_t{l[0].x, l[0].y, l[1].x, l[1].y, l[2].x, l[2].y, l[3].x, l[3].y};
}

// Block logits z of head g's query heads (written to zbuf) and each query
// head's log-sum-exp partial (max, sum) of z + ln n_b over the tile
// (lse_part).  z[16 blocks x 16] = Kbar_g[16 x d] Q_g^T[d x 16] on
// v_mfma_f32_16x16x32_bf16 (columns: the G query heads of g, zero-padded),
// three MFMAs per k-step over the exact split of the fp32 summaries, so
// every product is exact and only the fp32 accumulation rounds.  K-slot
// (gq, e) of step ks is dim 32 ks + 4 gq + e for e < 4 and
// 32 ks + 16 + 4 gq + (e - 4) for e >= 4, in both operands.
// The B operand of head g's query heads for lane (r16, gq): slot 2 ks holds
// dims 32 ks + 4 gq .. +3, slot 2 ks + 1 dims 32 ks + 16 + 4 gq .. +3.
// Every load is issued at once, from a valid head's address (the padding
// columns r16 >= G are zeroed where they are used, so nothing waits here).
template <int D>
__device__ __forceinline__ void score_q_load(const uint16_t* __restrict__ q, int b, int g, int Hkv,
                                             int G, uint2 (&qv)[D / 16]) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, gq = lane >> 4;
  const uint16_t* qh =
      q + (static_cast<long long>(b) * Hkv * G + g * G + min(r16, G - 1)) * D + gq * 4;
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    qv[2 * ks] = *reinterpret_cast<const uint2*>(qh + 32 * ks);
    qv[2 * ks + 1] = *reinterpret_cast<const uint2*>(qh + 32 * ks + 16);
  }
}

// With store false (G <= 8 only) the block logits are not written: they are
// returned packed two per lane for store_held_z to write later (lanes r16 < 8
// keep blocks 4 gq, 4 gq + 1 of head r16; lanes r16 >= 8 take blocks
// 4 gq + 2, 4 gq + 3 of head r16 - 8, from the padding columns' lanes).
template <int D>
__device__ __forceinline__ sf32x2_t score_head_compute(
    const uint2 (&qv)[D / 16], const float4 (&buf)[kScoreSlots],
    float* __restrict__ zbuf, float* __restrict__ lse_part, int b, int ch, int g, int N, int nb,
    int Hkv, int G, int MAXB, int nch_max, float scale, bool store) {
  constexpr int KS = D / 32;
  const int Hq = Hkv * G;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, gq = lane >> 4;
  const int jt = ch * kMfmaChunk;
  sf32x4_t acc = sf32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const uint2 zero = make_uint2(0u, 0u);
    const uint2 q0 = r16 < G ? qv[2 * ks] : zero, q1 = r16 < G ? qv[2 * ks + 1] : zero;
    sbf16x8_t hi, mid, lo;
    split3(buf[2 * ks], buf[2 * ks + 1], hi, mid, lo);
    const sbf16x8_t bq = __builtin_bit_cast(sbf16x8_t, make_uint4(q0.x, q0.y, q1.x, q1.y));
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, bq, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(mid, bq, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, bq, acc, 0, 0, 0);
  }
  // acc[e]: block jt + 4 gq + e, query head g G + r16 (columns r16 >= G are padding).
  const float ln_last = logf(static_cast<float>(N - kBlock * (nb - 1)));
  const float ln_full = logf(static_cast<float>(kBlock));
  float* zrow = zbuf + (static_cast<long long>(b) * MAXB + jt) * Hq;
  float l[4], zv[4];
  float m = -INFINITY;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = jt + 4 * gq + e;
    const float z = acc[e] * scale;
    zv[e] = z;
    const bool ok = j < nb;
    if (store && ok && r16 < G) zrow[(4 * gq + e) * Hq + g * G + r16] = z;
    l[e] = ok ? z + ((j == nb - 1) ? ln_last : ln_full) : -INFINITY;
    m = fmaxf(m, l[e]);
  }
  m = fmaxf(m, __shfl_xor(m, 16));
  m = fmaxf(m, __shfl_xor(m, 32));
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) sum += (l[e] == -INFINITY) ? 0.f : expf(l[e] - m);
  sum += __shfl_xor(sum, 16);
  sum += __shfl_xor(sum, 32);
  if (gq == 0 && r16 < G) {
    float* lp = lse_part + ((static_cast<long long>(b) * nch_max + ch) * Hq + g * G + r16) * 2;
    lp[0] = m;
    lp[1] = sum;
  }
  if (store) return sf32x2_t{0.f, 0.f};
  const int src = r16 >= 8 ? lane - 8 : lane;
  const float z2 = __shfl(zv[2], src), z3 = __shfl(zv[3], src);
  return r16 < 8 ? sf32x2_t{zv[0], zv[1]} : sf32x2_t{z2, z3};
}

// Writes the block logits that score_head_compute returned packed (tile ch
// of sequence b with nb blocks, KV head g; G <= 8).
__device__ __forceinline__ void store_held_z(sf32x2_t v, float* __restrict__ zbuf, int b, int ch,
                                             int g, int nb, int Hkv, int G, int MAXB) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, gq = lane >> 4;
  const int h = r16 & 7, e0 = 4 * gq + (r16 < 8 ? 0 : 2);
  if (h >= G) return;
  const int Hq = Hkv * G;
  const int jt = ch * kMfmaChunk;
  float* zrow = zbuf + (static_cast<long long>(b) * MAXB + jt) * Hq + g * G + h;
  if (jt + e0 < nb) zrow[e0 * Hq] = v.x;
  if (jt + e0 + 1 < nb) zrow[(e0 + 1) * Hq] = v.y;
}

template <int G, int L>
__device__ __forceinline__ float reduce_heads(float (&a)[G], int li) {
#pragma unroll
  for (int n = G, s = L / 2; n > 1; n >>= 1, s >>= 1) {
    const bool up = (li & s) != 0;
#pragma unroll
    for (int i = 0; i < n / 2; ++i) {
      const float keep = up ? a[i + n / 2] : a[i];
      const float send = up ? a[i] : a[i + n / 2];
      a[i] = keep + __shfl_xor(send, s);
    }
  }
  float v = a[0];
#pragma unroll
  for (int s = L / (2 * G); s >= 1; s >>= 1) v += __shfl_xor(v, s);
  return v;
}

// smem: q [Hq][D] fp32, then z tile [kValuChunk][Hq].
template <int D, int G>
__device__ __forceinline__ void score_valu_body(
    const float* __restrict__ q, const float* __restrict__ ksum, const int* __restrict__ tables,
    const int* __restrict__ ctx_lens, float* __restrict__ zbuf, float* __restrict__ lse_part,
    int Hkv, int MAXB, int P, int nch_max, float scale, unsigned* flags, int ch, int b,
    float* smem) {
  constexpr int L = D / 4;
  static_assert(G <= L, "heads per KV head exceed the lane group");
  const int Hq = Hkv * G;
  float* qs = smem;
  float* zt = smem + Hq * D;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int li = lane % L;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;    // flagged by the selection kernel
  const int nb = (N + kBlock - 1) / kBlock;
  const int j_lo = ch * kValuChunk;
  if (j_lo >= nb) return;
  const int nblk = min(kValuChunk, nb - j_lo);
  const int jw = j_lo + wave * kValuPerWave;
  const int nmine = max(0, min(kValuPerWave, nb - jw));
  int my_p = 0;
  if (lane < nmine) {
    my_p = tables[static_cast<long long>(b) * MAXB + jw + lane];
    if (my_p < 0 || my_p >= P) {
      raise_flag(flags, ENT_DEV_BAD_TABLE);
      my_p = 0;
    }
  }
  for (int e = t; e < Hq * D; e += kScoreThreads) qs[e] = q[static_cast<long long>(b) * Hq * D + e];
  __syncthreads();
  const int nfl = Hkv * D;
  const int np = (nfl + 255) >> 8;
  for (int blk = 0; blk < nmine; ++blk) {
    const int p = __shfl(my_p, blk);
    for (int k = 0; k < np; ++k) {
      const int f = 256 * k + 4 * lane;
      const bool gv = f < nfl;
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f);
      if (gv) kv = *reinterpret_cast<const float4*>(ksum + static_cast<long long>(p) * nfl + f);
      const int g = f / D, dd = f % D;
      float a[G];
#pragma unroll
      for (int r = 0; r < G; ++r) {
        float4 qq = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gv) qq = *reinterpret_cast<const float4*>(qs + (g * G + r) * D + dd);
        a[r] = qq.x * kv.x + qq.y * kv.y + qq.z * kv.z + qq.w * kv.w;
      }
      const float z = reduce_heads<G, L>(a, li) * scale;
      if (gv && (li % (L / G)) == 0) zt[(wave * kValuPerWave + blk) * Hq + g * G + li / (L / G)] = z;
    }
  }
  __syncthreads();
  float* zrow = zbuf + (static_cast<long long>(b) * MAXB + j_lo) * Hq;
  for (int e = t; e < nblk * Hq; e += kScoreThreads) zrow[e] = zt[e];
  chunk_lse(zt, nblk, Hq, j_lo, nb, N, lse_part + (static_cast<long long>(b) * nch_max + ch) * Hq * 2);
}

__device__ __forceinline__ unsigned float_key(float f) {
  const unsigned u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Budget k in float32, operation by operation (no contraction), so that the
// integer matches a float32 evaluation of the same formula elsewhere: the
// kept fraction from the guarded entropy, bounded below by the previous
// step's fraction minus dkappa (kprev NaN: no previous step), then
// k = min(nb, max(min(B_min, nb), ceil(kappa nb))).  kappa_used (nullable)
// receives the fraction.
__device__ __forceinline__ int keep_budget(float h, int nb, const Budget& bu, float kprev,
                                           float* kappa_used = nullptr) {
  // Plain operators under this pragma: the _rn intrinsics are header
  // functions whose bodies the pragma does not reach, and after inlining the
  // compiler would fuse kappa_min + (1 - kappa_min) u into one multiply-add.
#pragma clang fp contract(off)
  if (nb <= 0) return 0;
  const float hg = fmaxf(h + bu.eps_h, bu.h_min);
  float u = __fdiv_rn(hg - bu.h_min, bu.log_v - bu.h_min);
  u = fminf(fmaxf(u, 0.f), 1.f);
  const float span = 1.f - bu.kappa_min;
  const float grow = span * u;
  float kappa = bu.kappa_min + grow;
  if (!isnan(kprev)) kappa = fmaxf(kappa, kprev - bu.dkappa);
  if (kappa_used) *kappa_used = kappa;
  const float kn = kappa * static_cast<float>(nb);
  const int k = static_cast<int>(ceilf(kn));
  return min(nb, max(min(bu.b_min, nb), k));
}

// The previous step's kept fraction of sequence b (NaN when there is none
// or no state array).
__device__ __forceinline__ float budget_prev(const Budget& bu, int b) {
  return bu.kappa ? bu.kappa[b] : NAN;
}

// Records the kept fraction of a sequence with blocks (first thread).
__device__ __forceinline__ void budget_record(const Budget& bu, int b, float kappa) {
  if (bu.kappa && threadIdx.x == 0) bu.kappa[b] = kappa;
}

// Kept set of one sequence.  Three steps:
//  A. L_h = ln sum_b n_b e^{z_bh}, merged from the scoring pass's per-tile
//     partials (one workgroup per sequence);
//  B. I_b = (1/H_q) sum_h e^{z_bh + ln n_b - L_h} (L_h - z_bh) for every
//     block, H_q / 4 lanes per block (block_score_body);
//  C. budget k from the entropy, the k-th largest score by an 8-bit radix
//     select over the bits in which the scores differ, and ascending
//     compaction of {b : I_b >= theta} with wave ballots.
// When the block tables are short enough for the registers
// (select_one_launch), one workgroup per sequence runs all three; otherwise
// (the long-table forms) B runs over the whole chip, so long sequences
// spread their exponentials: the per-stage entry point in three launches
// (per-sequence A, B per 64 blocks, per-sequence C), the fused step in one
// or two (A and B together per tile of 256 blocks, lse_block_score_body,
// and C on the last of a sequence's workgroups to finish, or in a launch of
// its own when that would lower the tile launch's residency or its grid is
// many rounds of it).
// All forms perform the same arithmetic in the same order, so their results
// are identical.
constexpr int kRowThreads = 256;          // threads of the chip-wide block-score launch
constexpr int kTileBlocks = 64;           // blocks per scoring workgroup of step B
constexpr int kSelThreads = 512;          // step C (and the one-launch form)
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelMaxBlocks = 2048;       // block-table width of the one-launch form, at most (LDS)

// Step A's fold of the per-tile partials (max, sum) of head h into L_h is
// defined over kFoldThreads virtual threads, VPH = kFoldThreads / H_q per
// head: virtual thread (h, v) folds tiles v, v + VPH, v + 2 VPH, ... (their
// maximum first, then the rescaled sums: independent loads, no serial
// rescaling chain), and the VPH partials of head h are then merged by a
// fixed pairwise tree.  Launches of any size evaluate exactly this.
constexpr int kFoldThreads = 512;

// The fold of virtual thread vt (head vt % H_q) over the nch tiles.  Up to
// kFoldRegs tiles per virtual thread are loaded at once into registers; past
// that the two passes stream them (same arithmetic).
constexpr int kFoldRegs = 16;
__device__ __forceinline__ void lse_fold_vthread(const float* __restrict__ lse_part, int Hq,
                                                 int nch, int nch_max, int b, int vt, float& m,
                                                 float& sum) {
  const int vph = kFoldThreads / Hq;
  m = -INFINITY;
  sum = 0.f;
  if (vt >= vph * Hq) return;
  const int h = vt % Hq;
  const float* lp = lse_part + (static_cast<long long>(b) * nch_max * Hq + h) * 2;
  const int c0 = vt / Hq;
  const int n = c0 < nch ? (nch - c0 + vph - 1) / vph : 0;     // tiles of this virtual thread
  if (n <= kFoldRegs) {
    float2 x[kFoldRegs];
#pragma unroll
    for (int u = 0; u < kFoldRegs; ++u)
      x[u] = u < n ? *reinterpret_cast<const float2*>(lp + static_cast<long long>(c0 + u * vph) * Hq * 2)
                   : make_float2(-INFINITY, 0.f);
#pragma unroll
    for (int u = 0; u < kFoldRegs; ++u) m = fmaxf(m, x[u].x);
    if (m != -INFINITY)
#pragma unroll
      for (int u = 0; u < kFoldRegs; ++u)
        if (u < n) sum += x[u].y * expf(x[u].x - m);
    return;
  }
  for (int c = c0; c < nch; c += vph) m = fmaxf(m, lp[static_cast<long long>(c) * Hq * 2]);
  if (m != -INFINITY)
    for (int c = c0; c < nch; c += vph) {
      const float mc = lp[static_cast<long long>(c) * Hq * 2];
      sum += lp[static_cast<long long>(c) * Hq * 2 + 1] * expf(mc - m);
    }
}

// The merge of each head's VPH partials (s_pm, s_ps indexed by virtual
// thread v H_q + h), as a fixed pairwise tree: while n > 1 partials remain
// (n = VPH at first), partial v < n - h takes in partial v + h, in place,
// with h = ceil(n / 2), and n becomes h (for a power of two, the strides
// VPH / 2, VPH / 4, ..., 1).  Every thread of the workgroup must call it (it
// holds the barriers); afterwards L_h = s_pm[h] + ln s_ps[h] (lse_merged).
__device__ __forceinline__ void lse_merge_tree(float* s_pm, float* s_ps, int Hq) {
  for (int n = kFoldThreads / Hq; n > 1;) {
    const int st = (n + 1) >> 1;
    for (int i = threadIdx.x; i < (n - st) * Hq; i += blockDim.x) {
      const float m1 = s_pm[i], s1 = s_ps[i];
      const float m2 = s_pm[i + st * Hq], s2 = s_ps[i + st * Hq];
      if (m2 == -INFINITY) continue;
      if (m1 == -INFINITY) {
        s_pm[i] = m2;
        s_ps[i] = s2;
        continue;
      }
      const float mn = fmaxf(m1, m2);
      s_pm[i] = mn;
      s_ps[i] = s1 * expf(m1 - mn) + s2 * expf(m2 - mn);
    }
    __syncthreads();
    n = st;
  }
}

__device__ __forceinline__ float lse_merged(const float* s_pm, const float* s_ps, int h) {
  return s_pm[h] == -INFINITY ? -INFINITY : s_pm[h] + logf(s_ps[h]);
}

// Step A for sequence b (kFoldThreads threads: one virtual thread each):
// writes L_h to Lout[h] (-inf for an empty or invalid sequence); every thread
// of the workgroup must call it; Lout may be global or LDS memory; s_pm,
// s_ps: LDS [kFoldThreads].
__device__ __forceinline__ void lse_merge_body(const float* __restrict__ lse_part,
                                               const int* __restrict__ ctx_lens, float* Lout,
                                               int Hq, int MAXB, int nch_max, int b, float* s_pm,
                                               float* s_ps) {
  const int t = threadIdx.x;
  const int N = ctx_lens[b];
  const int nb = (N >= 0 && N <= MAXB * kBlock) ? (N + kBlock - 1) / kBlock : 0;
  const int nch = (nb + kMfmaChunk - 1) / kMfmaChunk;
  if (t < kFoldThreads) lse_fold_vthread(lse_part, Hq, nch, nch_max, b, t, s_pm[t], s_ps[t]);
  __syncthreads();
  lse_merge_tree(s_pm, s_ps, Hq);
  if (t < Hq) Lout[t] = lse_merged(s_pm, s_ps, t);
}

// Step B's sum over query heads.  A block's H_q heads are split between
// LPB lanes of HPLN = H_q / LPB consecutive heads each: when H_q / 4 is a
// power of two, LPB = min(4, H_q / 4) and a lane's block logits are HPLN / 4
// 16-byte loads (a wave reads whole spans of the block-logit rows);
// otherwise one lane takes all H_q heads.  A lane adds its heads' terms in
// head order, then the LPB lanes add by an xor butterfly, which leaves the
// same float in each of them; both selection forms use exactly this order.
__host__ __device__ inline int lanes_per_block(int Hq) {
  const int l = Hq / 4;
  if (Hq % 4 != 0 || (l & (l - 1)) != 0) return 1;
  return l < 4 ? l : 4;
}

// Term of head h in I_b: e^{z + ln n_b - L_h} (L_h - z).
__device__ __forceinline__ float score_term(float z, float lnn, float L) {
  return expf(z + lnn - L) * (L - z);
}

// LPB is 1, 2 or 4: constant offsets (cheap cross-lane moves), the levels
// past LPB skipped uniformly.
__device__ __forceinline__ float lanes_sum(float acc, int LPB) {
  if (LPB > 1) acc += __shfl_xor(acc, 1);
  if (LPB > 2) acc += __shfl_xor(acc, 2);
  return acc;
}

// ln n_b of block j (of nb; the last holds N - 16 (nb - 1) tokens).
__device__ __forceinline__ float block_ln_count(int j, int N, int nb) {
  return logf(static_cast<float>(j == nb - 1 ? N - kBlock * (nb - 1) : kBlock));
}

// Step B for blocks j0 .. j0 + TB - 1 of sequence b (context length N, nb
// blocks) by NT threads, in passes of NT / LPB blocks, L_h in LDS (sL).  A
// block's terms and their order do not depend on NT or TB.
// COH: the scores are stored at device scope (read by another workgroup of
// the same launch).
template <int NT, int TB, bool COH = false>
__device__ __forceinline__ void block_score_tile(const float* __restrict__ zbuf, const float* sL,
                                                 float* __restrict__ scores, int Hq, int MAXB,
                                                 int b, int N, int nb, int j0) {
  const int t = threadIdx.x;
  const int LPB = lanes_per_block(Hq);
  const int HPLN = Hq / LPB;
  const int bpp = NT / LPB;
  const int li = t % LPB;
  for (int jp = j0; jp < j0 + TB; jp += bpp) {
    const int j = jp + t / LPB;
    const bool ok = j < nb && j < j0 + TB;
    float acc = 0.f;
    if (ok) {
      const float lnn = block_ln_count(j, N, nb);
      const float* zr = zbuf + (static_cast<long long>(b) * MAXB + j) * Hq + li * HPLN;
      if (HPLN % 4 == 0) {
        // The lane's loads in batches of eight issued together (one batch
        // for four lanes per block; up to four when one lane takes all of
        // H_q <= 128 heads), the terms in head order.
        constexpr int kBatchF4 = 8;
        for (int f0 = 0; f0 < HPLN / 4; f0 += kBatchF4) {
          float4 z4[kBatchF4];
#pragma unroll
          for (int f = 0; f < kBatchF4; ++f)
            if (f0 + f < HPLN / 4) z4[f] = *reinterpret_cast<const float4*>(zr + 4 * (f0 + f));
#pragma unroll
          for (int f = 0; f < kBatchF4; ++f) {
            if (f0 + f >= HPLN / 4) break;
            const int h = li * HPLN + 4 * (f0 + f);
            acc += score_term(z4[f].x, lnn, sL[h]);
            acc += score_term(z4[f].y, lnn, sL[h + 1]);
            acc += score_term(z4[f].z, lnn, sL[h + 2]);
            acc += score_term(z4[f].w, lnn, sL[h + 3]);
          }
        }
      } else {
        for (int e = 0; e < HPLN; ++e) acc += score_term(zr[e], lnn, sL[li * HPLN + e]);
      }
    }
    acc = lanes_sum(acc, LPB);
    if (ok && li == 0) {
      float* dst = scores + static_cast<long long>(b) * MAXB + j;
      const float I = __fdiv_rn(acc, static_cast<float>(Hq));
      if (COH) __hip_atomic_store(dst, I, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else *dst = I;
    }
  }
}

// Step B as its own launch: blocks j0 .. j0 + 63 of sequence b by 256
// threads, L_h from the per-sequence launch of step A.
__device__ __forceinline__ void block_score_body(const float* __restrict__ zbuf,
                                                 const float* __restrict__ L,
                                                 const int* __restrict__ ctx_lens,
                                                 float* __restrict__ scores, int Hq, int MAXB,
                                                 int b, int j0, float* sL) {
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;    // flagged in step C
  const int nb = (N + kBlock - 1) / kBlock;
  if (j0 >= nb) return;
  for (int h = threadIdx.x; h < Hq; h += kRowThreads) sL[h] = L[static_cast<long long>(b) * Hq + h];
  __syncthreads();
  block_score_tile<kRowThreads, kTileBlocks>(zbuf, sL, scores, Hq, MAXB, b, N, nb, j0);
}

// Steps A and B together for blocks j0 .. j0 + kStepTileBlocks - 1 of
// sequence b, by kFoldThreads threads (the fused step's long-table form):
// L_h merged in LDS exactly as step A's own launch merges it, then the
// tile's scores.  Every thread must call it.
constexpr int kStepTileBlocks = 256;
template <bool COH = false>
__device__ __forceinline__ void lse_block_score_body(const float* __restrict__ zbuf,
                                                     const float* __restrict__ lse_part,
                                                     const int* __restrict__ ctx_lens,
                                                     float* __restrict__ scores, int Hq, int MAXB,
                                                     int nch_max, int b, int j0, float* s_pm,
                                                     float* s_ps, float* sL) {
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;    // flagged in step C
  const int nb = (N + kBlock - 1) / kBlock;
  if (j0 >= nb) return;
  lse_merge_body(lse_part, ctx_lens, sL, Hq, MAXB, nch_max, b, s_pm, s_ps);
  __syncthreads();
  block_score_tile<kFoldThreads, kStepTileBlocks, COH>(zbuf, sL, scores, Hq, MAXB, b, N, nb, j0);
}

constexpr int kSelRankMax = 64;    // prefix groups this small are finished by counting ranks

struct SelectShared {
  unsigned hist[256];                // radix histogram, then the last candidates
  unsigned red[2 * kSelWaves];
  float pm[kFoldThreads], ps[kFoldThreads], L[128];
  int digit, krem, ncand, wcnt[kSelWaves];
  unsigned rv;
};

// Physical block p of logical block j (of nb) for the decode's unit lists:
// p, with bit 30 set for the sequence's last block; -1 when p is outside the
// pool (the decode flags it).  Pools hold fewer than 2^30 blocks.
__device__ __forceinline__ int encode_phys(int p, int j, int nb, int P) {
  if (p < 0 || p >= P) return -1;
  return p | (j == nb - 1 ? (1 << 30) : 0);
}

// Step C core: the nb keys of sequence b are in LDS (keys), k >= 1.
// tbl: LDS [nb] physical block of each block, encoded (encode_phys);
// kphys (global [B, MAXB]) receives them in kept order.
__device__ __forceinline__ void select_core(unsigned* keys, const int* tbl, int nb, int k,
                                            float* __restrict__ theta_out, int* __restrict__ kept,
                                            int* __restrict__ kphys, int* __restrict__ n_kept,
                                            int MAXB, int b, SelectShared& sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  unsigned kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int i = t; i < nb; i += kSelThreads) {
    const unsigned key = keys[i];
    kmin = min(kmin, key);
    kmax = max(kmax, key);
  }
  kmin = wave_min_u(kmin);
  kmax = wave_max_u(kmax);
  if (lane == 0) {
    sh.red[wave] = kmin;
    sh.red[kSelWaves + wave] = kmax;
  }
  if (t == 0) sh.krem = k;
  __syncthreads();
  kmin = sh.red[0];
  kmax = sh.red[kSelWaves];
#pragma unroll
  for (int w = 1; w < kSelWaves; ++w) {
    kmin = min(kmin, sh.red[w]);
    kmax = max(kmax, sh.red[kSelWaves + w]);
  }
  // Radix select of the k-th largest key over the differing bits, 8 at a
  // time from the top (the common leading bits are the prefix already);
  // once at most kSelRankMax keys share the prefix, the answer is found
  // among them by counting ranks.
  const unsigned diff = kmin ^ kmax;
  const int top = diff ? 31 - __clz(diff) : -1;    // highest differing bit
  unsigned mask = diff ? ~((2u << top) - 1u) : 0xFFFFFFFFu;
  if (top == 31) mask = 0u;
  unsigned prefix = kmax & mask;
  for (int hi = top; hi >= 0; hi -= 8) {
    const int shift = max(hi - 7, 0);
    const int width = hi - shift + 1;
    const unsigned dmask = (1u << width) - 1u;
    if (t < 256) sh.hist[t] = 0u;
    __syncthreads();
    for (int i = t; i < nb; i += kSelThreads) {
      const unsigned key = keys[i];
      if ((key & mask) == prefix) atomicAdd(&sh.hist[(key >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // Bins 4*lane .. 4*lane+3; suffix sums over lanes locate the digit
      // holding the k_rem-th largest remaining key.
      const unsigned c0 = sh.hist[4 * lane], c1 = sh.hist[4 * lane + 1],
                     c2 = sh.hist[4 * lane + 2], c3 = sh.hist[4 * lane + 3];
      const unsigned cl = c0 + c1 + c2 + c3;
      unsigned suf = cl;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned n = __shfl_down(suf, o);
        if (lane + o < 64) suf += n;
      }
      const unsigned krem = static_cast<unsigned>(sh.krem);
      const unsigned above = suf - cl;       // keys in higher lanes' bins
      if (above < krem && suf >= krem) {
        unsigned run = above;
        const unsigned cs[4] = {c0, c1, c2, c3};
        int d = 4 * lane;
        for (int x = 3; x >= 0; --x) {
          if (run + cs[x] >= krem) {
            d = 4 * lane + x;
            break;
          }
          run += cs[x];
        }
        sh.digit = d;
        sh.krem = static_cast<int>(krem - run);
      }
    }
    __syncthreads();
    prefix |= static_cast<unsigned>(sh.digit) << shift;
    mask |= dmask << shift;
    const int c = static_cast<int>(sh.hist[sh.digit]);   // keys sharing the new prefix
    const int krem = sh.krem;
    __syncthreads();                       // every thread has read both before reuse
    if (shift > 0 && c <= kSelRankMax) {
      if (t == 0) sh.ncand = 0;
      __syncthreads();
      for (int i = t; i < nb; i += kSelThreads) {
        const unsigned key = keys[i];
        if ((key & mask) == prefix) sh.hist[atomicAdd(&sh.ncand, 1)] = key;
      }
      __syncthreads();
      if (t < c) {
        const unsigned v = sh.hist[t];
        int gt = 0, ge = 0;
        for (int j = 0; j < c; ++j) {
          const unsigned x = sh.hist[j];
          gt += x > v;
          ge += x >= v;
        }
        if (gt < krem && ge >= krem) sh.rv = v;   // equal keys write the same value
      }
      __syncthreads();
      prefix = sh.rv;
      break;
    }
  }
  const unsigned tkey = prefix;

  // Compaction in ascending block order.
  int total = 0;
  int* krow = kept + static_cast<long long>(b) * MAXB;
  for (int base = 0; base < nb; base += kSelThreads) {
    const int i = base + t;
    const bool f = i < nb && keys[i] >= tkey;
    const unsigned long long bal = __ballot(f);
    const int rank = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) sh.wcnt[wave] = __popcll(bal);
    __syncthreads();
    int off = total;
    for (int w = 0; w < wave; ++w) off += sh.wcnt[w];
    if (f) {
      krow[off + rank] = i;
      kphys[static_cast<long long>(b) * MAXB + off + rank] = tbl[i];
    }
    for (int w = 0; w < kSelWaves; ++w) total += sh.wcnt[w];
    __syncthreads();
  }
  if (t == 0) {
    n_kept[b] = total;
    if (theta_out) theta_out[b] = key_float(tkey);
  }
}

// Forced keeps: the first keep_first and the last keep_last of a sequence's
// nb blocks rank above every score (key of +inf) and count toward the
// budget, which becomes max(k, their number).
__device__ __forceinline__ bool forced_block(int j, int nb, const Budget& bu) {
  return j < bu.keep_first || j >= nb - bu.keep_last;
}
__device__ __forceinline__ int forced_budget(int k, int nb, const Budget& bu) {
  const int nf = min(nb, min(bu.keep_first, nb) + min(bu.keep_last, nb));
  return max(k, nf);
}
__device__ __forceinline__ unsigned select_key(float I, int j, int nb, const Budget& bu) {
  return forced_block(j, nb, bu) ? float_key(INFINITY) : float_key(I);
}

// No block kept: the outputs of sequence b.
__device__ __forceinline__ void select_none(float* __restrict__ theta_out, int* __restrict__ n_kept,
                                            int b) {
  if (threadIdx.x == 0) {
    n_kept[b] = 0;
    if (theta_out) theta_out[b] = INFINITY;
  }
}

// Validates sequence b's context and returns its blocks and budget; false
// (outputs written) when the context is invalid or empty.  Uniform across
// the workgroup.
__device__ __forceinline__ bool select_prepare(int N, float hval, float* __restrict__ theta_out,
                                               int* __restrict__ n_kept, int MAXB,
                                               const Budget& bu, float kprev, unsigned* flags,
                                               int b, int& nb, int& k) {
  const int t = threadIdx.x;
  if (N < 0 || N > MAXB * kBlock) {
    if (t == 0) {
      raise_flag(flags, ENT_DEV_BAD_CTXLEN);
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return false;
  }
  nb = (N + kBlock - 1) / kBlock;
  k = keep_budget(hval, nb, bu, kprev);
  if (nb == 0) {
    select_none(theta_out, n_kept, b);
    return false;
  }
  return true;
}

// Step C as its own launch: keys from step B's scores (COH: read at device
// scope, written by other workgroups of the same launch).
template <bool COH = false>
__device__ __forceinline__ void select_row_body(
    const float* __restrict__ scores, const int* __restrict__ ctx_lens,
    const int* __restrict__ tables, float hval, float* __restrict__ theta_out,
    int* __restrict__ kept, int* __restrict__ kphys, int* __restrict__ n_kept, int MAXB, int P,
    const Budget& bu, unsigned* flags, int b, unsigned* keys, int* tbl, SelectShared& sh) {
  const int N = ctx_lens[b];
  const float kprev = budget_prev(bu, b);
  int nb, k;
  if (!select_prepare(N, hval, theta_out, n_kept, MAXB, bu, kprev, flags, b, nb, k))
    return;
  {
    float ku;
    keep_budget(hval, nb, bu, kprev, &ku);
    __syncthreads();              // every thread has read the previous fraction
    budget_record(bu, b, ku);
  }
  k = forced_budget(k, nb, bu);
  if (k <= 0) {
    select_none(theta_out, n_kept, b);
    return;
  }
  const float* sr = scores + static_cast<long long>(b) * MAXB;
  const int* tr = tables + static_cast<long long>(b) * MAXB;
  for (int i = threadIdx.x; i < nb; i += kSelThreads) {
    const float I = COH ? __hip_atomic_load(sr + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : sr[i];
    keys[i] = select_key(I, i, nb, bu);
    tbl[i] = encode_phys(tr[i], i, nb, P);
  }
  __syncthreads();
  select_core(keys, tbl, nb, k, theta_out, kept, kphys, n_kept, MAXB, b, sh);
}

// Steps A, B and C in one workgroup (block tables up to kSelMaxBlocks wide
// and H_q x width up to kSelMaxTerms, H_q / 4 a power of two), in two parts
// so that a caller can overlap other work with the loads: select_load
// issues every global read of the sequence at once into registers, for the
// whole block-table row, so that no load waits for the context length
// (entries past the sequence's blocks are read and never used): the block
// logits (LPB lanes per block, F4 = H_q / (4 LPB) 16-byte loads of four
// heads per lane and pass), the table entries (thread t takes entries t,
// t + 512, ...) and the per-tile log-sum-exp partials of the L merge;
// select_finish merges L, scores the blocks and selects.  The arithmetic,
// and its order, is that of the long-table forms (lse_merge_body,
// block_score_tile, select_core).  The block logits take kSelZRegs float4
// registers: 16 / F4 passes of kSelThreads / LPB blocks.
constexpr int kSelTableRegs = kSelMaxBlocks / kSelThreads;
constexpr int kSelZRegs = 16;
constexpr int kSelTiles = 4;              // L-merge tiles per thread, at most
constexpr int kSelMaxTerms = 32768;       // H_q x block-table width, at most

typedef float sel_f32x4 __attribute__((ext_vector_type(4)));

template <int F4>
struct SelectRegs {
  static constexpr int kPasses = kSelZRegs / F4;
  sel_f32x4 z[kSelZRegs];
  float2 pr[kSelTiles];
  int tb[kSelTableRegs];
};

// F4 of the one-launch form (1, 2, 4 or 8), or 0 when the long-table forms
// apply.  Both the staged and the fused step decide with this, so they take
// the same selection arithmetic.  One workgroup evaluates every head's term
// of every block of its sequence: beyond kSelMaxTerms the chip-wide block
// scores of the long-table forms are faster (64 heads x 1028 blocks: 37 us
// against 28 us for the three launches and 20 us for the fused step's two).
__host__ __device__ inline int select_one_launch(int MAXB, int Hq) {
  if (Hq > 128 || Hq % 4 != 0 || MAXB > kSelMaxBlocks) return 0;
  const int lpb = lanes_per_block(Hq);
  if (lpb * 4 > Hq || ((Hq / 4) & (Hq / 4 - 1)) != 0) return 0;
  if (static_cast<long long>(Hq) * MAXB > kSelMaxTerms) return 0;
  const int f4 = Hq / (4 * lpb);
  const int bpp = kSelThreads / lpb;
  const int passes = (MAXB + bpp - 1) / bpp;
  const int nch = (MAXB + kMfmaChunk - 1) / kMfmaChunk;
  const int vph = kFoldThreads / Hq;
  const int tiles = (nch + vph - 1) / vph;
  if (passes * f4 > kSelZRegs || tiles > kSelTiles) return 0;
  return f4;
}

template <int F4>
__device__ __forceinline__ void select_load(const float* __restrict__ zbuf,
                                            const float* __restrict__ lse_part,
                                            const int* __restrict__ tables, int MAXB,
                                            int nch_max, int b, int Hq, SelectRegs<F4>& R) {
  const int t = threadIdx.x;
  const int LPB = lanes_per_block(Hq);
  const int lg = LPB == 4 ? 2 : LPB - 1;      // log2 LPB
  const int bpp = kSelThreads >> lg;
  const int li = t & (LPB - 1);
#pragma unroll
  for (int p = 0; p < SelectRegs<F4>::kPasses; ++p) {
    const int j = p * bpp + (t >> lg);
    if (j < MAXB) {
      const float* zr = zbuf + (static_cast<long long>(b) * MAXB + j) * Hq + li * (4 * F4);
#pragma unroll
      for (int f = 0; f < F4; ++f) R.z[p * F4 + f] = *reinterpret_cast<const sel_f32x4*>(zr + 4 * f);
    }
  }
#pragma unroll
  for (int i = 0; i < kSelTableRegs; ++i) {
    const int j = t + i * kSelThreads;
    if (j < MAXB) R.tb[i] = tables[static_cast<long long>(b) * MAXB + j];
  }
  static_assert(kSelThreads == kFoldThreads, "one virtual fold thread per thread");
  const int nch = (MAXB + kMfmaChunk - 1) / kMfmaChunk;
  const int vph = kFoldThreads / Hq;
  if (t < vph * Hq) {
    const float* lp = lse_part + (static_cast<long long>(b) * nch_max * Hq + t % Hq) * 2;
#pragma unroll
    for (int i = 0; i < kSelTiles; ++i) {
      const int c = t / Hq + i * vph;
      if (c < nch) R.pr[i] = *reinterpret_cast<const float2*>(lp + static_cast<long long>(c) * Hq * 2);
    }
  }
}

template <int F4>
__device__ __forceinline__ void select_finish(
    const SelectRegs<F4>& R, int N, int nb, float hval, float* __restrict__ scores_out,
    float* __restrict__ theta_out, int* __restrict__ kept, int* __restrict__ kphys,
    int* __restrict__ n_kept, int MAXB, int P, const Budget& bu, float kprev, int b, int Hq,
    unsigned* keys, int* tbl, SelectShared& sh) {
  const int vph = kFoldThreads / Hq;
  const int t = threadIdx.x;
  // Step A (lse_fold_vthread and lse_merge_tree, from the registers).
  const int nch = (nb + kMfmaChunk - 1) / kMfmaChunk;
  {
    float m = -INFINITY, sum = 0.f;
    if (t < vph * Hq) {
#pragma unroll
      for (int i = 0; i < kSelTiles; ++i)
        if (t / Hq + i * vph < nch) m = fmaxf(m, R.pr[i].x);
      if (m != -INFINITY) {
#pragma unroll
        for (int i = 0; i < kSelTiles; ++i)
          if (t / Hq + i * vph < nch) sum += R.pr[i].y * expf(R.pr[i].x - m);
      }
    }
    sh.pm[t] = m;
    sh.ps[t] = sum;
  }
  __syncthreads();
  lse_merge_tree(sh.pm, sh.ps, Hq);
  if (t < Hq) sh.L[t] = lse_merged(sh.pm, sh.ps, t);
  __syncthreads();
  // Step B (block_score_body's head sum, on the registers).
  const int LPB = lanes_per_block(Hq);
  const int lg = LPB == 4 ? 2 : LPB - 1;
  const int bpp = kSelThreads >> lg;
  const int li = t & (LPB - 1);
#pragma unroll
  for (int p = 0; p < SelectRegs<F4>::kPasses; ++p) {
    if (p * bpp >= nb) break;
    const int j = p * bpp + (t >> lg);
    float acc = 0.f;
    if (j < nb) {
      const float lnn = block_ln_count(j, N, nb);
#pragma unroll
      for (int f = 0; f < F4; ++f) {
        const int h = li * (4 * F4) + 4 * f;
        const sel_f32x4 z = R.z[p * F4 + f];
        acc += score_term(z.x, lnn, sh.L[h]);
        acc += score_term(z.y, lnn, sh.L[h + 1]);
        acc += score_term(z.z, lnn, sh.L[h + 2]);
        acc += score_term(z.w, lnn, sh.L[h + 3]);
      }
    }
    acc = lanes_sum(acc, LPB);
    const float I = __fdiv_rn(acc, static_cast<float>(Hq));
    if (j < nb && li == 0) {
      keys[j] = select_key(I, j, nb, bu);
      if (scores_out) scores_out[static_cast<long long>(b) * MAXB + j] = I;
    }
  }
#pragma unroll
  for (int i = 0; i < kSelTableRegs; ++i) {
    const int j = t + i * kSelThreads;
    if (j < nb) tbl[j] = encode_phys(R.tb[i], j, nb, P);
  }
  __syncthreads();
  float ku;
  const int k = forced_budget(keep_budget(hval, nb, bu, kprev, &ku), nb, bu);
  budget_record(bu, b, ku);       // every thread read kprev before the barriers above
  if (k <= 0) {
    select_none(theta_out, n_kept, b);
    return;
  }
  select_core(keys, tbl, nb, k, theta_out, kept, kphys, n_kept, MAXB, b, sh);
}

// The one-launch selection of sequence b with its entropy in hval.
template <int F4>
__device__ __forceinline__ void select_fused_body(
    const float* __restrict__ zbuf, const float* __restrict__ lse_part,
    const int* __restrict__ ctx_lens, const int* __restrict__ tables, float hval,
    float* __restrict__ scores_out, float* __restrict__ theta_out, int* __restrict__ kept,
    int* __restrict__ kphys, int* __restrict__ n_kept, int MAXB, int P, int nch_max, int Hq,
    const Budget& bu, unsigned* flags, int b, unsigned* keys, int* tbl, SelectShared& sh) {
  SelectRegs<F4> R;
  select_load<F4>(zbuf, lse_part, tables, MAXB, nch_max, b, Hq, R);
  const int N = ctx_lens[b];
  const float kprev = budget_prev(bu, b);
  int nb, k;
  if (!select_prepare(N, hval, theta_out, n_kept, MAXB, bu, kprev, flags, b, nb, k))
    return;
  select_finish<F4>(R, N, nb, hval, scores_out, theta_out, kept, kphys, n_kept, MAXB, P, bu, kprev,
                    b, Hq, keys, tbl, sh);
}

// Append of one token to sequence b's cache by one workgroup of
// kAppendThreads threads (ent_kv_append): write its key and value at
// position N = ctx_lens[b], refresh its block's mean key, set ctx_lens[b] =
// N + 1.  The block's mean is the sum of its valid slots in slot order,
// divided by their number (correctly rounded), as the summary pass computes
// it, so both give the same bits.
constexpr int kAppendThreads = 256;

template <typename T>
__device__ __forceinline__ void append_body(const AppendArgs& a, int b) {
  const T* __restrict__ k_new = static_cast<const T*>(a.k_new);
  const T* __restrict__ v_new = static_cast<const T*>(a.v_new);
  const int* __restrict__ tables = a.tables;
  int* __restrict__ ctx_lens = a.ctx_lens;
  T* __restrict__ kc = static_cast<T*>(a.kc);
  T* __restrict__ vc = static_cast<T*>(a.vc);
  float* __restrict__ ksum = a.ksum;
  const int Hkv = a.Hkv, D = a.D, MAXB = a.MAXB, P = a.P;
  unsigned* flags = a.flags;
  const int N = ctx_lens[b];
  if (N < 0 || N >= MAXB * kBlock) {
    if (threadIdx.x == 0) raise_flag(flags, N < 0 ? ENT_DEV_BAD_CTXLEN : ENT_DEV_CACHE_FULL);
    return;
  }
  const int j = N / kBlock, slot = N % kBlock;
  const int p = tables[static_cast<long long>(b) * MAXB + j];
  if (p < 0 || p >= P) {
    if (threadIdx.x == 0) raise_flag(flags, ENT_DEV_BAD_TABLE);
    return;
  }
  // A 16-byte piece of one KV head's row (VE elements) at a time: the new
  // key and value, and (for the block's mean) the earlier slots' keys, all
  // loaded at once (slots from `slot` on are read and not used: the tile
  // always holds 16); each element is then summed in slot order, the new key
  // last.  When the workgroup has two threads per piece, the first loads and
  // sums slots 0..7 and hands its sums through LDS to the second, which
  // continues with slots 8..14 (the same additions in the same order, half
  // the registers each).
  constexpr int VE = 16 / sizeof(T);
  constexpr int kHalf = kBlock / 2;           // slots of the first thread of a pair
  __shared__ float s_part[kAppendThreads / 2 * VE];
  const int items = Hkv * D / VE;
  if (2 * items <= kAppendThreads) {
    const int half = threadIdx.x / items, v = threadIdx.x - half * items;
    const bool act = half < 2;
    const int e0 = v * VE;
    const int g = e0 / D, dd = e0 % D;
    const long long src = (static_cast<long long>(b) * Hkv + g) * D + dd;
    const long long tile = (static_cast<long long>(p) * Hkv + g) * kBlock * D;
    uint4 kraw = make_uint4(0u, 0u, 0u, 0u), vraw = kraw;
    uint4 raw[kHalf];
    if (act) {
      kraw = *reinterpret_cast<const uint4*>(k_new + src);
      if (half == 0) vraw = *reinterpret_cast<const uint4*>(v_new + src);
      if (ksum) {
#pragma unroll
        for (int i = 0; i < kHalf; ++i)
          if (half == 0 || i < kHalf - 1)
            raw[i] = *reinterpret_cast<const uint4*>(kc + tile + (half * kHalf + i) * D + dd);
      }
    }
    float sum[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) sum[i] = 0.f;
    if (act && half == 0) {
      *reinterpret_cast<uint4*>(kc + tile + slot * D + dd) = kraw;
      const T* vx = reinterpret_cast<const T*>(&vraw);
#pragma unroll
      for (int i = 0; i < VE; ++i) vc[tile + (dd + i) * kBlock + slot] = vx[i];
      if (ksum) {
#pragma unroll
        for (int s2 = 0; s2 < kHalf; ++s2) {
          const T* x = reinterpret_cast<const T*>(&raw[s2]);
          if (s2 < slot) {
#pragma unroll
            for (int i = 0; i < VE; ++i) sum[i] += load_elem<T>(x + i);
          }
        }
#pragma unroll
        for (int i = 0; i < VE; ++i) s_part[v * VE + i] = sum[i];
      }
    }
    __syncthreads();
    if (act && half == 1 && ksum) {
#pragma unroll
      for (int i = 0; i < VE; ++i) sum[i] = s_part[v * VE + i];
#pragma unroll
      for (int s2 = kHalf; s2 < kBlock - 1; ++s2) {
        const T* x = reinterpret_cast<const T*>(&raw[s2 - kHalf]);
        if (s2 < slot) {
#pragma unroll
          for (int i = 0; i < VE; ++i) sum[i] += load_elem<T>(x + i);
        }
      }
      const T* kx = reinterpret_cast<const T*>(&kraw);
      float* out = ksum + (static_cast<long long>(p) * Hkv + g) * D + dd;
#pragma unroll
      for (int i = 0; i < VE; ++i) out[i] = __fdiv_rn(sum[i] + load_elem<T>(kx + i), static_cast<float>(slot + 1));
    }
  } else {
    for (int v = threadIdx.x; v < items; v += kAppendThreads) {
      const int e0 = v * VE;
      const int g = e0 / D, dd = e0 % D;
      const long long src = (static_cast<long long>(b) * Hkv + g) * D + dd;
      const long long tile = (static_cast<long long>(p) * Hkv + g) * kBlock * D;
      const uint4 kraw = *reinterpret_cast<const uint4*>(k_new + src);
      const uint4 vraw = *reinterpret_cast<const uint4*>(v_new + src);
      // The earlier slots in two halves of kHalf rows through one array.
      uint4 raw[kHalf];
      if (ksum) {
#pragma unroll
        for (int i = 0; i < kHalf; ++i) raw[i] = *reinterpret_cast<const uint4*>(kc + tile + i * D + dd);
      }
      *reinterpret_cast<uint4*>(kc + tile + slot * D + dd) = kraw;
      const T* kx = reinterpret_cast<const T*>(&kraw);
      const T* vx = reinterpret_cast<const T*>(&vraw);
#pragma unroll
      for (int i = 0; i < VE; ++i) vc[tile + (dd + i) * kBlock + slot] = vx[i];
      if (ksum) {
        float sum[VE];
#pragma unroll
        for (int i = 0; i < VE; ++i) sum[i] = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < kHalf; ++s2) {
          const T* x = reinterpret_cast<const T*>(&raw[s2]);
          if (s2 < slot) {
#pragma unroll
            for (int i = 0; i < VE; ++i) sum[i] += load_elem<T>(x + i);
          }
        }
        if (slot > kHalf) {
#pragma unroll
          for (int i = 0; i < kHalf - 1; ++i)
            raw[i] = *reinterpret_cast<const uint4*>(kc + tile + (kHalf + i) * D + dd);
#pragma unroll
          for (int s2 = kHalf; s2 < kBlock - 1; ++s2) {
            const T* x = reinterpret_cast<const T*>(&raw[s2 - kHalf]);
            if (s2 < slot) {
#pragma unroll
              for (int i = 0; i < VE; ++i) sum[i] += load_elem<T>(x + i);
            }
          }
        }
        float* out = ksum + (static_cast<long long>(p) * Hkv + g) * D + dd;
#pragma unroll
        for (int i = 0; i < VE; ++i) out[i] = __fdiv_rn(sum[i] + load_elem<T>(kx + i), static_cast<float>(slot + 1));
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) ctx_lens[b] = N + 1;
}

}  // namespace
}  // namespace ent
