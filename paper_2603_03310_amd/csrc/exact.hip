// Exact token-level block scores, the conservative scoring mode (Section 3.2
// of the paper: a block's entropic contribution is the attention-weighted
// surprisal of its tokens, here with the exact attention weights of the
// current query over every valid key of the sequence).
//
// For query head h, token scores s_i = scale <q_h, k_i>, weights
// a_i = e^{s_i - L_h} with L_h = ln sum_i e^{s_i}, and
//   I_bh = sum_{i in b} a_i (L_h - s_i) = e^{l_bh - L_h} (L_h - zbar_bh),
//   l_bh    = ln sum_{i in b} e^{s_i}                   (the block's log mass)
//   zbar_bh = sum_{i in b} e^{s_i} s_i / sum_{i in b} e^{s_i}   (its mean logit)
// so one pass over K gives, per block and head, the pair (l, zbar), and per
// tile of 16 blocks the log-sum-exp partial (max l, sum e^{l - max}) in the
// same format as the mean-key scoring.  L_h then comes from the selection's
// merge of those partials, I_b = (1/H_q) sum_h I_bh from the pairs, and the
// selection is the mean-key mode's.
//
// bf16 (MFMA).  Workgroup = (KV head g, tile of 16 blocks, sequence); each
// of its eight waves takes two blocks and issues both K tiles at once.
// Per block S^T[16 tok x 16] = K[16 x d] . Q_g^T[d x 16] on
// v_mfma_f32_16x16x32_bf16 (columns: the G query heads of g, zero-padded);
// lane (r16, gq) holds tokens 4 gq .. 4 gq + 3 of head r16, and the block's
// max, sum and weighted sum reduce over gq with two shuffles.
// fp32 (VALU).  Same grid; lane (token r16, head slot l / 16) forms full dot
// products (queries in LDS), four heads per pass, and reduces over the 16
// tokens with shuffles.

#include "blocks_dev.h"

namespace ent {
namespace {

constexpr int kExThreads = 512;   // 2 blocks per wave: measured faster than 1, 4 or 8
constexpr int kExWaves = kExThreads / 64;
constexpr int kExPerWave = kMfmaChunk / kExWaves;   // blocks per wave

typedef __bf16 xbf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef unsigned u32x4nt_t __attribute__((ext_vector_type(4)));
typedef float xf32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

struct ExactArgs {
  const void* q;
  const void* kc;
  const int* tables;
  const int* ctx_lens;
  float2* ex;          // [B, MAXB, H_q] (l, zbar)
  float* lse_part;     // [B, nch_max, H_q, 2]
  unsigned* flags;
  int Hkv, G, MAXB, P, nch_max;
  float scale;
};

// Physical block of logical block j (< nb) of sequence b, validated (0 and a
// flag when outside the pool; such a block is still read, never trusted).
__device__ __forceinline__ int exact_phys(const ExactArgs& a, int b, int j, int nb) {
  if (j >= nb) return 0;
  int p = a.tables[static_cast<long long>(b) * a.MAXB + j];
  if (p < 0 || p >= a.P) {
    raise_flag(a.flags, ENT_DEV_BAD_TABLE);
    p = 0;
  }
  return p;
}

// Running log-sum-exp (m, s) of the block log masses seen so far, for one head.
__device__ __forceinline__ void lse_push(float& m, float& s, float l) {
  const float mn = fmaxf(m, l);
  s = s * expf(m - mn) + expf(l - mn);
  m = mn;
}

// The tile's partial of each query head of g from the waves' running pairs
// (LDS s_m, s_s [kExWaves][16], written by the caller).
__device__ __forceinline__ void write_tile_partial(const ExactArgs& a, int b, int ch, int g,
                                                   const float (*s_m)[16], const float (*s_s)[16]) {
  const int t = threadIdx.x;
  if (t >= a.G) return;
  float m = -INFINITY;
#pragma unroll
  for (int w = 0; w < kExWaves; ++w) m = fmaxf(m, s_m[w][t]);
  float sum = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int w = 0; w < kExWaves; ++w)
      if (s_m[w][t] != -INFINITY) sum += s_s[w][t] * expf(s_m[w][t] - m);
  }
  const int Hq = a.Hkv * a.G;
  float* lp = a.lse_part + ((static_cast<long long>(b) * a.nch_max + ch) * Hq + g * a.G + t) * 2;
  lp[0] = m;
  lp[1] = sum;
}

template <int D>
__global__ __launch_bounds__(kExThreads) void exact_score_bf16_kernel(ExactArgs a) {
  constexpr int KS = D / 32;
  __shared__ float s_m[kExWaves][16], s_s[kExWaves][16];
  // Each wave's K tile on its way into the MFMA layout, rows padded by 16 B.
  __shared__ __attribute__((aligned(16))) uint16_t s_kst[kExWaves * kBlock * (D + 8)];
  const int g = blockIdx.x, ch = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r16 = lane & 15, gq = lane >> 4;
  const int N = a.ctx_lens[b];
  if (N < 0 || N > a.MAXB * kBlock) return;      // flagged by the selection
  const int nb = (N + kBlock - 1) / kBlock;
  const int j0 = ch * kMfmaChunk + wave * kExPerWave;
  if (ch * kMfmaChunk >= nb) return;             // the whole workgroup
  const int G = a.G, Hq = a.Hkv * G;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  const uint16_t* kc = static_cast<const uint16_t*>(a.kc);
  // Every load first: the queries (B operand; MFMA k-slot (gq, e) of step ks
  // = dim 32 ks + 8 gq + e) and the wave's K tiles, each load instruction
  // covering 1 KB of a tile whole (lane l its 16 bytes l): against loads
  // straight into the MFMA layout (64 B of each of the 16 token rows per
  // instruction) the staged selection took 148 us against 153 us, and 135 us
  // with the non-temporal bit on these loads (which made the same loads in
  // the MFMA layout slower).
  xbf16x8_t qreg[KS];
  const long long qh = (static_cast<long long>(b) * Hq + g * G + r16) * D;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qreg[ks] = r16 < G ? __builtin_bit_cast(xbf16x8_t, *reinterpret_cast<const uint4*>(q + qh + 32 * ks + 8 * gq))
                       : __builtin_bit_cast(xbf16x8_t, make_uint4(0u, 0u, 0u, 0u));
  xbf16x8_t kr[kExPerWave][KS];
#pragma unroll
  for (int i = 0; i < kExPerWave; ++i) {
    const int p = exact_phys(a, b, j0 + i, nb);
    const long long tile = (static_cast<long long>(p) * a.Hkv + g) * kBlock * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kr[i][ks] = __builtin_bit_cast(
          xbf16x8_t, __builtin_nontemporal_load(
                         reinterpret_cast<const u32x4nt_t*>(kc + tile + ks * (kBlock * D / KS) + lane * 8)));
  }
  uint16_t* st = s_kst + wave * kBlock * (D + 8);
  float run_m = -INFINITY, run_s = 0.f;
#pragma unroll
  for (int i = 0; i < kExPerWave; ++i) {
    const int j = j0 + i;
    if (j >= nb) break;                          // uniform in the wave
    // The tile through the wave's own LDS rows into the MFMA layout (A
    // operand: token row r16); wave-level barriers order the exchange.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int e0 = ks * (kBlock * D / KS) + lane * 8;
      *reinterpret_cast<xbf16x8_t*>(st + (e0 / D) * (D + 8) + (e0 % D)) = kr[i][ks];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    xbf16x8_t kmf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kmf[ks] = *reinterpret_cast<const xbf16x8_t*>(st + r16 * (D + 8) + 32 * ks + 8 * gq);
    xf32x4_t acc = xf32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kmf[ks], qreg[ks], acc, 0, 0, 0);
    // acc[e]: token 4 gq + e, query head g G + r16.
    const int nv = j == nb - 1 ? N - kBlock * (nb - 1) : kBlock;
    float s[4];
    float m = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s[e] = acc[e] * a.scale;
      if (4 * gq + e < nv) m = fmaxf(m, s[e]);
    }
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    float S = 0.f, W = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (4 * gq + e < nv) {
        const float w = expf(s[e] - m);
        S += w;
        W += w * s[e];
      }
    }
    S += __shfl_xor(S, 16);
    S += __shfl_xor(S, 32);
    W += __shfl_xor(W, 16);
    W += __shfl_xor(W, 32);
    const float l = m + logf(S);
    if (gq == 0 && r16 < G)
      a.ex[(static_cast<long long>(b) * a.MAXB + j) * Hq + g * G + r16] = make_float2(l, W / S);
    lse_push(run_m, run_s, l);
  }
  if (gq == 0) {
    s_m[wave][r16] = run_m;
    s_s[wave][r16] = run_s;
  }
  __syncthreads();
  write_tile_partial(a, b, ch, g, s_m, s_s);
}

template <int D>
__global__ __launch_bounds__(kExThreads) void exact_score_f32_kernel(ExactArgs a) {
  extern __shared__ float s_q[];                 // [G, D]
  __shared__ float s_m[kExWaves][16], s_s[kExWaves][16];
  const int g = blockIdx.x, ch = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int tok = lane & 15, hs = lane >> 4;
  const int N = a.ctx_lens[b];
  if (N < 0 || N > a.MAXB * kBlock) return;
  const int nb = (N + kBlock - 1) / kBlock;
  if (ch * kMfmaChunk >= nb) return;
  const int G = a.G, Hq = a.Hkv * G;
  const float* q = static_cast<const float*>(a.q);
  const float* kc = static_cast<const float*>(a.kc);
  for (int e = t; e < G * D; e += kExThreads)
    s_q[e] = q[(static_cast<long long>(b) * Hq + g * G) * D + e];
  __syncthreads();
  // Lanes with tok == 0 keep the running pair of heads hs, hs + 4, ...
  float run_m[kMaxGroup / 4], run_s[kMaxGroup / 4];
#pragma unroll
  for (int u = 0; u < kMaxGroup / 4; ++u) {
    run_m[u] = -INFINITY;
    run_s[u] = 0.f;
  }
  const int j0 = ch * kMfmaChunk + wave * kExPerWave;
  for (int i = 0; i < kExPerWave; ++i) {
    const int j = j0 + i;
    if (j >= nb) break;                          // uniform in the wave
    const int p = exact_phys(a, b, j, nb);
    const int nv = j == nb - 1 ? N - kBlock * (nb - 1) : kBlock;
    const float* krow = kc + ((static_cast<long long>(p) * a.Hkv + g) * kBlock + tok) * D;
#pragma unroll
    for (int u = 0; u < kMaxGroup / 4; ++u) {
      const int h = hs + 4 * u;
      if (4 * u >= G) break;                     // uniform
      float dot = 0.f;
      if (h < G) {
        const float* qr = s_q + h * D;
#pragma unroll 8
        for (int dd = 0; dd < D; dd += 4) {
          const float4 k4 = *reinterpret_cast<const float4*>(krow + dd);
          dot += k4.x * qr[dd] + k4.y * qr[dd + 1] + k4.z * qr[dd + 2] + k4.w * qr[dd + 3];
        }
      }
      const bool ok = tok < nv;
      const float s = dot * a.scale;
      float m = ok ? s : -INFINITY;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
      const float w = ok ? expf(s - m) : 0.f;
      float S = w, W = ok ? w * s : 0.f;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        S += __shfl_xor(S, o);
        W += __shfl_xor(W, o);
      }
      const float l = m + logf(S);
      if (tok == 0 && h < G) {
        a.ex[(static_cast<long long>(b) * a.MAXB + j) * Hq + g * G + h] = make_float2(l, W / S);
        lse_push(run_m[u], run_s[u], l);
      }
    }
  }
  if (tok == 0) {
#pragma unroll
    for (int u = 0; u < kMaxGroup / 4; ++u) {
      const int h = hs + 4 * u;
      if (h < G) {
        s_m[wave][h] = run_m[u];
        s_s[wave][h] = run_s[u];
      }
    }
  }
  __syncthreads();
  write_tile_partial(a, b, ch, g, s_m, s_s);
}

// I_b from the pairs and L_h: blocks j0 .. j0 + 63 of sequence b, four lanes
// per block (heads qq, qq + 4, ...), as the mean-key mode's block scores.
__global__ __launch_bounds__(kRowThreads) void exact_block_score_kernel(
    const float2* __restrict__ ex, const float* __restrict__ L, const int* __restrict__ ctx_lens,
    float* __restrict__ scores, int Hq, int MAXB) {
  __shared__ float sL[128];
  const int t = threadIdx.x, b = blockIdx.y, j0 = blockIdx.x * kTileBlocks;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;        // flagged by the selection
  const int nb = (N + kBlock - 1) / kBlock;
  if (j0 >= nb) return;
  for (int h = t; h < Hq; h += kRowThreads) sL[h] = L[static_cast<long long>(b) * Hq + h];
  __syncthreads();
  const int j = j0 + (t >> 2), qq = t & 3;
  float acc = 0.f;
  if (j < nb) {
    const float2* er = ex + (static_cast<long long>(b) * MAXB + j) * Hq;
    for (int h = qq; h < Hq; h += 4) {
      const float2 e = er[h];
      acc += expf(e.x - sL[h]) * (sL[h] - e.y);
    }
  }
  acc += __shfl_xor(acc, 1);
  acc += __shfl_xor(acc, 2);
  if (j < nb && qq == 0) scores[static_cast<long long>(b) * MAXB + j] = __fdiv_rn(acc, static_cast<float>(Hq));
}

}  // namespace

hipError_t launch_exact_scores(const ent_ctx* c, int B, const void* q, const void* k_cache,
                               const int* tables, const int* ctx_lens, hipStream_t s) {
  const ent_config& cf = c->cfg;
  ExactArgs a;
  a.q = q;
  a.kc = k_cache;
  a.tables = tables;
  a.ctx_lens = ctx_lens;
  a.ex = c->exbuf;
  a.lse_part = c->lse_part;
  a.flags = c->dev_flags;
  a.Hkv = cf.num_kv_heads;
  a.G = c->group;
  a.MAXB = cf.max_blocks_per_seq;
  a.P = cf.num_pool_blocks;
  a.nch_max = c->lse_chunks;
  a.scale = cf.scale;
  if (!a.ex) return hipErrorInvalidValue;
  // KV heads vary fastest, so the workgroups in flight together read the
  // heads of the same blocks (each block's heads are contiguous).
  const dim3 grid(cf.num_kv_heads, (cf.max_blocks_per_seq + kMfmaChunk - 1) / kMfmaChunk, B);
  if (cf.kv_dtype == ENT_BF16) {
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(exact_score_bf16_kernel<128>, grid, dim3(kExThreads), 0, s, a);
    else
      hipLaunchKernelGGL(exact_score_bf16_kernel<64>, grid, dim3(kExThreads), 0, s, a);
  } else {
    const size_t lds = static_cast<size_t>(c->group) * cf.head_dim * sizeof(float);
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(exact_score_f32_kernel<128>, grid, dim3(kExThreads), lds, s, a);
    else
      hipLaunchKernelGGL(exact_score_f32_kernel<64>, grid, dim3(kExThreads), lds, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_exact_block_scores(const ent_ctx* c, int B, const int* ctx_lens, float* scores,
                                     hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid((cf.max_blocks_per_seq + kTileBlocks - 1) / kTileBlocks, B);
  hipLaunchKernelGGL(exact_block_score_kernel, grid, dim3(kRowThreads), 0, s, c->exbuf, c->lrow,
                     ctx_lens, scores, cf.num_q_heads, cf.max_blocks_per_seq);
  return hipGetLastError();
}

}  // namespace ent
