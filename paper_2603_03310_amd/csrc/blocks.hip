// Block summaries, block scores, the entropy-driven kept set, and token append.
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
//
// Kernels:
//   summary_kernel   per-block mean keys (setup)
//   score_kernel     z for 64 blocks x all heads per workgroup; per-chunk
//                    log-sum-exp partials per head
//   select_kernel    merges the partials, computes I_b for its 64 blocks; the
//                    last workgroup of a sequence (atomic ticket) runs a 4-pass
//                    8-bit radix select for the k-th largest score and compacts
//                    the kept blocks in ascending order with wave ballots
//   append_kernel    writes one token and refreshes its block's mean key

#include "ent_internal.h"

#include <math.h>

namespace ent {
namespace {

constexpr int kThreads = 256;

template <typename T>
__device__ __forceinline__ float load_elem(const T* p);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// Mean over slots [0, n) of element (g, dd) of physical block p's K tile, in
// slot order.  Shared by the summary and append kernels so both produce the
// same bits.  `last` (slot n-1) is passed in by the caller.
template <typename T>
__device__ __forceinline__ float block_mean(const T* __restrict__ kc, long long tile, int D, int dd,
                                            int n, float last) {
  float s = 0.f;
  for (int slot = 0; slot < n - 1; ++slot) s += load_elem<T>(kc + tile + slot * D + dd);
  s += last;
  return __fdiv_rn(s, static_cast<float>(n));
}

template <typename T>
__global__ __launch_bounds__(kThreads) void summary_kernel(
    const T* __restrict__ kc, const int* __restrict__ tables, const int* __restrict__ ctx_lens,
    float* __restrict__ ksum, int Hkv, int D, int MAXB, int P, unsigned* flags) {
  const int j = blockIdx.x, b = blockIdx.y;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) {
    if (j == 0 && threadIdx.x == 0) raise_flag(flags, ENT_DEV_BAD_CTXLEN);
    return;
  }
  const int nb = (N + kBlock - 1) / kBlock;
  if (j >= nb) return;
  const int p = tables[static_cast<long long>(b) * MAXB + j];
  if (p < 0 || p >= P) {
    if (threadIdx.x == 0) raise_flag(flags, ENT_DEV_BAD_TABLE);
    return;
  }
  const int n = (j == nb - 1) ? N - kBlock * (nb - 1) : kBlock;
  for (int e = threadIdx.x; e < Hkv * D; e += kThreads) {
    const int g = e / D, dd = e % D;
    const long long tile = (static_cast<long long>(p) * Hkv + g) * kBlock * D;
    const float last = load_elem<T>(kc + tile + (n - 1) * D + dd);
    ksum[(static_cast<long long>(p) * Hkv + g) * D + dd] = block_mean<T>(kc, tile, D, dd, n, last);
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void append_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, const int* __restrict__ tables,
    int* __restrict__ ctx_lens, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ ksum,
    int Hkv, int D, int MAXB, int P, unsigned* flags) {
  const int b = blockIdx.x;
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
  for (int e = threadIdx.x; e < Hkv * D; e += kThreads) {
    const int g = e / D, dd = e % D;
    const long long src = (static_cast<long long>(b) * Hkv + g) * D + dd;
    const long long tile = (static_cast<long long>(p) * Hkv + g) * kBlock * D;
    const T kv = k_new[src];
    kc[tile + slot * D + dd] = kv;
    vc[tile + dd * kBlock + slot] = v_new[src];
    ksum[(static_cast<long long>(p) * Hkv + g) * D + dd] =
        block_mean<T>(kc, tile, D, dd, slot + 1, load_elem<T>(&kv));
  }
  __syncthreads();
  if (threadIdx.x == 0) ctx_lens[b] = N + 1;
}

// ---------------------------------------------------------------------------
// Scoring.  Lane layout: a group of L = D/4 lanes covers one (block, KV head)
// summary, 4 dims per lane (float4 loads, fully coalesced); a wave covers
// U = 64/L KV heads per instruction.  Each lane forms G partial dot products
// (one per query head of its KV head); a halving butterfly reduces them over
// the L lanes, leaving head r = li * G / L in lane li.
// ---------------------------------------------------------------------------
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

template <typename T>
__device__ __forceinline__ void load_q4(const T* p, float (&o)[4]);
template <>
__device__ __forceinline__ void load_q4<float>(const float* p, float (&o)[4]) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  o[0] = x.x; o[1] = x.y; o[2] = x.z; o[3] = x.w;
}
template <>
__device__ __forceinline__ void load_q4<uint16_t>(const uint16_t* p, float (&o)[4]) {
  const uint2 x = *reinterpret_cast<const uint2*>(p);
  o[0] = bf16_to_f32(static_cast<uint16_t>(x.x & 0xffffu));
  o[1] = bf16_to_f32(static_cast<uint16_t>(x.x >> 16));
  o[2] = bf16_to_f32(static_cast<uint16_t>(x.y & 0xffffu));
  o[3] = bf16_to_f32(static_cast<uint16_t>(x.y >> 16));
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void score_kernel(
    const T* __restrict__ q, const float* __restrict__ ksum, const int* __restrict__ tables,
    const int* __restrict__ ctx_lens, float* __restrict__ zbuf, float* __restrict__ lse_part,
    int Hkv, int MAXB, int P, int nch, float scale, unsigned* flags) {
  constexpr int L = D / 4;
  constexpr int U = 64 / L;
  static_assert(G <= L, "heads per KV head exceed the lane group");
  extern __shared__ float zt[];              // [kScoreChunk][Hq]
  const int Hq = Hkv * G;
  const int ch = blockIdx.x, b = blockIdx.y;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;    // flagged by the select kernel
  const int nb = (N + kBlock - 1) / kBlock;
  const int j_lo = ch * kScoreChunk;
  if (j_lo >= nb) return;
  const int nblk = min(kScoreChunk, nb - j_lo);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int u = lane / L, li = lane % L;
  const int* trow = tables + static_cast<long long>(b) * MAXB;

  for (int gp = 0; gp * U < Hkv; ++gp) {
    const int g = gp * U + u;
    const bool gv = g < Hkv;
    float qv[G][4];
#pragma unroll
    for (int r = 0; r < G; ++r) {
      if (gv) {
        load_q4<T>(q + (static_cast<long long>(b) * Hq + g * G + r) * D + 4 * li, qv[r]);
      } else {
        qv[r][0] = qv[r][1] = qv[r][2] = qv[r][3] = 0.f;
      }
    }
    for (int i = wave; i < nblk; i += 4) {
      int p = trow[j_lo + i];
      if (p < 0 || p >= P) {
        if (lane == 0) raise_flag(flags, ENT_DEV_BAD_TABLE);
        p = 0;
      }
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f);
      if (gv) kv = *reinterpret_cast<const float4*>(ksum + (static_cast<long long>(p) * Hkv + g) * D + 4 * li);
      float a[G];
#pragma unroll
      for (int r = 0; r < G; ++r)
        a[r] = qv[r][0] * kv.x + qv[r][1] * kv.y + qv[r][2] * kv.z + qv[r][3] * kv.w;
      const float z = reduce_heads<G, L>(a, li) * scale;
      const int r = li / (L / G);
      if (gv && (li % (L / G)) == 0) zt[i * Hq + g * G + r] = z;
    }
  }
  __syncthreads();
  float* zrow = zbuf + (static_cast<long long>(b) * MAXB + j_lo) * Hq;
  for (int e = threadIdx.x; e < nblk * Hq; e += kThreads) zrow[e] = zt[e];
  // Per-head log-sum-exp of l = z + ln n_b over this chunk's blocks.
  const float ln_last = logf(static_cast<float>(N - kBlock * (nb - 1)));
  const float ln_full = logf(static_cast<float>(kBlock));
  for (int h = threadIdx.x; h < Hq; h += kThreads) {
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
    float* lp = lse_part + ((static_cast<long long>(b) * nch + ch) * Hq + h) * 2;
    lp[0] = m;
    lp[1] = s;
  }
}

__device__ __forceinline__ unsigned float_key(float f) {
  const unsigned u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Budget k in float32, operation by operation (no contraction), so that the
// integer matches a float32 evaluation of the same formula elsewhere.
__device__ __forceinline__ int keep_budget(float h, int nb, float eps_h, float h_min,
                                           float log_v, float kappa_min, int b_min) {
  if (nb <= 0) return 0;
  const float hg = fmaxf(__fadd_rn(h, eps_h), h_min);
  float u = __fdiv_rn(__fsub_rn(hg, h_min), __fsub_rn(log_v, h_min));
  u = fminf(fmaxf(u, 0.f), 1.f);
  const float kappa = __fadd_rn(kappa_min, __fmul_rn(__fsub_rn(1.f, kappa_min), u));
  const int k = static_cast<int>(ceilf(__fmul_rn(kappa, static_cast<float>(nb))));
  return min(nb, max(min(b_min, nb), k));
}

__global__ __launch_bounds__(kThreads) void select_kernel(
    const float* __restrict__ zbuf, const float* __restrict__ lse_part,
    const int* __restrict__ ctx_lens, const float* __restrict__ hvec,
    float* __restrict__ score_ws, float* __restrict__ scores_out, float* __restrict__ theta_out,
    int* __restrict__ kept, int* __restrict__ n_kept, unsigned* __restrict__ ticket,
    int Hq, int MAXB, int nch_max, float eps_h, float h_min, float log_v, float kappa_min,
    int b_min, unsigned* flags) {
  extern __shared__ unsigned keys[];        // [MAXB] (also holds L_h before selection)
  __shared__ unsigned hist[256];
  __shared__ int s_last, s_digit, s_krem, s_wcnt[4];
  __shared__ float sL[128];
  const int ch = blockIdx.x, b = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) {
    if (ch == 0 && t == 0) {
      raise_flag(flags, ENT_DEV_BAD_CTXLEN);
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return;
  }
  const int nb = (N + kBlock - 1) / kBlock;
  if (nb == 0) {
    if (ch == 0 && t == 0) {
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return;
  }
  const int j_lo = ch * kScoreChunk;
  if (j_lo >= nb) return;
  const int nblk = min(kScoreChunk, nb - j_lo);
  const int nch = (nb + kScoreChunk - 1) / kScoreChunk;

  // L_h = ln sum_b n_b e^{z_bh}, merged from the per-chunk partials.
  for (int h = t; h < Hq; h += kThreads) {
    const float* lp = lse_part + (static_cast<long long>(b) * nch_max * Hq + h) * 2;
    float m = -INFINITY;
    for (int c = 0; c < nch; ++c) m = fmaxf(m, lp[c * Hq * 2]);
    float s = 0.f;
    for (int c = 0; c < nch; ++c) s += lp[c * Hq * 2 + 1] * expf(lp[c * Hq * 2] - m);
    sL[h] = m + logf(s);
  }
  __syncthreads();

  // Scores of this chunk's blocks: 4 threads per block, heads strided by 4.
  const float ln_last = logf(static_cast<float>(N - kBlock * (nb - 1)));
  const float ln_full = logf(static_cast<float>(kBlock));
  {
    const int i = t >> 2, q4 = t & 3;
    float acc = 0.f;
    if (i < nblk) {
      const float lnn = (j_lo + i == nb - 1) ? ln_last : ln_full;
      const float* zr = zbuf + (static_cast<long long>(b) * MAXB + j_lo + i) * Hq;
      for (int h = q4; h < Hq; h += 4) {
        const float z = zr[h];
        const float Lh = sL[h];
        acc += expf(z + lnn - Lh) * (Lh - z);
      }
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    if (i < nblk && q4 == 0) {
      const float I = __fdiv_rn(acc, static_cast<float>(Hq));
      score_ws[static_cast<long long>(b) * MAXB + j_lo + i] = I;
      if (scores_out) scores_out[static_cast<long long>(b) * MAXB + j_lo + i] = I;
    }
  }

  // The last workgroup of this sequence selects.
  __syncthreads();
  if (t == 0) {
    __threadfence();
    const unsigned prev = atomicAdd(&ticket[b], 1u);
    s_last = (prev == static_cast<unsigned>(nch - 1));
    if (s_last) __threadfence();
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  const int k = keep_budget(hvec[b], nb, eps_h, h_min, log_v, kappa_min, b_min);
  for (int i = t; i < nb; i += kThreads)
    keys[i] = float_key(score_ws[static_cast<long long>(b) * MAXB + i]);
  if (t == 0) s_krem = k;
  __syncthreads();

  unsigned prefix = 0u, mask = 0u;
  if (k > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      hist[t] = 0u;
      __syncthreads();
      for (int i = t; i < nb; i += kThreads) {
        const unsigned key = keys[i];
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        // Bins 4*lane .. 4*lane+3; suffix sums over lanes locate the digit
        // holding the k_rem-th largest remaining key.
        const unsigned c0 = hist[4 * lane], c1 = hist[4 * lane + 1], c2 = hist[4 * lane + 2],
                       c3 = hist[4 * lane + 3];
        const unsigned cl = c0 + c1 + c2 + c3;
        unsigned suf = cl;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const unsigned n = __shfl_down(suf, o);
          if (lane + o < 64) suf += n;
        }
        const unsigned krem = static_cast<unsigned>(s_krem);
        const unsigned above = suf - cl;     // keys in higher lanes' bins
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
          s_digit = d;
          s_krem = static_cast<int>(krem - run);
        }
      }
      __syncthreads();
      prefix |= static_cast<unsigned>(s_digit) << shift;
      mask |= 255u << shift;
      __syncthreads();
    }
  }
  const unsigned tkey = prefix;

  // Compaction in ascending block order.
  int total = 0;
  int* krow = kept + static_cast<long long>(b) * MAXB;
  if (k > 0) {
    for (int base = 0; base < nb; base += kThreads) {
      const int i = base + t;
      const bool f = i < nb && keys[i] >= tkey;
      const unsigned long long bal = __ballot(f);
      const int rank = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) s_wcnt[wave] = __popcll(bal);
      __syncthreads();
      int off = total;
      for (int w = 0; w < wave; ++w) off += s_wcnt[w];
      if (f) krow[off + rank] = i;
      total += s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
      __syncthreads();
    }
  }
  if (t == 0) {
    n_kept[b] = total;
    if (theta_out) theta_out[b] = (k > 0) ? key_float(tkey) : INFINITY;
    ticket[b] = 0u;
  }
}

template <typename T, int D>
hipError_t launch_score_d(const ent_ctx* c, int B, const void* q, const float* ksum,
                          const int* tables, const int* ctx_lens, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid(c->score_chunks, B);
  const size_t lds = static_cast<size_t>(kScoreChunk) * cf.num_q_heads * sizeof(float);
  const T* qq = static_cast<const T*>(q);
#define ENT_SCORE_CASE(GG)                                                                     \
  case GG:                                                                                     \
    hipLaunchKernelGGL((score_kernel<T, D, GG>), grid, dim3(kThreads), lds, s, qq, ksum, tables, \
                       ctx_lens, c->zbuf, c->lse_part, cf.num_kv_heads, cf.max_blocks_per_seq,   \
                       cf.num_pool_blocks, c->score_chunks, cf.scale, c->dev_flags);           \
    break;
  switch (c->group) {
    ENT_SCORE_CASE(1)
    ENT_SCORE_CASE(2)
    ENT_SCORE_CASE(4)
    ENT_SCORE_CASE(8)
    ENT_SCORE_CASE(16)
    default:
      return hipErrorInvalidValue;
  }
#undef ENT_SCORE_CASE
  return hipGetLastError();
}

}  // namespace

hipError_t launch_block_summary(const ent_ctx* c, int B, const void* k_cache, const int* tables,
                                const int* ctx_lens, float* ksum, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid(cf.max_blocks_per_seq, B);
  if (cf.kv_dtype == ENT_BF16)
    hipLaunchKernelGGL(summary_kernel<uint16_t>, grid, dim3(kThreads), 0, s,
                       static_cast<const uint16_t*>(k_cache), tables, ctx_lens, ksum,
                       cf.num_kv_heads, cf.head_dim, cf.max_blocks_per_seq, cf.num_pool_blocks,
                       c->dev_flags);
  else
    hipLaunchKernelGGL(summary_kernel<float>, grid, dim3(kThreads), 0, s,
                       static_cast<const float*>(k_cache), tables, ctx_lens, ksum,
                       cf.num_kv_heads, cf.head_dim, cf.max_blocks_per_seq, cf.num_pool_blocks,
                       c->dev_flags);
  return hipGetLastError();
}

hipError_t launch_block_select(const ent_ctx* c, int B, const void* q, const float* ksum,
                               const int* tables, const int* ctx_lens, const float* h, int* kept,
                               int* n_kept, float* scores, float* theta, hipStream_t s) {
  const ent_config& cf = c->cfg;
  hipError_t e;
  if (cf.kv_dtype == ENT_BF16)
    e = cf.head_dim == 128 ? launch_score_d<uint16_t, 128>(c, B, q, ksum, tables, ctx_lens, s)
                           : launch_score_d<uint16_t, 64>(c, B, q, ksum, tables, ctx_lens, s);
  else
    e = cf.head_dim == 128 ? launch_score_d<float, 128>(c, B, q, ksum, tables, ctx_lens, s)
                           : launch_score_d<float, 64>(c, B, q, ksum, tables, ctx_lens, s);
  if (e != hipSuccess) return e;
  const size_t lds = static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned);
  hipLaunchKernelGGL(select_kernel, dim3(c->score_chunks, B), dim3(kThreads), lds, s, c->zbuf,
                     c->lse_part, ctx_lens, h, c->score_ws, scores, theta, kept, n_kept,
                     c->sel_ticket, cf.num_q_heads, cf.max_blocks_per_seq, c->score_chunks,
                     cf.eps_h, cf.h_min, cf.log_v, cf.kappa_min, cf.b_min, c->dev_flags);
  return hipGetLastError();
}

hipError_t launch_kv_append(const ent_ctx* c, int B, const void* k_new, const void* v_new,
                            const int* tables, int* ctx_lens, void* k_cache, void* v_cache,
                            float* ksum, hipStream_t s) {
  const ent_config& cf = c->cfg;
  if (cf.kv_dtype == ENT_BF16)
    hipLaunchKernelGGL(append_kernel<uint16_t>, dim3(B), dim3(kThreads), 0, s,
                       static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                       tables, ctx_lens, static_cast<uint16_t*>(k_cache),
                       static_cast<uint16_t*>(v_cache), ksum, cf.num_kv_heads, cf.head_dim,
                       cf.max_blocks_per_seq, cf.num_pool_blocks, c->dev_flags);
  else
    hipLaunchKernelGGL(append_kernel<float>, dim3(B), dim3(kThreads), 0, s,
                       static_cast<const float*>(k_new), static_cast<const float*>(v_new), tables,
                       ctx_lens, static_cast<float*>(k_cache), static_cast<float*>(v_cache), ksum,
                       cf.num_kv_heads, cf.head_dim, cf.max_blocks_per_seq, cf.num_pool_blocks,
                       c->dev_flags);
  return hipGetLastError();
}

}  // namespace ent
