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
//   score_kernel        z for 16 blocks x all heads per workgroup
//   select_kernel       per sequence: the per-head log-sum-exp L_h, computes
//                       I_b, the budget, a 4-pass 8-bit radix select of the
//                       k-th largest score, ascending compaction with ballots
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
// Scoring.  A workgroup of 4 waves takes 16 blocks of one sequence, 4 per
// wave, and writes z_bh = scale <q_h, kbar_b,g(h)> for all of them.  The
// critical path is two memory round trips: the wave's table entries and the
// query heads (staged once in LDS as fp32) are loaded together, then all
// summary loads of the wave's 4 blocks are in flight at once.  A block's
// summary (H_kv x d floats) is read as NP passes of 256 floats, one float4
// per lane per pass, fully coalesced.  In a pass, a group of L = d/4 lanes
// covers one KV head: each lane forms G partial dot products (one per query
// head of that KV head) and a halving butterfly reduces them over the L
// lanes, leaving head r = li * G / L in lane li.
// ---------------------------------------------------------------------------
constexpr int kScoreThreads = 256;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kScorePerWave = kScoreChunk / kScoreWaves;   // 4 blocks per wave

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

template <typename T, int D, int G, int kMaxPasses>   // np <= kMaxPasses
__global__ __launch_bounds__(kScoreThreads) void score_kernel(
    const T* __restrict__ q, const float* __restrict__ ksum, const int* __restrict__ tables,
    const int* __restrict__ ctx_lens, float* __restrict__ zbuf, int Hkv, int MAXB, int P,
    float scale, unsigned* flags) {
  constexpr int L = D / 4;
  static_assert(G <= L, "heads per KV head exceed the lane group");
  extern __shared__ float smem[];            // q [Hq][D] fp32, then z tile [kScoreChunk][Hq]
  const int Hq = Hkv * G;
  float* qs = smem;
  float* zt = smem + Hq * D;
  const int ch = blockIdx.x, b = blockIdx.y;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int li = lane % L;
  const int j_lo = ch * kScoreChunk;
  const int jw = j_lo + wave * kScorePerWave;
  // Table entries are read before the context length is known (the row has
  // MAXB entries, so the read is in bounds); invalid ones are masked below.
  int my_p = 0;
  if (lane < kScorePerWave && jw + lane < MAXB) my_p = tables[static_cast<long long>(b) * MAXB + jw + lane];
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) return;    // flagged by the selection kernel
  const int nb = (N + kBlock - 1) / kBlock;
  if (j_lo >= nb) return;
  const int nblk = min(kScoreChunk, nb - j_lo);
  const int nmine = max(0, min(kScorePerWave, nb - jw));
  if (lane < nmine && (my_p < 0 || my_p >= P)) {
    raise_flag(flags, ENT_DEV_BAD_TABLE);
    my_p = 0;
  }
  if (lane >= nmine) my_p = 0;
  const int nfl = Hkv * D;
  const int np = (nfl + 255) >> 8;

  float4 kv[kScorePerWave][kMaxPasses];
#pragma unroll
  for (int blk = 0; blk < kScorePerWave; ++blk) {
    const int p = __shfl(my_p, blk);
#pragma unroll
    for (int k = 0; k < kMaxPasses; ++k) {
      const int f = 256 * k + 4 * lane;
      if (blk < nmine && k < np && f < nfl)
        kv[blk][k] = *reinterpret_cast<const float4*>(ksum + static_cast<long long>(p) * nfl + f);
      else
        kv[blk][k] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  for (int e = t; e < Hq * D; e += kScoreThreads)
    qs[e] = load_elem<T>(q + static_cast<long long>(b) * Hq * D + e);
  __syncthreads();

#pragma unroll
  for (int blk = 0; blk < kScorePerWave; ++blk) {
    if (blk >= nmine) continue;
#pragma unroll
    for (int k = 0; k < kMaxPasses; ++k) {
      if (k >= np) continue;
      const int f = 256 * k + 4 * lane;
      const bool gv = f < nfl;
      const int g = f / D, dd = f % D;
      float a[G];
#pragma unroll
      for (int r = 0; r < G; ++r) {
        float4 qq = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gv) qq = *reinterpret_cast<const float4*>(qs + (g * G + r) * D + dd);
        a[r] = qq.x * kv[blk][k].x + qq.y * kv[blk][k].y + qq.z * kv[blk][k].z +
               qq.w * kv[blk][k].w;
      }
      const float z = reduce_heads<G, L>(a, li) * scale;
      if (gv && (li % (L / G)) == 0)
        zt[(wave * kScorePerWave + blk) * Hq + g * G + li / (L / G)] = z;
    }
    // Keep the next block's LDS reads from being hoisted above this point.
    asm volatile("" ::: "memory");
  }
  __syncthreads();
  float* zrow = zbuf + (static_cast<long long>(b) * MAXB + j_lo) * Hq;
  for (int e = t; e < nblk * Hq; e += kScoreThreads) zrow[e] = zt[e];
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

// Kept set of one sequence (one workgroup of 512 threads):
//  1. L_h = ln sum_b n_b e^{z_bh}, from the block logits z;
//  2. I_b = (1/H_q) sum_h e^{z_bh + ln n_b - L_h} (L_h - z_bh) for every block,
//     held in LDS as order-preserving integer keys;
//  3. budget k from the entropy, the k-th largest key by a 4-pass 8-bit radix
//     select, and ascending compaction of {b : I_b >= theta} with wave ballots.
constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / 64;

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const float* __restrict__ zbuf, const int* __restrict__ ctx_lens,
    const float* __restrict__ hvec, float* __restrict__ scores_out,
    float* __restrict__ theta_out, int* __restrict__ kept, int* __restrict__ n_kept, int Hq,
    int MAXB, float eps_h, float h_min,
    float log_v, float kappa_min, int b_min, unsigned* flags) {
  extern __shared__ unsigned keys[];        // [MAXB]
  __shared__ unsigned hist[256];
  __shared__ float s_pm[kSelThreads], s_ps[kSelThreads], sL[128];
  __shared__ int s_digit, s_krem, s_wcnt[kSelWaves];
  const int b = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int N = ctx_lens[b];
  if (N < 0 || N > MAXB * kBlock) {
    if (t == 0) {
      raise_flag(flags, ENT_DEV_BAD_CTXLEN);
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return;
  }
  const int nb = (N + kBlock - 1) / kBlock;
  const int k = keep_budget(hvec[b], nb, eps_h, h_min, log_v, kappa_min, b_min);
  if (nb == 0) {
    if (t == 0) {
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return;
  }
  // 1. L_h = ln sum_b n_b e^{z_bh}: each thread folds, online, a strided
  //    subset of the blocks for head t % Hq; one thread per head folds the
  //    subsets.
  const float ln_last = logf(static_cast<float>(N - kBlock * (nb - 1)));
  const float ln_full = logf(static_cast<float>(kBlock));
  const float* zb = zbuf + static_cast<long long>(b) * MAXB * Hq;
  const int per_head = kSelThreads / Hq;     // threads per head (Hq <= 128)
  {
    float m = -INFINITY, sum = 0.f;
    if (t < per_head * Hq) {
      const int h = t % Hq;
      for (int j = t / Hq; j < nb; j += per_head) {
        const float l = zb[static_cast<long long>(j) * Hq + h] + ((j == nb - 1) ? ln_last : ln_full);
        if (l > m) {
          sum = sum * expf(m - l) + 1.f;
          m = l;
        } else {
          sum += expf(l - m);
        }
      }
    }
    s_pm[t] = m;
    s_ps[t] = sum;
  }
  __syncthreads();
  if (t < Hq) {
    float m = -INFINITY, sum = 0.f;
    for (int i = 0; i < per_head; ++i) {
      const float mc = s_pm[i * Hq + t], sc = s_ps[i * Hq + t];
      if (mc == -INFINITY) continue;
      const float mn = fmaxf(m, mc);
      sum = sum * expf(m - mn) + sc * expf(mc - mn);
      m = mn;
    }
    sL[t] = m + logf(sum);
  }
  __syncthreads();

  // 2. Block scores.
  for (int j = t; j < nb; j += kSelThreads) {
    const float lnn = (j == nb - 1) ? ln_last : ln_full;
    const float* zr = zb + static_cast<long long>(j) * Hq;
    float acc = 0.f;
    for (int h = 0; h < Hq; ++h) {
      const float z = zr[h];
      const float Lh = sL[h];
      acc += expf(z + lnn - Lh) * (Lh - z);
    }
    const float I = __fdiv_rn(acc, static_cast<float>(Hq));
    keys[j] = float_key(I);
    if (scores_out) scores_out[static_cast<long long>(b) * MAXB + j] = I;
  }
  if (k <= 0) {
    if (t == 0) {
      n_kept[b] = 0;
      if (theta_out) theta_out[b] = INFINITY;
    }
    return;
  }
  if (t == 0) s_krem = k;
  __syncthreads();

  // 3. Radix select of the k-th largest key.
  unsigned prefix = 0u, mask = 0u;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (t < 256) hist[t] = 0u;
    __syncthreads();
    for (int i = t; i < nb; i += kSelThreads) {
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
        s_digit = d;
        s_krem = static_cast<int>(krem - run);
      }
    }
    __syncthreads();
    prefix |= static_cast<unsigned>(s_digit) << shift;
    mask |= 255u << shift;
    __syncthreads();
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
    if (lane == 0) s_wcnt[wave] = __popcll(bal);
    __syncthreads();
    int off = total;
    for (int w = 0; w < wave; ++w) off += s_wcnt[w];
    if (f) krow[off + rank] = i;
    for (int w = 0; w < kSelWaves; ++w) total += s_wcnt[w];
    __syncthreads();
  }
  if (t == 0) {
    n_kept[b] = total;
    if (theta_out) theta_out[b] = key_float(tkey);
  }
}

template <typename T, int D>
hipError_t launch_score_d(const ent_ctx* c, int B, const void* q, const float* ksum,
                          const int* tables, const int* ctx_lens, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid(c->score_chunks, B);
  const size_t lds = (static_cast<size_t>(cf.num_q_heads) * D +
                      static_cast<size_t>(kScoreChunk) * cf.num_q_heads) * sizeof(float);
  const T* qq = static_cast<const T*>(q);
  const int np = (cf.num_kv_heads * D + 255) / 256;
#define ENT_SCORE_CASE(GG)                                                                      \
  case GG:                                                                                      \
    if (np <= 4)                                                                                \
      hipLaunchKernelGGL((score_kernel<T, D, GG, 4>), grid, dim3(kScoreThreads), lds, s, qq,    \
                         ksum, tables, ctx_lens, c->zbuf, cf.num_kv_heads,                      \
                         cf.max_blocks_per_seq, cf.num_pool_blocks, cf.scale, c->dev_flags);    \
    else                                                                                        \
      hipLaunchKernelGGL((score_kernel<T, D, GG, 8>), grid, dim3(kScoreThreads), lds, s, qq,    \
                         ksum, tables, ctx_lens, c->zbuf, cf.num_kv_heads,                      \
                         cf.max_blocks_per_seq, cf.num_pool_blocks, cf.scale, c->dev_flags);    \
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
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(kSelThreads), lds, s, c->zbuf, ctx_lens, h,
                     scores, theta, kept, n_kept, cf.num_q_heads, cf.max_blocks_per_seq, cf.eps_h, cf.h_min, cf.log_v, cf.kappa_min, cf.b_min,
                     c->dev_flags);
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
