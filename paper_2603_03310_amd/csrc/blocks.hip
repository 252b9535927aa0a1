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
//   (bf16 scoring runs in the persistent kernel of prologue.hip)
//   score_valu_kernel   z for 16 blocks x all heads per workgroup (fp32, VALU)
//   select_fused_kernel per sequence (tables that fit its registers): L_h, I_b, the
//                       budget, an 8-bit radix select of the k-th largest
//                       score, ascending compaction with ballots
//   lse_merge_kernel,   the same in three launches for long block tables
//   block_score_kernel, (the per-stage entry point): per sequence L_h; per 64
//   select_kernel       blocks I_b; per sequence the selection (the fused step
//                       runs L_h and I_b per 256-block tile in one launch,
//                       step.hip, with the selection on each sequence's last
//                       workgroup or in select_kernel after it)
//   append_kernel    writes one token and refreshes its block's mean key

#include "blocks_dev.h"

namespace ent {
namespace {

constexpr int kThreads = 256;

// A block's mean key is the sum of its valid slots in slot order, divided by
// their number (correctly rounded): the summary and append kernels both
// evaluate it so, and give the same bits.

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
  // Each thread takes VE consecutive elements of one KV head's row: the 16
  // slots' 16-byte loads are all issued at once (slots past n are read and
  // not used: the tile always holds 16), then each element is summed in slot
  // order.
  constexpr int VE = 16 / sizeof(T);
  for (int v = threadIdx.x; v < Hkv * D / VE; v += kThreads) {
    const int e0 = v * VE;
    const int g = e0 / D, dd = e0 % D;
    const long long tile = (static_cast<long long>(p) * Hkv + g) * kBlock * D;
    uint4 raw[kBlock];
#pragma unroll
    for (int slot = 0; slot < kBlock; ++slot)
      raw[slot] = *reinterpret_cast<const uint4*>(kc + tile + slot * D + dd);
    float sum[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) sum[i] = 0.f;
#pragma unroll
    for (int slot = 0; slot < kBlock; ++slot) {
      const T* x = reinterpret_cast<const T*>(&raw[slot]);
      if (slot < n) {
#pragma unroll
        for (int i = 0; i < VE; ++i) sum[i] += load_elem<T>(x + i);
      }
    }
    float* out = ksum + (static_cast<long long>(p) * Hkv + g) * D + dd;
#pragma unroll
    for (int i = 0; i < VE; ++i) out[i] = __fdiv_rn(sum[i], static_cast<float>(n));
  }
}

template <typename T>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(AppendArgs a) {
  append_body<T>(a, blockIdx.x);
}

// Per-stage kernels over the shared bodies.
template <int D, int G>
__global__ __launch_bounds__(kScoreThreads) void score_valu_kernel(
    const float* __restrict__ q, const float* __restrict__ ksum, const int* __restrict__ tables,
    const int* __restrict__ ctx_lens, float* __restrict__ zbuf, float* __restrict__ lse_part,
    int Hkv, int MAXB, int P, int nch_max, float scale, unsigned* flags) {
  extern __shared__ float smem[];
  score_valu_body<D, G>(q, ksum, tables, ctx_lens, zbuf, lse_part, Hkv, MAXB, P, nch_max, scale,
                        flags, blockIdx.x, blockIdx.y, smem);
}

__global__ __launch_bounds__(kFoldThreads) void lse_merge_kernel(
    const float* __restrict__ lse_part, const int* __restrict__ ctx_lens, float* __restrict__ L,
    int Hq, int MAXB, int nch_max) {
  __shared__ float s_pm[kFoldThreads], s_ps[kFoldThreads];
  lse_merge_body(lse_part, ctx_lens, L + static_cast<long long>(blockIdx.x) * Hq, Hq, MAXB, nch_max,
                 blockIdx.x, s_pm, s_ps);
}

__global__ __launch_bounds__(kRowThreads) void block_score_kernel(
    const float* __restrict__ zbuf, const float* __restrict__ L, const int* __restrict__ ctx_lens,
    float* __restrict__ scores, int Hq, int MAXB) {
  __shared__ float sL[128];
  block_score_body(zbuf, L, ctx_lens, scores, Hq, MAXB, blockIdx.y, blockIdx.x * kTileBlocks, sL);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const float* __restrict__ scores, const int* __restrict__ ctx_lens,
    const int* __restrict__ tables, const float* __restrict__ hvec, float* __restrict__ theta_out,
    int* __restrict__ kept, int* __restrict__ kphys, int* __restrict__ n_kept, int MAXB, int P,
    Budget bu, unsigned* flags) {
  extern __shared__ unsigned keys[];        // [MAXB] keys, then [MAXB] encoded blocks
  __shared__ SelectShared sh;
  const int b = blockIdx.x;
  select_row_body(scores, ctx_lens, tables, hvec[b], theta_out, kept, kphys, n_kept, MAXB, P, bu,
                  flags, b, keys, reinterpret_cast<int*>(keys + MAXB), sh);
}

// All three selection steps per sequence (short block tables).
template <int F4>
__global__ __launch_bounds__(kSelThreads) void select_fused_kernel(
    const float* __restrict__ zbuf, const float* __restrict__ lse_part,
    const int* __restrict__ ctx_lens, const int* __restrict__ tables,
    const float* __restrict__ hvec, float* __restrict__ scores, float* __restrict__ theta_out,
    int* __restrict__ kept, int* __restrict__ kphys, int* __restrict__ n_kept, int MAXB, int P,
    int nch_max, int Hq, Budget bu, unsigned* flags) {
  extern __shared__ unsigned keys[];        // [MAXB] keys, then [MAXB] encoded blocks
  __shared__ SelectShared sh;
  const int b = blockIdx.x;
  select_fused_body<F4>(zbuf, lse_part, ctx_lens, tables, hvec[b], scores, theta_out, kept, kphys,
                        n_kept, MAXB, P, nch_max, Hq, bu, flags, b, keys,
                        reinterpret_cast<int*>(keys + MAXB), sh);
}

template <int D>
hipError_t launch_score_valu_d(const ent_ctx* c, int B, const float* q, const float* ksum,
                               const int* tables, const int* ctx_lens, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const int Hq = cf.num_q_heads;
  const dim3 grid((cf.max_blocks_per_seq + kValuChunk - 1) / kValuChunk, B);
  const size_t lds = (static_cast<size_t>(Hq) * D + static_cast<size_t>(kValuChunk) * Hq) * sizeof(float);
#define ENT_SCORE_CASE(GG)                                                                    \
  case GG:                                                                                    \
    hipLaunchKernelGGL((score_valu_kernel<D, GG>), grid, dim3(kScoreThreads), lds, s, q,      \
                       ksum, tables, ctx_lens, c->zbuf, c->lse_part, cf.num_kv_heads,         \
                       cf.max_blocks_per_seq, cf.num_pool_blocks, c->lse_chunks, cf.scale,    \
                       c->dev_flags);                                                         \
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

hipError_t launch_score_valu(const ent_ctx* c, int B, const void* q, const float* ksum,
                             const int* tables, const int* ctx_lens, hipStream_t s) {
  const float* qq = static_cast<const float*>(q);
  return c->cfg.head_dim == 128 ? launch_score_valu_d<128>(c, B, qq, ksum, tables, ctx_lens, s)
                                : launch_score_valu_d<64>(c, B, qq, ksum, tables, ctx_lens, s);
}

Budget make_budget(const ent_config& cf, float* kappa) {
  Budget bu;
  bu.eps_h = cf.eps_h;
  bu.h_min = cf.h_min;
  bu.log_v = cf.log_v;
  bu.kappa_min = cf.kappa_min;
  bu.dkappa = cf.dkappa;
  bu.b_min = cf.b_min;
  bu.keep_first = cf.keep_first;
  bu.keep_last = cf.keep_last;
  bu.kappa = kappa;
  return bu;
}

hipError_t launch_block_select(const ent_ctx* c, int B, const void* q, const float* ksum,
                               const void* k_cache, const int* tables, const int* ctx_lens,
                               const float* h, int* kept, int* n_kept, float* scores,
                               float* theta, float* kappa, hipStream_t s) {
  const ent_config& cf = c->cfg;
  hipError_t e;
  if (cf.scoring == ENT_SCORE_EXACT) {
    // Exact token-level weights: per-block triples from one pass over K,
    // then the selection's three phases with the exact block scores.
    e = launch_exact_scores(c, B, q, k_cache, tables, ctx_lens, s);
    if (e != hipSuccess) return e;
    e = launch_lse_merge(c, B, ctx_lens, s);
    if (e != hipSuccess) return e;
    float* sc = scores ? scores : c->iscores;
    e = launch_exact_block_scores(c, B, ctx_lens, sc, s);
    if (e != hipSuccess) return e;
    return launch_select_rows(c, B, tables, ctx_lens, h, sc, theta, kept, n_kept, kappa, s);
  }
  if (cf.kv_dtype == ENT_BF16) {
    PrologueArgs a{};
    a.B = B;
    a.do_score = 1;
    a.q = static_cast<const uint16_t*>(q);
    a.ksum = ksum;
    a.tables = tables;
    a.ctx_lens = ctx_lens;
    a.zbuf = c->zbuf;
    a.lse_part = c->lse_part;
    a.Hkv = cf.num_kv_heads;
    a.G = c->group;
    a.MAXB = cf.max_blocks_per_seq;
    a.P = cf.num_pool_blocks;
    a.nch_max = c->lse_chunks;
    a.scale = cf.scale;
    a.flags = c->dev_flags;
    e = launch_prologue(c, a, s);
  } else {
    e = launch_score_valu(c, B, q, ksum, tables, ctx_lens, s);
  }
  if (e != hipSuccess) return e;
  return launch_selection(c, B, tables, ctx_lens, h, scores, theta, kept, n_kept, kappa, s);
}

hipError_t launch_selection(const ent_ctx* c, int B, const int* tables, const int* ctx_lens,
                            const float* h, float* scores, float* theta, int* kept, int* n_kept,
                            float* kappa, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const Budget bu = make_budget(cf, kappa);
  const size_t lds = static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned);
  const int form = select_one_launch(cf.max_blocks_per_seq, cf.num_q_heads);
  if (form) {
    const size_t lds = 2 * static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned);
#define ENT_SEL_LAUNCH(FF)                                                                      \
  hipLaunchKernelGGL((select_fused_kernel<FF>), dim3(B), dim3(kSelThreads), lds, s, c->zbuf,     \
                     c->lse_part, ctx_lens, tables, h, scores, theta, kept, c->kept_phys,        \
                     n_kept, cf.max_blocks_per_seq, cf.num_pool_blocks, c->lse_chunks,           \
                     cf.num_q_heads, bu, c->dev_flags)
    switch (form) {
      case 1: ENT_SEL_LAUNCH(1); break;
      case 2: ENT_SEL_LAUNCH(2); break;
      case 4: ENT_SEL_LAUNCH(4); break;
      case 8: ENT_SEL_LAUNCH(8); break;
      default: return hipErrorInvalidValue;
    }
#undef ENT_SEL_LAUNCH
    return hipGetLastError();
  }
  hipError_t e = launch_lse_merge(c, B, ctx_lens, s);
  if (e != hipSuccess) return e;
  float* sc = scores ? scores : c->iscores;
  e = launch_block_scores(c, B, ctx_lens, sc, s);
  if (e != hipSuccess) return e;
  return launch_select_rows(c, B, tables, ctx_lens, h, sc, theta, kept, n_kept, kappa, s);
}

hipError_t launch_lse_merge(const ent_ctx* c, int B, const int* ctx_lens, hipStream_t s) {
  const ent_config& cf = c->cfg;
  hipLaunchKernelGGL(lse_merge_kernel, dim3(B), dim3(kFoldThreads), 0, s, c->lse_part, ctx_lens,
                     c->lrow, cf.num_q_heads, cf.max_blocks_per_seq, c->lse_chunks);
  return hipGetLastError();
}

hipError_t launch_block_scores(const ent_ctx* c, int B, const int* ctx_lens, float* scores,
                               hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid((cf.max_blocks_per_seq + kTileBlocks - 1) / kTileBlocks, B);
  hipLaunchKernelGGL(block_score_kernel, grid, dim3(kRowThreads), 0, s, c->zbuf, c->lrow, ctx_lens,
                     scores, cf.num_q_heads, cf.max_blocks_per_seq);
  return hipGetLastError();
}

hipError_t launch_select_rows(const ent_ctx* c, int B, const int* tables, const int* ctx_lens,
                              const float* h, const float* scores, float* theta, int* kept,
                              int* n_kept, float* kappa, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const size_t lds = 2 * static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned);
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(kSelThreads), lds, s, scores, ctx_lens, tables,
                     h, theta, kept, c->kept_phys, n_kept, cf.max_blocks_per_seq,
                     cf.num_pool_blocks, make_budget(cf, kappa), c->dev_flags);
  return hipGetLastError();
}

AppendArgs make_append_args(const ent_ctx* c, const void* k_new, const void* v_new,
                            const int* tables, int* ctx_lens, void* k_cache, void* v_cache,
                            float* ksum) {
  const ent_config& cf = c->cfg;
  AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.tables = tables;
  a.ctx_lens = ctx_lens;
  a.kc = k_cache;
  a.vc = v_cache;
  a.ksum = ksum;
  a.Hkv = cf.num_kv_heads;
  a.D = cf.head_dim;
  a.MAXB = cf.max_blocks_per_seq;
  a.P = cf.num_pool_blocks;
  a.flags = c->dev_flags;
  a.bf16 = cf.kv_dtype == ENT_BF16;
  return a;
}

hipError_t launch_kv_append(const ent_ctx* c, int B, const void* k_new, const void* v_new,
                            const int* tables, int* ctx_lens, void* k_cache, void* v_cache,
                            float* ksum, hipStream_t s) {
  const AppendArgs a = make_append_args(c, k_new, v_new, tables, ctx_lens, k_cache, v_cache, ksum);
  if (a.bf16)
    hipLaunchKernelGGL(append_kernel<uint16_t>, dim3(B), dim3(kAppendThreads), 0, s, a);
  else
    hipLaunchKernelGGL(append_kernel<float>, dim3(B), dim3(kAppendThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ent
