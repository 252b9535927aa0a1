// One whole decode step (ent_decode_step).  Each launch runs
// the same device bodies as the per-stage entry points, so the results are
// bit-identical to calling ent_entropy_temperature, ent_block_select,
// ent_sparse_paged_decode and ent_sample in sequence:
//
//   A  block scoring and the entropy chunk passes in one persistent grid
//      (prologue.hip): both stream from HBM (block summaries, logits) and
//      do not depend on each other (fp32 queries: scoring is a second
//      launch, on the VALU); each row's T_t is recorded in temp_used;
//   B  one workgroup per sequence: the row's entropy from the chunk triples,
//      the controller update and the kept-block selection under the
//      entropy-driven budget; in the same launch, on workgroups of their
//      own, sampling at T_t (it needs only the row statistics of A, so it
//      runs on the CUs the per-sequence selection leaves idle).  For long
//      block tables: entropy and controller per sequence and, on workgroups
//      of their own, L_h and the block scores per tile of 256 blocks, each
//      sequence's selection on the last of its workgroups to finish (a
//      ticket per sequence); sampling moves to D;
//   C  kept-block decode attention;
//   D  the merge of split decode segments (and, on workgroups of their own,
//      ent_decode_step_append's append of the new token's K/V and, for long
//      block tables, the sampling).

#include "blocks_dev.h"
#include "estimate_dev.h"

#include <algorithm>

namespace ent {
namespace {

// Sampling of row b - B by a workgroup of the launch that runs the
// per-sequence stage (blockIdx.x >= B); every thread must call it.
template <bool VEC>
__device__ __forceinline__ void step_sample(const SampleArgs& sa, int b, SampleShared& sh) {
  const int tok = sample_body<VEC>(sa.logits, sa.ld, sa.V, sa.C, sa.stats, sa.temp_used[b] * sa.t_cal,
                                   sa.uniforms[b], b, sh);
  if (threadIdx.x == 0) sa.tokens[b] = tok;
}

// The ticket and, on the last workgroup of sequence seq, its selection.
__device__ __forceinline__ void step_b1_select(int seq, const int* __restrict__ ctx_lens,
                                            const float* h_out, const float* scores,
                                            const int* __restrict__ tables, float* theta,
                                            int* kept, int* kphys, int* n_kept, int MAXB, int P,
                                            Budget bu, unsigned* flags, unsigned* tickets,
                                            unsigned* dyn_lds) {
  __shared__ SelectShared ssel;
  __shared__ int s_last;
  const int N = ctx_lens[seq];
  const bool ok = N >= 0 && N <= MAXB * kBlock;
  const int nb = ok ? (N + kBlock - 1) / kBlock : 0;
  const unsigned parts = static_cast<unsigned>((nb + kStepTileBlocks - 1) / kStepTileBlocks) + 1u;
  __builtin_amdgcn_s_waitcnt(0);           // this wave's device-scope stores have completed
  __syncthreads();
  if (threadIdx.x == 0)
    s_last = __hip_atomic_fetch_add(tickets + seq, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             parts - 1;
  __syncthreads();
  if (!s_last) return;
  if (threadIdx.x == 0) tickets[seq] = 0u;
  const float hval = __hip_atomic_load(h_out + seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  select_row_body<true>(scores, ctx_lens, tables, hval, theta, kept, kphys, n_kept, MAXB, P, bu,
                        flags, seq, dyn_lds, reinterpret_cast<int*>(dyn_lds + MAXB), ssel);
}

// Block tables too wide for the one-launch selection: workgroups 0 .. B-1
// take a row's entropy from the chunk triples and the controller update (with
// an estimator, the estimate first), and the rest one (sequence, tile of
// kStepTileBlocks blocks) each: the sequence's L_h, merged as the per-stage
// launch merges it, then the tile's block scores.  Tiles past a sequence's
// blocks exit at once.  With TICK, each sequence's selection
// runs on whichever of its workgroups (the entropy one and those of its
// tiles with blocks) finishes last: each stores what the selection reads
// (the entropy, the scores) at device scope, waits for those stores, then
// takes a ticket from the sequence's device-scope counter; the one that
// takes the last ticket resets the counter and selects, as the per-stage
// selection launch does.  Nothing waits for another workgroup.  Without,
// the selection launch follows.  (Sampling runs in the merge launch of this
// form.)
template <bool VEC, bool TICK>
__global__ __launch_bounds__(kFoldThreads) void step_b1_kernel(
    int B, const float* __restrict__ part, int C, float* temp, float* h_prev, float* tau,
    float* h_out, Control ct, const float* __restrict__ zbuf, const float* __restrict__ lse_part,
    const int* __restrict__ ctx_lens, float* __restrict__ scores, int Hq, int MAXB, int nch_max,
    int ntile, SampleArgs sa, int est, int est_k, const float* __restrict__ tmax,
    const int* __restrict__ tables, float* __restrict__ theta, int* __restrict__ kept,
    int* __restrict__ kphys, int* __restrict__ n_kept, int P, Budget bu, unsigned* flags,
    unsigned* tickets) {
  static_assert(kFoldThreads >= kEstThreads && kFoldThreads == kSelThreads, "workgroup size");
  // Estimator LDS, then (the selecting workgroup) the keys and encoded blocks.
  extern __shared__ __attribute__((aligned(16))) unsigned dyn_lds[];
  __shared__ float s_pm[kFoldThreads], s_ps[kFoldThreads], sL[128];
  __shared__ EstShared esh;
  int seq;
  if (blockIdx.x >= B) {
    const int r = blockIdx.x - B;
    seq = r / ntile;
    const int j0 = (r - seq * ntile) * kStepTileBlocks;
    const int N = ctx_lens[seq];
    if (N < 0 || N > MAXB * kBlock || j0 >= (N + kBlock - 1) / kBlock) return;   // no blocks
    lse_block_score_body<TICK>(zbuf, lse_part, ctx_lens, scores, Hq, MAXB, nch_max, seq, j0, s_pm,
                               s_ps, sL);
  } else {
    seq = blockIdx.x;
    if (est != ENT_EST_EXACT) {
      const float T = temp[seq];
      const float H = row_estimate(est, est_k, part, tmax, sa.logits, sa.ld, sa.V, C, T * sa.t_cal,
                                   seq, dyn_lds, esh);
      if (threadIdx.x == 0) controller_update(seq, H, T, h_prev, tau, temp, h_out, nullptr, ct);
    } else if (threadIdx.x < 64) {
      const float H = row_entropy(part, C, seq);
      if (threadIdx.x == 0) controller_update(seq, H, temp[seq], h_prev, tau, temp, h_out, nullptr, ct);
    }
    if constexpr (TICK)
      if (threadIdx.x == 0) __hip_atomic_store(h_out + seq, h_out[seq], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if constexpr (TICK)
    step_b1_select(seq, ctx_lens, h_out, scores, tables, theta, kept, kphys, n_kept, MAXB, P, bu,
                   flags, tickets, dyn_lds);
}

// Per sequence, block tables that fit the one-launch selection: the
// selection's loads are issued first, then the first wave computes the row's
// entropy and the controller update while they are in flight (with an
// estimator, the estimate comes first), then the whole kept-block selection;
// workgroups B .. 2B-1 sample.
template <int F4, bool VEC>
__global__ __launch_bounds__(kSelThreads) void step_b_kernel(
    int B, const float* __restrict__ part, int C, float* temp, float* h_prev, float* tau,
    float* h_out, Control ct, const float* __restrict__ zbuf, const float* __restrict__ lse_part,
    const int* __restrict__ ctx_lens, const int* __restrict__ tables, float* __restrict__ scores,
    float* __restrict__ theta, int* __restrict__ kept, int* __restrict__ kphys,
    int* __restrict__ n_kept, int MAXB, int P, int nch_max, int Hq, Budget bu, unsigned* flags,
    SampleArgs sa, int est, int est_k, const float* __restrict__ tmax) {
  static_assert(kSelThreads >= kSampleThreads && kSelThreads >= kEstThreads, "workgroup size");
  extern __shared__ __attribute__((aligned(16))) unsigned keys[];   // [MAXB] keys, [MAXB] blocks, estimator
  __shared__ SelectShared sh;
  __shared__ EstShared esh;
  __shared__ SampleShared ssh;
  __shared__ float s_H;
  const int b = blockIdx.x;
  if (b >= B) {
    step_sample<VEC>(sa, b - B, ssh);
    return;
  }
  SelectRegs<F4> R;
  if (est != ENT_EST_EXACT) {
    // The estimate needs most registers itself: the selection's loads follow it.
    const float T = temp[b];
    const float H = row_estimate(est, est_k, part, tmax, sa.logits, sa.ld, sa.V, C, T * sa.t_cal, b,
                                 keys + est_lds_offset(2 * MAXB), esh);
    if (threadIdx.x == 0) s_H = controller_update(b, H, T, h_prev, tau, temp, h_out, nullptr, ct);
    select_load<F4>(zbuf, lse_part, tables, MAXB, nch_max, b, Hq, R);
  } else {
    select_load<F4>(zbuf, lse_part, tables, MAXB, nch_max, b, Hq, R);
    if (threadIdx.x < 64) {
      const float H = row_entropy(part, C, b);
      if (threadIdx.x == 0)
        s_H = controller_update(b, H, temp[b], h_prev, tau, temp, h_out, nullptr, ct);
    }
  }
  const int N = ctx_lens[b];
  const float kprev = budget_prev(bu, b);
  const bool ok = N >= 0 && N <= MAXB * kBlock;
  const int nb = ok ? (N + kBlock - 1) / kBlock : 0;
  __syncthreads();
  const float H = s_H;
  int nb2, k;
  if (!select_prepare(N, H, theta, n_kept, MAXB, bu, kprev, flags, b, nb2, k)) return;
  select_finish<F4>(R, N, nb, H, scores, theta, kept, kphys, n_kept, MAXB, P, bu, kprev, b, Hq,
                    keys, reinterpret_cast<int*>(keys + MAXB), sh);
}
}  // namespace

// Dynamic LDS of the tile launch: the estimator's, and with the selection
// inside, at least the keys and encoded blocks of a table row.
static size_t step_b1_lds(const ent_ctx* c, bool tickets) {
  const ent_config& cf = c->cfg;
  const size_t est = uses_estimate(cf) ? est_lds_bytes(c->chunks, cf.est_k) : 0;
  return tickets ? std::max(est, 2 * static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned))
                 : est;
}

void step_occupancy(ent_ctx* c) {
  c->b1_occ_plain = 0;
  c->b1_occ_ticket = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&c->b1_occ_plain, step_b1_kernel<true, false>,
                                                   kFoldThreads, step_b1_lds(c, false)) != hipSuccess)
    c->b1_occ_plain = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&c->b1_occ_ticket, step_b1_kernel<true, true>,
                                                   kFoldThreads, step_b1_lds(c, true)) != hipSuccess)
    c->b1_occ_ticket = 0;
}

hipError_t launch_decode_step(const ent_ctx* c, int B, const float* logits, long long ld,
                              ent_state st, const void* q, const void* k_cache,
                              const void* v_cache, const float* ksum, const int* tables,
                              const int* ctx_lens, const float* uniforms, float* h_out,
                              float* temp_used, float* row_stats, int* kept, int* n_kept,
                              float* out, float* lse, int* tokens, float* scores, float* theta,
                              hipStream_t s, const AppendArgs* ap) {
  const ent_config& cf = c->cfg;
  float* stats = row_stats ? row_stats : c->stats_tmp;
  const bool bf16 = cf.kv_dtype == ENT_BF16;
  PrologueArgs pa{};
  pa.B = B;
  pa.do_entropy = 1;
  pa.logits = logits;
  pa.ld = ld;
  pa.V = cf.vocab;
  pa.C = c->chunks;
  pa.temp = st.temp;
  pa.t_cal = cf.t_cal;
  pa.part = c->ent_part;
  pa.row_stats = stats;
  pa.temp_used = temp_used;
  const bool est = uses_estimate(cf);
  const int est_mode = est ? cf.estimator : ENT_EST_EXACT;
  const size_t est_lds = est ? est_lds_bytes(c->chunks, cf.est_k) : 0;
  pa.tmax = est ? c->tmax : nullptr;
  pa.do_score = bf16 ? 1 : 0;
  pa.q = static_cast<const uint16_t*>(q);
  pa.ksum = ksum;
  pa.tables = tables;
  pa.ctx_lens = ctx_lens;
  pa.zbuf = c->zbuf;
  pa.lse_part = c->lse_part;
  pa.Hkv = cf.num_kv_heads;
  pa.G = c->group;
  pa.MAXB = cf.max_blocks_per_seq;
  pa.P = cf.num_pool_blocks;
  pa.nch_max = c->lse_chunks;
  pa.scale = cf.scale;
  pa.flags = c->dev_flags;
  hipError_t e = launch_prologue(c, pa, s);
  if (e != hipSuccess) return e;
  if (!bf16) {
    e = launch_score_valu(c, B, q, ksum, tables, ctx_lens, s);
    if (e != hipSuccess) return e;
  }

  SampleArgs sa;
  sa.logits = logits;
  sa.ld = ld;
  sa.V = cf.vocab;
  sa.C = c->chunks;
  sa.stats = stats;
  sa.temp_used = temp_used;
  sa.uniforms = uniforms;
  sa.tokens = tokens;
  sa.t_cal = cf.t_cal;
  const Control ct = make_control(cf);
  const Budget bu = make_budget(cf, st.kappa);
  const bool vec = row_vec_ok(logits, ld);
  const int form = select_one_launch(cf.max_blocks_per_seq, cf.num_q_heads);
  if (form) {
    const size_t lds =
        static_cast<size_t>(est_lds_offset(2 * cf.max_blocks_per_seq)) * sizeof(unsigned) + est_lds;
#define ENT_STEPB_CASE(FF, VV)                                                                   \
  hipLaunchKernelGGL((step_b_kernel<FF, VV>), dim3(2 * B), dim3(kSelThreads), lds, s, B,        \
                     c->ent_part, c->chunks, st.temp, st.h_prev, st.tau, h_out, ct, c->zbuf,     \
                     c->lse_part, ctx_lens, tables, scores, theta, kept, c->kept_phys, n_kept,   \
                     cf.max_blocks_per_seq, cf.num_pool_blocks, c->lse_chunks, cf.num_q_heads,  \
                     bu, c->dev_flags, sa, est_mode, cf.est_k, c->tmax)
#define ENT_STEPB_F4(FF)                               \
  case FF:                                             \
    if (vec) ENT_STEPB_CASE(FF, true);                 \
    else ENT_STEPB_CASE(FF, false);                    \
    break;
    switch (form) {
      ENT_STEPB_F4(1)
      ENT_STEPB_F4(2)
      ENT_STEPB_F4(4)
      ENT_STEPB_F4(8)
      default:
        return hipErrorInvalidValue;
    }
#undef ENT_STEPB_F4
#undef ENT_STEPB_CASE
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else {
    float* sc = scores ? scores : c->iscores;
    const int ntile = (cf.max_blocks_per_seq + kStepTileBlocks - 1) / kStepTileBlocks;
    const int grid = B + B * ntile;
    // The selection inside the tile launch pays when its keys leave the
    // launch's residency as it is and the grid takes at most two rounds of
    // it (else the selecting workgroups hold slots that tiles wait for): on
    // the 70B-shaped loop 2 us faster, at 8192-block tables (one workgroup
    // per CU less) and a 2304-workgroup grid 18 and 10 us slower.
    const bool tick = c->b1_occ_ticket >= c->b1_occ_plain &&
                      grid <= 2 * c->num_cu * c->b1_occ_plain;
    const size_t lds = tick ? step_b1_lds(c, true) : step_b1_lds(c, false);
    auto k1 = tick ? (vec ? step_b1_kernel<true, true> : step_b1_kernel<false, true>)
                   : (vec ? step_b1_kernel<true, false> : step_b1_kernel<false, false>);
    hipLaunchKernelGGL(k1, dim3(grid), dim3(kFoldThreads), lds, s, B, c->ent_part,
                       c->chunks, st.temp, st.h_prev, st.tau, h_out, ct, c->zbuf, c->lse_part,
                       ctx_lens, sc, cf.num_q_heads, cf.max_blocks_per_seq, c->lse_chunks, ntile, sa,
                       est_mode, cf.est_k, c->tmax, tables, theta, kept, c->kept_phys, n_kept,
                       cf.num_pool_blocks, bu, c->dev_flags, tick ? c->tickets : nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (!tick) {
      e = launch_select_rows(c, B, tables, ctx_lens, h_out, sc, theta, kept, n_kept, st.kappa, s);
      if (e != hipSuccess) return e;
    }
    return launch_decode(c, B, q, k_cache, v_cache, tables, ctx_lens, kept, n_kept, out, lse, s,
                         c->kept_phys, ap, &sa);
  }
  return launch_decode(c, B, q, k_cache, v_cache, tables, ctx_lens, kept, n_kept, out, lse, s,
                       c->kept_phys, ap);
}

}  // namespace ent
