// One whole decode step in four launches (ent_decode_step).  Each launch runs
// the same device bodies as the per-stage entry points, so the results are
// bit-identical to calling ent_entropy_temperature, ent_block_select,
// ent_sparse_paged_decode and ent_sample in sequence:
//
//   A  block scoring and the entropy chunk passes in one persistent grid
//      (prologue.hip): both stream from HBM (block summaries, logits) and
//      do not depend on each other (fp32 queries: scoring is a second
//      launch, on the VALU);
//   B  one workgroup per sequence: the row's entropy from the chunk triples,
//      the controller update, and the kept-block selection under the
//      entropy-driven budget;
//   C  kept-block decode attention;
//   D  the merge of split decode segments and, in the same launch, sampling
//      at the temperature the step used (independent of the merge).

#include "blocks_dev.h"
#include "entropy_dev.h"

namespace ent {
namespace {

struct StepBArgs {
  const float* part;
  int C;
  float* temp;
  float* h_prev;
  float* tau;
  float* h_out;
  float* temp_used;
  float eta, h_target, t_min, t_max;
  const float* zbuf;
  const float* lse_part;
  const int* ctx_lens;
  float* scores;
  float* theta;
  int* kept;
  int* n_kept;
  int Hq, MAXB, chunk, nch_max;
  float eps_h, h_min, log_v, kappa_min;
  int b_min;
  unsigned* flags;
};

__global__ __launch_bounds__(kSelThreads) void step_b_kernel(StepBArgs a) {
  extern __shared__ unsigned keys[];        // [MAXB]
  __shared__ SelectShared ssh;
  __shared__ float s_H;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  if (t < 64) {
    const float H = row_entropy(a.part, a.C, b);
    if (t == 0) {
      s_H = H;
      controller_update(b, H, a.temp[b], a.h_prev, a.tau, a.temp, a.h_out, a.temp_used, a.eta,
                        a.h_target, a.t_min, a.t_max);
    }
  }
  __syncthreads();
  const float H = s_H;
  select_body(a.zbuf, a.lse_part, a.ctx_lens, H, a.scores, a.theta, a.kept, a.n_kept, a.Hq,
              a.MAXB, a.chunk, a.nch_max, a.eps_h, a.h_min, a.log_v, a.kappa_min, a.b_min,
              a.flags, b, keys, ssh);
}

}  // namespace

hipError_t launch_decode_step(const ent_ctx* c, int B, const float* logits, long long ld,
                              ent_state st, const void* q, const void* k_cache,
                              const void* v_cache, const float* ksum, const int* tables,
                              const int* ctx_lens, const float* uniforms, float* h_out,
                              float* temp_used, float* row_stats, int* kept, int* n_kept,
                              float* out, float* lse, int* tokens, float* scores, float* theta,
                              hipStream_t s) {
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
  pa.part = c->ent_part;
  pa.row_stats = stats;
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

  StepBArgs a;
  a.part = c->ent_part;
  a.C = c->chunks;
  a.temp = st.temp;
  a.h_prev = st.h_prev;
  a.tau = st.tau;
  a.h_out = h_out;
  a.temp_used = temp_used;
  a.eta = cf.eta;
  a.h_target = cf.h_target;
  a.t_min = cf.t_min;
  a.t_max = cf.t_max;
  a.zbuf = c->zbuf;
  a.lse_part = c->lse_part;
  a.ctx_lens = ctx_lens;
  a.scores = scores;
  a.theta = theta;
  a.kept = kept;
  a.n_kept = n_kept;
  a.Hq = cf.num_q_heads;
  a.MAXB = cf.max_blocks_per_seq;
  a.chunk = cf.kv_dtype == ENT_BF16 ? kMfmaChunk : kValuChunk;
  a.nch_max = c->lse_chunks;
  a.eps_h = cf.eps_h;
  a.h_min = cf.h_min;
  a.log_v = cf.log_v;
  a.kappa_min = cf.kappa_min;
  a.b_min = cf.b_min;
  a.flags = c->dev_flags;
  const size_t lds = static_cast<size_t>(cf.max_blocks_per_seq) * sizeof(unsigned);
  hipLaunchKernelGGL(step_b_kernel, dim3(B), dim3(kSelThreads), lds, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  SampleArgs sa;
  sa.logits = logits;
  sa.ld = ld;
  sa.V = cf.vocab;
  sa.C = c->chunks;
  sa.stats = stats;
  sa.temp_used = temp_used;
  sa.uniforms = uniforms;
  sa.tokens = tokens;
  return launch_decode(c, B, q, k_cache, v_cache, tables, ctx_lens, kept, n_kept, out, lse, s,
                       &sa);
}

}  // namespace ent
