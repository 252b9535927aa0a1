// Per-stage kernels of the entropy / controller and sampling entry points
// (device bodies and their description in entropy_dev.h; the chunk passes run
// in the persistent kernel of prologue.hip).

#include "estimate_dev.h"

namespace ent {
namespace {

// One workgroup per row: the top-k or tail-corrected estimate from the chunk
// triples, the thread maxima and the re-read logits, then the controller.
constexpr int kEstFinalizeThreads = 512;

__global__ __launch_bounds__(kEstFinalizeThreads) void estimate_finalize_kernel(
    int est, int k, int V, int C, const float* __restrict__ part, const float* __restrict__ tmax,
    const float* __restrict__ logits, long long ld, float* __restrict__ temp,
    float* __restrict__ h_prev, float* __restrict__ tau, float* __restrict__ h_out,
    float* __restrict__ temp_used, Control ct, float t_cal) {
  extern __shared__ __attribute__((aligned(16))) unsigned est_lds[];
  __shared__ EstShared esh;
  const int b = blockIdx.x;
  const float T = temp[b];
  const float H = row_estimate(est, k, part, tmax, logits, ld, V, C, T * t_cal, b, est_lds, esh);
  if (threadIdx.x == 0) controller_update(b, H, T, h_prev, tau, temp, h_out, temp_used, ct);
}

// One wave per row: merge of the row's chunk triples, then the controller.
__global__ __launch_bounds__(256) void entropy_finalize_kernel(
    int B, int C, const float* __restrict__ part, float* __restrict__ temp,
    float* __restrict__ h_prev, float* __restrict__ tau, float* __restrict__ h_out,
    float* __restrict__ temp_used, Control ct) {
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const float H = row_entropy(part, C, b);
  if ((threadIdx.x & 63) == 0) controller_update(b, H, temp[b], h_prev, tau, temp, h_out, temp_used, ct);
}

template <bool VEC>
__global__ __launch_bounds__(kSampleThreads) void sample_kernel(
    const float* __restrict__ logits, long long ld, int V, int C,
    const float* __restrict__ row_stats, const float* __restrict__ temp_used,
    const float* __restrict__ uniforms, int* __restrict__ tokens, float t_cal) {
  __shared__ SampleShared sh;
  const int b = blockIdx.x;
  const int tok = sample_body<VEC>(logits, ld, V, C, row_stats, temp_used[b] * t_cal, uniforms[b], b,
                                   sh);
  if (threadIdx.x == 0) tokens[b] = tok;
}

}  // namespace

Control make_control(const ent_config& cf) {
  Control ct;
  ct.eta = cf.eta;
  ct.h_target = cf.h_target;
  ct.t_min = cf.t_min;
  ct.t_max = cf.t_max;
  ct.rho_t = cf.rho_t;
  ct.h_bias = cf.h_bias;
  return ct;
}

hipError_t launch_entropy(const ent_ctx* c, int B, const float* logits, long long ld,
                          ent_state st, float* h_out, float* temp_used, float* row_stats,
                          bool controller, hipStream_t s) {
  const ent_config& cf = c->cfg;
  // Without the controller (statistics for the sampler) the temperatures are
  // the ones passed in temp_used.
  PrologueArgs a{};
  a.B = B;
  a.do_entropy = 1;
  a.logits = logits;
  a.ld = ld;
  a.V = cf.vocab;
  a.C = c->chunks;
  a.temp = controller ? st.temp : temp_used;
  a.t_cal = cf.t_cal;
  a.part = controller ? c->ent_part : nullptr;
  a.row_stats = row_stats;
  const bool est = controller && uses_estimate(cf);
  a.tmax = est ? c->tmax : nullptr;
  a.Hkv = cf.num_kv_heads;
  a.G = c->group;
  a.MAXB = cf.max_blocks_per_seq;
  a.flags = c->dev_flags;
  hipError_t e = launch_prologue(c, a, s);
  if (e != hipSuccess || !controller) return e;
  if (est) {
    hipLaunchKernelGGL(estimate_finalize_kernel, dim3(B), dim3(kEstFinalizeThreads),
                       est_lds_bytes(c->chunks, cf.est_k), s, cf.estimator, cf.est_k, cf.vocab,
                       c->chunks, c->ent_part, c->tmax, logits, ld, st.temp, st.h_prev, st.tau,
                       h_out, temp_used, make_control(cf), cf.t_cal);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(entropy_finalize_kernel, dim3((B + 3) / 4), dim3(256), 0, s, B, c->chunks,
                     c->ent_part, st.temp, st.h_prev, st.tau, h_out, temp_used, make_control(cf));
  return hipGetLastError();
}

hipError_t launch_sample(const ent_ctx* c, int B, const float* logits, long long ld,
                         const float* row_stats, const float* temp_used, const float* uniforms,
                         int* tokens, hipStream_t s) {
  const bool vec = row_vec_ok(logits, ld);
  auto k = vec ? sample_kernel<true> : sample_kernel<false>;
  hipLaunchKernelGGL(k, dim3(B), dim3(kSampleThreads), 0, s, logits, ld, c->cfg.vocab, c->chunks,
                     row_stats, temp_used, uniforms, tokens, c->cfg.t_cal);
  return hipGetLastError();
}

}  // namespace ent
