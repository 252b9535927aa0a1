// Entropy-aware scheduling (Section 3.1 of the paper: the priority
// pi(s) = E[Delta H_s] / (alpha C_s + beta M_s + gamma L_s); Section 7: bounded
// priorities, no starvation).  One workgroup over the whole pool of active
// sequences, before the decode step:
//   * a sequence that ran since the last call (age 0) folds its entropy drop
//     since then, d = tau - tau_last, into its mean: g = (1 - lam) g + lam d;
//   * pi = max(g, gain_floor) / (alpha kept + beta held + gamma slack), with
//     kept = blocks it kept at its last step, held = ceil(N / 16) and
//     slack = max(slo - age, slack_floor), in float32 in this order with no
//     fused multiply-add (the selection is an integer decided by floats);
//   * the B_sel largest priorities are selected, equal priorities to the
//     lower index: the B_sel-th largest key by an exact radix select, then
//     the selected indices in ascending order by wave ballots (all keys above
//     it, and the first ties up to the quota);
//   * selected sequences get age 0, the others age + 1.

#include "estimate_dev.h"

namespace ent {
namespace {

constexpr int kSchedThreads = 1024;
constexpr int kSchedWaves = kSchedThreads / 64;

struct SchedArgs {
  int N, b_sel;
  float alpha, beta, gamma, slo, slack_floor, gain_floor, lam;
  const float* tau;
  const int* n_kept;
  const int* ctx_lens;
  float* tau_last;
  float* gain;
  int* age;
  int* selected;
  int* n_selected;
  float* priority;
};

// Pool entries per thread: sequence s = t + kSchedThreads i is thread t's
// entry i in every phase, so its state stays in registers.
constexpr int kSchedPer = ENT_SCHED_MAX_POOL / kSchedThreads;
static_assert(ENT_SCHED_MAX_POOL % kSchedThreads == 0, "whole entries per thread");
static_assert(ENT_SCHED_MAX_POOL / 64 <= kEstBins / 2, "run counts fit half the histogram");

__device__ __forceinline__ float sched_priority(const SchedArgs& a, bool ran, float tau, int kept,
                                                int len, int age, float& g, float& tl) {
#pragma clang fp contract(off)
  if (ran) {
    const float d = tau - tl;
    const float keep = (1.f - a.lam) * g;
    const float add = a.lam * d;
    g = keep + add;
    tl = tau;
  }
  const float num = fmaxf(g, a.gain_floor);
  const float held = static_cast<float>((max(len, 0) + 15) / 16);
  const float slack = fmaxf(a.slo - static_cast<float>(age), a.slack_floor);
  float den = a.alpha * static_cast<float>(max(kept, 0));
  den = den + a.beta * held;
  den = den + a.gamma * slack;
  return __fdiv_rn(num, den);
}

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(SchedArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned keys[];   // [N rounded up to 4]
  __shared__ EstShared esh;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int N = a.N;
  const int N4 = (N + 3) & ~3;
  // Every load of the thread's entries is issued before any is used (the
  // state arrays are updated in place): indices past the pool are clamped to
  // its last entry (N >= 1) so the loads need no branch.
  float tau[kSchedPer], g[kSchedPer], tl[kSchedPer];
  int kept[kSchedPer], len[kSchedPer], age[kSchedPer];
#pragma unroll
  for (int i = 0; i < kSchedPer; ++i) {
    const int s = min(t + kSchedThreads * i, N - 1);
    tau[i] = a.tau[s];
    g[i] = a.gain[s];
    tl[i] = a.tau_last[s];
    kept[i] = a.n_kept[s];
    len[i] = a.ctx_lens[s];
    age[i] = a.age[s];
  }
  // Priorities (and the running means of the sequences that ran); keys in
  // LDS, padding below every priority.
#pragma unroll
  for (int i = 0; i < kSchedPer; ++i) {
    const int s = t + kSchedThreads * i;
    if (s < N) {
      const bool ran = age[i] == 0;
      const float pri = sched_priority(a, ran, tau[i], kept[i], len[i], age[i], g[i], tl[i]);
      if (ran) {
        a.gain[s] = g[i];
        a.tau_last[s] = tl[i];
      }
      if (a.priority) a.priority[s] = pri;
      keys[s] = est_key(pri);
    } else if (s < N4) {
      keys[s] = 0u;
    }
  }
  __syncthreads();
  const int take = min(max(a.b_sel, 0), N);
  unsigned theta = 0u;
  int n_gt = 0;
  if (take > 0 && take < N)
    theta = est_kth_largest<EstLdsKeys, true>(EstLdsKeys{keys}, N4 / 4, 1u, take, esh, n_gt);
  const int quota = take - n_gt;    // ties at theta to take, in index order
  const bool all = take == N;
  // Selected: key > theta, or key == theta among the first `quota` ties.
  // Run counts of both kinds (run r = indices 64 r .. 64 r + 63, i.e. wave
  // w's entry i is run w + 16 i), one wave's scan, then every selected index
  // at its place.
  unsigned* cgt = esh.hist;
  unsigned* ceq = esh.hist + kEstBins / 2;
  const int nrun = (N + 63) / 64;
  bool gt[kSchedPer], eq[kSchedPer];
#pragma unroll
  for (int i = 0; i < kSchedPer; ++i) {
    const int s = t + kSchedThreads * i;
    const unsigned k = s < N ? keys[s] : 0u;
    gt[i] = s < N && (all || (take > 0 && k > theta));
    eq[i] = s < N && !all && take > 0 && k == theta;
    const int r = wave + kSchedWaves * i;
    if (r < nrun) {
      const unsigned long long bg = __ballot(gt[i]), be = __ballot(eq[i]);
      if (lane == 0) {
        cgt[r] = static_cast<unsigned>(__popcll(bg));
        ceq[r] = static_cast<unsigned>(__popcll(be));
      }
    }
  }
  __syncthreads();
  if (wave == 0) {
    const int per = (nrun + 63) / 64;
    unsigned lg = 0, le = 0;
    for (int j = 0; j < per; ++j) {
      const int r = lane * per + j;
      if (r < nrun) {
        lg += cgt[r];
        le += ceq[r];
      }
    }
    unsigned ig = lg, ie = le;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned ng = __shfl_up(ig, o), ne = __shfl_up(ie, o);
      if (lane >= o) {
        ig += ng;
        ie += ne;
      }
    }
    unsigned rg = ig - lg, re = ie - le;
    for (int j = 0; j < per; ++j) {
      const int r = lane * per + j;
      if (r < nrun) {
        const unsigned cg = cgt[r], ce = ceq[r];
        cgt[r] = rg;
        ceq[r] = re;
        rg += cg;
        re += ce;
      }
    }
  }
  __syncthreads();
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int i = 0; i < kSchedPer; ++i) {
    const int s = t + kSchedThreads * i;
    const int r = wave + kSchedWaves * i;
    if (r < nrun) {
      const unsigned long long bg = __ballot(gt[i]), be = __ballot(eq[i]);
      const int gt_before = static_cast<int>(cgt[r]) + __popcll(bg & below);
      const int eq_before = static_cast<int>(ceq[r]) + __popcll(be & below);
      const bool sel = gt[i] || (eq[i] && eq_before < quota);
      if (sel) a.selected[gt_before + min(eq_before, quota)] = s;
      if (s < N) a.age[s] = sel ? 0 : age[i] + 1;
    }
  }
  if (t == 0) *a.n_selected = take;
}

}  // namespace

hipError_t launch_schedule(int N, const ent_sched_params& p, const float* tau, const int* n_kept,
                           const int* ctx_lens, float* tau_last, float* gain, int* age, int b_sel,
                           int* selected, int* n_selected, float* priority, hipStream_t s) {
  SchedArgs a;
  a.N = N;
  a.b_sel = b_sel;
  a.alpha = p.alpha;
  a.beta = p.beta;
  a.gamma = p.gamma;
  a.slo = p.slo;
  a.slack_floor = p.slack_floor;
  a.gain_floor = p.gain_floor;
  a.lam = p.ewma_rate;
  a.tau = tau;
  a.n_kept = n_kept;
  a.ctx_lens = ctx_lens;
  a.tau_last = tau_last;
  a.gain = gain;
  a.age = age;
  a.selected = selected;
  a.n_selected = n_selected;
  a.priority = priority;
  const size_t lds = static_cast<size_t>((N + 3) & ~3) * sizeof(unsigned);
  hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(kSchedThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace ent
