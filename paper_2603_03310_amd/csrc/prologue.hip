// The two streaming passes that open a decode step, as one grid of 256-thread
// workgroups that walk a compact list of jobs of two kinds:
//
//   * block scoring (bf16 queries): job (sequence b, tile of 16 blocks,
//     group of four KV heads); wave w takes KV head 4 hg + w
//     (score_job / score_head_compute, Section 3.2);
//   * entropy chunk passes: job (row b, chunk c) of 4096 logits
//     (entropy_chunk_body, Section 2.1); chunk 0's job also records the
//     row's temperature T_t in temp_used when asked (the fused step's
//     sampler reads it in the next launch, while the controller replaces
//     temp with T_{t+1}).
//
// Both read HBM once (block summaries, logits) at a few flops per byte and
// do not depend on each other; scoring jobs come first.  Every workgroup
// keeps at most 128 registers a lane and 33.8 KB of LDS (the scoring waves'
// staging rows, at d = 128), so four workgroups per CU have their loads in
// flight at once.  Two grid forms: dense (one workgroup per job slot; slots
// for tiles past a sequence's end exit at once) and, when the block tables
// are much wider than the sequences, compact (the grid is sized to the
// chip's resident capacity and walks the list of tiles that exist, a prefix
// over the sequences' tile counts built in LDS by every workgroup).  In the
// compact form a workgroup's first kHeldJobs scoring jobs keep their block
// logits in registers and write them after its last job: on the 70B-shaped
// loop the prologue took 86.9 us against 90.2 us with every job's logits
// written as it ends (the stores then leave in the middle of the reads).
// The per-stage entry points run the same kernel with one kind of job only,
// which keeps their results bit-identical to the fused step's.

#include "blocks_dev.h"
#include "entropy_dev.h"

#include <algorithm>

namespace ent {
namespace {

constexpr int kProThreads = 256;
typedef float nt_f32x4_t __attribute__((ext_vector_type(4)));
constexpr int kProWaves = kProThreads / 64;

__host__ __device__ inline int head_groups(int Hkv) { return (Hkv + kProWaves - 1) / kProWaves; }

// s_pref[b] = first scoring tile of sequence b (s_pref[B] = all tiles);
// s_N[b] = its context length (-1 when invalid: no tiles, flagged later).
__device__ void tile_plan(const int* __restrict__ ctx_lens, int B, int MAXB, int* s_pref, int* s_N,
                          int* s_red) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = (B + kProThreads - 1) / kProThreads;
  int loc = 0;
  for (int i = 0; i < per; ++i) {
    const int b = t * per + i;
    if (b < B) {
      const int N = ctx_lens[b];
      const bool ok = N >= 0 && N <= MAXB * kBlock;
      s_N[b] = ok ? N : -1;
      loc += ok ? (N + kBlock * kMfmaChunk - 1) / (kBlock * kMfmaChunk) : 0;
    }
  }
  int incl = loc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(incl, o);
    if (lane >= o) incl += n;
  }
  if (lane == 63) s_red[wave] = incl;
  __syncthreads();
  int run = incl - loc;
  for (int w = 0; w < wave; ++w) run += s_red[w];
  for (int i = 0; i < per; ++i) {
    const int b = t * per + i;
    if (b < B) {
      s_pref[b] = run;
      const int N = s_N[b];
      run += N >= 0 ? (N + kBlock * kMfmaChunk - 1) / (kBlock * kMfmaChunk) : 0;
    }
  }
  if (t == kProThreads - 1) s_pref[B] = run;
  __syncthreads();
}

// One scoring job: tile ch of sequence b (context length N), KV heads of
// group hg (wave w takes head 4 hg + w); entry: the lane's table entry
// (score_tile_entry).  The wave's 16 summaries (512 B each at d = 128) are
// read with every load instruction covering whole summaries (lanes
// l*LPB .. l*LPB + LPB - 1 read one block's d floats), staged in the wave's
// LDS rows and read back in the MFMA layout: against loads straight into the
// MFMA layout (64 B of each of 16 blocks per instruction) the scoring pass
// got 4.7 us faster on the 8B shape and 7.6 us on the 70B-shaped loop.  The
// summaries are read once per step: non-temporal loads (the nt bit), 2 us
// faster on the 70B-shaped loop's prologue and 1 us on the 8B shape's.
template <int D>
__device__ __forceinline__ sf32x2_t score_job(const PrologueArgs& a, int b, int ch, int hg, int N,
                                              int entry, float* s_stage, bool store) {
  const int w = threadIdx.x >> 6;
  const int g = hg * kProWaves + w;
  if (g >= a.Hkv) return sf32x2_t{0.f, 0.f};
  const int nb = (N + kBlock - 1) / kBlock;
  const int p = score_tile_check(entry, ch, nb, a.P, a.flags);   // block r16's, lane r16
  const int lane = threadIdx.x & 63;
  constexpr int LPB = D / 4;              // lanes per summary (one float4 each)
  constexpr int BPI = 64 / LPB;           // summaries per load instruction
  constexpr int NI = kMfmaChunk / BPI;    // load instructions
  constexpr int RS = D + 4;               // LDS row stride (floats), padded
  float4 buf[kScoreSlots];
#pragma unroll
  for (int k = 0; k < NI; ++k) {
    const int blk = k * BPI + lane / LPB;
    const int pb = __shfl(p, blk);
    const nt_f32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const nt_f32x4_t*>(
        a.ksum + (static_cast<long long>(pb) * a.Hkv + g) * D + (lane % LPB) * 4));
    buf[k] = make_float4(x.x, x.y, x.z, x.w);
  }
  uint2 qv[D / 16];
  score_q_load<D>(a.q, b, g, a.Hkv, a.G, qv);
  // Every load above is issued before any arithmetic: one memory round trip.
  __builtin_amdgcn_sched_barrier(0);
  float* st = s_stage + w * kMfmaChunk * RS;
#pragma unroll
  for (int k = 0; k < NI; ++k) {
    const int blk = k * BPI + lane / LPB;
    *reinterpret_cast<float4*>(st + blk * RS + (lane % LPB) * 4) = buf[k];
  }
  // The rows are the wave's own: a wave-level barrier orders the exchange.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int r16 = lane & 15, gq = lane >> 4;
#pragma unroll
  for (int j = 0; j < D / 16; ++j) buf[j] = *reinterpret_cast<const float4*>(st + r16 * RS + 16 * j + 4 * gq);
  return score_head_compute<D>(qv, buf, a.zbuf, a.lse_part, b, ch, g, N, nb, a.Hkv, a.G, a.MAXB,
                               a.nch_max, a.scale, store);
}

// Sequence of scoring tile `tile` in the compact job list: the largest b
// with s_pref[b] <= tile.
__device__ __forceinline__ int tile_seq(const int* s_pref, int B, int tile) {
  int lo = 0, hi = B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_pref[mid] <= tile) lo = mid; else hi = mid;
  }
  return lo;
}

// Scoring jobs of a compact-form workgroup whose block logits wait in
// registers (two per lane each, G <= 8) until its job loop ends, so that
// those stores leave after the workgroup's reads instead of between them.
constexpr int kHeldJobs = 10;

// Dense form: one workgroup per job slot, scoring slots (b, ch, hg) for every
// tile a sequence could have (slots past its end exit at once), then one per
// entropy chunk.  Compact form (COMPACT): the grid walks the list of jobs
// that exist.
template <bool VEC, int D, bool COMPACT>
__global__ __launch_bounds__(kProThreads) void prologue_kernel(PrologueArgs a) {
  extern __shared__ int s_mem[];           // compact: s_pref [B + 1], s_N [B]
  __shared__ int s_red[kProWaves];
  __shared__ float red[16];
  __shared__ __attribute__((aligned(16))) float s_stage[kProWaves * kMfmaChunk * (D + 4)];
  const int nhg = head_groups(a.Hkv);
  if (!COMPACT) {
    const int tiles = (a.MAXB + kMfmaChunk - 1) / kMfmaChunk;
    const int nsc = a.do_score ? a.B * tiles * nhg : 0;
    const int id = blockIdx.x;
    if (id < nsc) {
      const int b = id / (tiles * nhg);
      const int r = id - b * tiles * nhg;
      const int ch = r / nhg;
      // The context length and the tile's table entries load together.
      const int entry = score_tile_entry(a.tables, b, ch, a.MAXB);
      const int N = a.ctx_lens[b];
      if (N < 0 || N > a.MAXB * kBlock) return;    // flagged by the selection stage
      if (ch * kMfmaChunk * kBlock >= N) return;
      score_job<D>(a, b, ch, r - ch * nhg, N, entry, s_stage, true);
      return;
    }
    const int e = id - nsc;
    const int b = e / a.C;
    entropy_chunk_body<VEC>(a.logits, a.ld, a.V, a.C, a.temp, a.t_cal, a.part, a.row_stats,
                            a.tmax, e - b * a.C, b, red);
    if (e == b * a.C && threadIdx.x == 0 && a.temp_used) a.temp_used[b] = a.temp[b];
    return;
  }
  int* s_pref = s_mem;
  int* s_N = s_mem + a.B + 1;
  int n_score = 0;
  if (a.do_score) {
    tile_plan(a.ctx_lens, a.B, a.MAXB, s_pref, s_N, s_red);
    n_score = s_pref[a.B] * nhg;
  }
  const int n_jobs = n_score + (a.do_entropy ? a.B * a.C : 0);
  const bool hold = a.G <= 8;
  sf32x2_t held[kHeldJobs];
  int it = 0;
  for (int job = blockIdx.x; job < n_jobs; job += gridDim.x, ++it) {
    if (job < n_score) {
      const int tile = job / nhg;
      const int lo = tile_seq(s_pref, a.B, tile);
      const int ch = tile - s_pref[lo];
      const bool keep = hold && it < kHeldJobs;
      const sf32x2_t z = score_job<D>(a, lo, ch, job - tile * nhg, s_N[lo],
                                      score_tile_entry(a.tables, lo, ch, a.MAXB), s_stage, !keep);
      if (keep) {
#pragma unroll
        for (int k = 0; k < kHeldJobs; ++k)
          if (k == it) held[k] = z;
      }
    } else {
      const int e = job - n_score;
      const int b = e / a.C;
      entropy_chunk_body<VEC>(a.logits, a.ld, a.V, a.C, a.temp, a.t_cal, a.part, a.row_stats,
                              a.tmax, e - b * a.C, b, red);
      if (e == b * a.C && threadIdx.x == 0 && a.temp_used) a.temp_used[b] = a.temp[b];
    }
  }
  if (!hold) return;
  const int w = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < kHeldJobs; ++k) {
    const int job = blockIdx.x + k * gridDim.x;
    if (job >= n_score) break;
    const int tile = job / nhg;
    const int lo = tile_seq(s_pref, a.B, tile);
    const int g = (job - tile * nhg) * kProWaves + w;
    if (g < a.Hkv)
      store_held_z(held[k], a.zbuf, lo, tile - s_pref[lo], g, (s_N[lo] + kBlock - 1) / kBlock,
                   a.Hkv, a.G, a.MAXB);
  }
}

template <bool VEC, int D>
int prologue_per_cu() {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, prologue_kernel<VEC, D, true>, kProThreads, 0) !=
          hipSuccess || n < 1)
    n = 1;
  return n;
}

}  // namespace

int prologue_grid_size(const ent_ctx* c) {
  const int n = c->cfg.head_dim == 128
                    ? std::min(prologue_per_cu<true, 128>(), prologue_per_cu<false, 128>())
                    : std::min(prologue_per_cu<true, 64>(), prologue_per_cu<false, 64>());
  return c->num_cu * n;
}

hipError_t launch_prologue(const ent_ctx* c, const PrologueArgs& a, hipStream_t s) {
  const ent_config& cf = c->cfg;
  // Dense job slots (every sequence at its largest length).
  long long slots = 0;
  if (a.do_score)
    slots += static_cast<long long>(a.B) * ((cf.max_blocks_per_seq + kMfmaChunk - 1) / kMfmaChunk) *
             head_groups(a.Hkv);
  if (a.do_entropy) slots += static_cast<long long>(a.B) * a.C;
  if (slots == 0) return hipSuccess;
  // Dispatching a workgroup costs time even when it exits at once: when the
  // dense slots outnumber what the chip holds many times over (short
  // sequences under a large block-table width), walk the compact job list.
  const bool compact = slots > 16ll * c->prologue_grid;
  const unsigned grid = static_cast<unsigned>(compact ? c->prologue_grid : slots);
  const size_t lds = compact ? static_cast<size_t>(2 * a.B + 1) * sizeof(int) : 0;
  const bool vec = !a.do_entropy || row_vec_ok(a.logits, a.ld);
#define ENT_PRO_LAUNCH(V, DD)                                                                  \
  do {                                                                                         \
    if (compact)                                                                               \
      hipLaunchKernelGGL((prologue_kernel<V, DD, true>), dim3(grid), dim3(kProThreads), lds, s, a); \
    else                                                                                       \
      hipLaunchKernelGGL((prologue_kernel<V, DD, false>), dim3(grid), dim3(kProThreads), 0, s, a); \
  } while (0)
  if (cf.head_dim == 128) {
    if (vec) ENT_PRO_LAUNCH(true, 128); else ENT_PRO_LAUNCH(false, 128);
  } else {
    if (vec) ENT_PRO_LAUNCH(true, 64); else ENT_PRO_LAUNCH(false, 64);
  }
#undef ENT_PRO_LAUNCH
  return hipGetLastError();
}

}  // namespace ent
