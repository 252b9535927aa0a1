// Internal declarations shared by the HIP translation units of libent.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "ent.h"

namespace ent {

constexpr int kBlock = ENT_BLOCK_SIZE;      // tokens per KV block
constexpr int kRowChunk = ENT_ROW_CHUNK;    // logits per entropy chunk
constexpr int kMinScoreChunk = 16;          // smallest scoring chunk (blocks)
constexpr int kMaxGroup = 16;               // query heads per KV head
constexpr int kMaxBlocksPerSeq = 16384;     // selection keeps all scores in LDS
constexpr int kEstChunkThreads = 256;       // threads of an entropy chunk job (maxima per chunk)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Parameters of the controller (Section 3.3 and Section 5): the signed gain,
// the target entropy, the temperature bounds, the bound on the temperature's
// log step per update, and the entropy offset of the stress tests.
struct Control {
  float eta, h_target, t_min, t_max, rho_t, h_bias;
};
Control make_control(const ent_config& cf);

// Parameters of the block budget and the kept-fraction state (Sections
// 3.2, 3.3, 5): the guarded entropy, the floor, the smallest fraction and
// count, and the bound on how fast the kept fraction may fall.
struct Budget {
  float eps_h, h_min, log_v, kappa_min, dkappa;
  int b_min;
  int keep_first, keep_last;   // blocks always kept at each end of a sequence
  float* kappa;   // nullable [B]: previous kept fraction (NaN = none), updated in place
};

// Arguments of the append body (ent_kv_append), which also runs inside the
// last launch of ent_decode_step_append.
struct AppendArgs {
  const void* k_new;
  const void* v_new;
  const int* tables;
  int* ctx_lens;
  void* kc;
  void* vc;
  float* ksum;
  int Hkv, D, MAXB, P;
  unsigned* flags;
  bool bf16;
};

}  // namespace ent

struct ent_ctx {
  ent_config cfg;
  int device = 0;
  int num_cu = 0;
  int group = 1;            // G = H_q / H_kv
  int chunks = 0;           // entropy chunks per logit row
  int lse_chunks = 0;       // log-sum-exp partials per sequence (finest chunking)
  int decode_grid = 0;      // persistent decode workgroups
  int prologue_grid = 0;    // resident entropy / scoring workgroups
  int b1_occ_plain = 0;     // resident tile-launch workgroups per CU, without the selection inside
  int b1_occ_ticket = 0;    // ... and with it

  void* ws = nullptr;       // one workspace allocation
  size_t ws_bytes = 0;
  float* ent_part = nullptr;      // [max_batch, chunks, 3]  (max, sum, weighted sum)
  float* stats_tmp = nullptr;     // [max_batch, chunks, 2]  row statistics scratch
  float* zbuf = nullptr;          // [max_batch, MAXB, H_q]  block logits
  float* lse_part = nullptr;      // [max_batch, lse_chunks, H_q, 2]
  float* lrow = nullptr;          // [max_batch, H_q]  L_h per sequence
  float* iscores = nullptr;       // [max_batch, MAXB]  block scores when the caller keeps none
  int* kept_phys = nullptr;       // [max_batch, MAXB]  physical blocks of the kept lists
  float* dec_acc = nullptr;       // [decode partial slots, G, d]
  float* dec_ml = nullptr;        // [decode partial slots, G, 2]
  int4* dec_rec = nullptr;        // [decode waves]  cut-segment records of the decode ranges
  float* tmax = nullptr;          // [max_batch, chunks, 256]  per-thread logit maxima (estimators)
  float2* exbuf = nullptr;        // [max_batch, MAXB, H_q]  exact mode: (log mass, mean logit) per block
  unsigned* tickets = nullptr;    // [max_batch]  per-sequence counters of the fused step (zero between launches)
  unsigned* dev_flags = nullptr;  // [1]

  std::string err;
};

namespace ent {

// Whether the controller acts on an estimate (top-k or tail-corrected) of
// the entropy: with k >= |V| both estimates are the exact entropy.
inline bool uses_estimate(const ent_config& cf) {
  return cf.estimator != ENT_EST_EXACT && cf.est_k < cf.vocab;
}

// Launchers (one per kernel family); each returns the launch status.
hipError_t launch_entropy(const ent_ctx* c, int B, const float* logits, long long ld,
                          ent_state st, float* h_out, float* temp_used, float* row_stats,
                          bool controller, hipStream_t s);
hipError_t launch_sample(const ent_ctx* c, int B, const float* logits, long long ld,
                         const float* row_stats, const float* temp_used, const float* uniforms,
                         int* tokens, hipStream_t s);
hipError_t launch_block_summary(const ent_ctx* c, int B, const void* k_cache,
                                const int* tables, const int* ctx_lens, float* ksum,
                                hipStream_t s);
hipError_t launch_block_select(const ent_ctx* c, int B, const void* q, const float* ksum,
                               const void* k_cache, const int* tables, const int* ctx_lens,
                               const float* h, int* kept, int* n_kept, float* scores,
                               float* theta, float* kappa, hipStream_t s);
// Exact token-level scoring: per block and query head (log mass, mean logit)
// into c->exbuf and the per-tile log-sum-exp partials into c->lse_part.
hipError_t launch_exact_scores(const ent_ctx* c, int B, const void* q, const void* k_cache,
                               const int* tables, const int* ctx_lens, hipStream_t s);
// Block scores of the exact mode from c->exbuf and c->lrow.
hipError_t launch_exact_block_scores(const ent_ctx* c, int B, const int* ctx_lens, float* scores,
                                     hipStream_t s);
// Selection phase A: L_h of every sequence into c->lrow from c->lse_part.
hipError_t launch_lse_merge(const ent_ctx* c, int B, const int* ctx_lens, hipStream_t s);
Budget make_budget(const ent_config& cf, float* kappa);
// The pass over logits and block summaries that opens a step:
// entropy chunk triples / row statistics (do_entropy) and block scoring of
// bf16 queries (do_score), in one grid.
struct PrologueArgs {
  int B;
  int do_entropy;
  const float* logits;
  long long ld;
  int V, C;
  const float* temp;
  float* part;          // chunk triples (nullable)
  float* row_stats;     // chunk (max, sum) (nullable)
  float* temp_used;     // nullable: receives temp[b] (written by chunk 0's job)
  float* tmax;          // nullable: per-thread maxima of the chunk, [B, C, 256] (estimators)
  float t_cal;          // calibration temperature: the chunk pass uses temp[b] * t_cal
  int do_score;
  const uint16_t* q;
  const float* ksum;
  const int* tables;
  const int* ctx_lens;
  float* zbuf;
  float* lse_part;
  int Hkv, G, MAXB, P, nch_max;
  float scale;
  unsigned* flags;
};
hipError_t launch_prologue(const ent_ctx* c, const PrologueArgs& a, hipStream_t s);
int prologue_grid_size(const ent_ctx* c);
// Residency of the fused step's tile launch with and without the selection
// inside (ent_ctx::b1_occ_*).
void step_occupancy(ent_ctx* c);
// The kept-block selection after scoring (L merge, block scores, radix
// select), given each sequence's entropy h.
hipError_t launch_selection(const ent_ctx* c, int B, const int* tables, const int* ctx_lens,
                            const float* h, float* scores, float* theta, int* kept, int* n_kept,
                            float* kappa, hipStream_t s);
// Selection phases B (block scores from c->lrow) and C (radix select).
hipError_t launch_block_scores(const ent_ctx* c, int B, const int* ctx_lens, float* scores,
                               hipStream_t s);
hipError_t launch_select_rows(const ent_ctx* c, int B, const int* tables, const int* ctx_lens,
                              const float* h, const float* scores, float* theta, int* kept,
                              int* n_kept, float* kappa, hipStream_t s);
hipError_t launch_score_valu(const ent_ctx* c, int B, const void* q, const float* ksum,
                             const int* tables, const int* ctx_lens, hipStream_t s);

// Sampling issued in the launch that runs the kept-block selection (the
// fused step), on workgroups of its own; the arguments of ent_sample.
struct SampleArgs {
  const float* logits;
  long long ld;
  int V, C;
  const float* stats;
  const float* temp_used;
  const float* uniforms;
  int* tokens;
  float t_cal;          // calibration temperature: sampling at temp_used[b] * t_cal
};

// kept_phys (nullable): the selection's encoded physical blocks of the same
// kept lists, read instead of kept + tables.
// ap (nullable): an append of one token per sequence, and sp (nullable) the
// sampling of every row, that share the launch merging the split attention
// segments (none of the three reads what another writes).
hipError_t launch_decode(const ent_ctx* c, int B, const void* q, const void* k_cache,
                         const void* v_cache, const int* tables, const int* ctx_lens,
                         const int* kept, const int* n_kept, float* out, float* lse,
                         hipStream_t s, const int* kept_phys = nullptr,
                         const AppendArgs* ap = nullptr, const SampleArgs* sp = nullptr);
hipError_t launch_decode_step(const ent_ctx* c, int B, const float* logits, long long ld,
                              ent_state st, const void* q, const void* k_cache,
                              const void* v_cache, const float* ksum, const int* tables,
                              const int* ctx_lens, const float* uniforms, float* h_out,
                              float* temp_used, float* row_stats, int* kept, int* n_kept,
                              float* out, float* lse, int* tokens, float* scores, float* theta,
                              hipStream_t s, const AppendArgs* ap = nullptr);
AppendArgs make_append_args(const ent_ctx* c, const void* k_new, const void* v_new,
                            const int* tables, int* ctx_lens, void* k_cache, void* v_cache,
                            float* ksum);
hipError_t launch_kv_append(const ent_ctx* c, int B, const void* k_new, const void* v_new,
                            const int* tables, int* ctx_lens, void* k_cache, void* v_cache,
                            float* ksum, hipStream_t s);
hipError_t launch_schedule(int N, const ent_sched_params& p, const float* tau, const int* n_kept,
                           const int* ctx_lens, float* tau_last, float* gain, int* age, int b_sel,
                           int* selected, int* n_selected, float* priority, hipStream_t s);

// Configuration check of ent_init (message, ENT_OK / ENT_E_INVAL /
// ENT_E_UNSUPPORTED in *code), and the message ent_last_error(NULL) returns
// (calls without a context: ent_init, ent_entropy_temperature_noalloc).
std::string config_error(const ent_config* cfg, int* code);
void set_free_error(const std::string& msg);

// Occupancy-derived persistent grid of the decode kernel, and the number of
// partial slots its split segments may use (waves + segments).
int decode_grid_size(const ent_ctx* c);
long long decode_partial_slots(int decode_grid, int max_batch, int num_kv_heads);

}  // namespace ent

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
#if defined(__HIPCC__)
namespace ent {

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even float -> bf16 bits (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ unsigned wave_min_u(unsigned v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, static_cast<unsigned>(__shfl_xor(static_cast<int>(v), o)));
  return v;
}

__device__ __forceinline__ unsigned wave_max_u(unsigned v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, static_cast<unsigned>(__shfl_xor(static_cast<int>(v), o)));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ void raise_flag(unsigned* flags, unsigned f) {
  atomicOr(flags, f);
}

}  // namespace ent
#endif
