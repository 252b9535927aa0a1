// Host side of the C ABI: configuration checks, the workspace, argument
// validation and launch sequencing.  No entry point allocates except
// ent_init; none synchronises except ent_init, ent_destroy and
// ent_device_status.

#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <string>

#include "ent_internal.h"

namespace {

thread_local std::string g_init_error;

constexpr int kMaxBatch = 4096;
constexpr int kMaxQHeads = 128;
constexpr int kMaxVocab = 256 * ENT_ROW_CHUNK;

bool is_pow2_group(int g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

std::string check_config(const ent_config* c, int* code) {
  *code = ENT_E_INVAL;
  if (!c) return "config is NULL";
  if (c->max_batch < 1 || c->max_batch > kMaxBatch) return "max_batch must be in [1, 4096]";
  if (c->num_kv_heads < 1 || c->num_q_heads < 1) return "head counts must be >= 1";
  if (c->num_q_heads % c->num_kv_heads != 0) return "num_q_heads must be a multiple of num_kv_heads";
  if (c->block_size != ENT_BLOCK_SIZE) return "block_size must be 16";
  if (c->max_blocks_per_seq < 1) return "max_blocks_per_seq must be >= 1";
  if (c->num_pool_blocks < 1) return "num_pool_blocks must be >= 1";
  if (c->vocab < 1) return "vocab must be >= 1";
  if (c->kv_dtype != ENT_F32 && c->kv_dtype != ENT_BF16) return "kv_dtype must be ENT_F32 or ENT_BF16";
  if (!isfinite(c->scale)) return "scale must be finite";
  if (!isfinite(c->eta) || !isfinite(c->h_target)) return "eta and h_target must be finite";
  if (!(c->t_min > 0.f) || !(c->t_max >= c->t_min) || !isfinite(c->t_max))
    return "need 0 < t_min <= t_max < inf";
  if (!(c->eps_h >= 0.f) || !isfinite(c->eps_h)) return "eps_h must be finite and >= 0";
  if (!isfinite(c->h_min) || !isfinite(c->log_v) || !(c->log_v > c->h_min))
    return "need finite h_min < log_v";
  if (!(c->kappa_min >= 0.f && c->kappa_min <= 1.f)) return "kappa_min must be in [0, 1]";
  if (c->b_min < 0) return "b_min must be >= 0";
  if (c->estimator != ENT_EST_EXACT && c->estimator != ENT_EST_TOPK && c->estimator != ENT_EST_TAIL)
    return "estimator must be ENT_EST_EXACT, ENT_EST_TOPK or ENT_EST_TAIL";
  if (c->estimator != ENT_EST_EXACT && (c->est_k < 1 || c->est_k > ENT_EST_MAX_K))
    return "est_k must be in [1, ENT_EST_MAX_K]";
  if (!(c->t_cal > 0.f) || !isfinite(c->t_cal)) return "t_cal must be finite and > 0";
  if (!(c->rho_t >= 0.f)) return "rho_t must be >= 0 (INFINITY: no bound)";
  if (!(c->dkappa >= 0.f && c->dkappa <= 1.f)) return "dkappa must be in [0, 1]";
  if (!isfinite(c->h_bias)) return "h_bias must be finite";
  if (c->scoring != ENT_SCORE_MEANKEY && c->scoring != ENT_SCORE_EXACT)
    return "scoring must be ENT_SCORE_MEANKEY or ENT_SCORE_EXACT";
  if (c->keep_first < 0 || c->keep_last < 0) return "keep_first and keep_last must be >= 0";
  *code = ENT_E_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
  if (!is_pow2_group(c->num_q_heads / c->num_kv_heads))
    return "num_q_heads / num_kv_heads must be 1, 2, 4, 8 or 16";
  if (c->num_q_heads > kMaxQHeads) return "num_q_heads must be <= 128";
  if (c->max_blocks_per_seq > ent::kMaxBlocksPerSeq) return "max_blocks_per_seq must be <= 16384";
  if (c->num_kv_heads * c->head_dim > 2048) return "num_kv_heads * head_dim must be <= 2048";
  if (c->vocab > kMaxVocab) return "vocab must be <= 1048576";
  if (c->num_pool_blocks >= (1 << 30)) return "num_pool_blocks must be < 2^30";
  if (static_cast<long long>(c->max_batch) * c->max_blocks_per_seq * c->num_kv_heads >= (1ll << 31))
    return "max_batch * max_blocks_per_seq * num_kv_heads must be < 2^31";
  *code = ENT_OK;
  return "";
}

int fail(ent_ctx* c, int code, const std::string& msg) {
  c->err = msg;
  return code;
}

int hip_fail(ent_ctx* c, hipError_t e, const char* what) {
  c->err = std::string(what) + ": " + hipGetErrorString(e);
  return ENT_E_HIP;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Kernels of a context run on the device that was current at ent_init.
int check_device(ent_ctx* c) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(c, e, "hipGetDevice");
  if (dev != c->device)
    return fail(c, ENT_E_INVAL, "the current HIP device is not the context's (the one current at ent_init)");
  return ENT_OK;
}

int check_batch(ent_ctx* c, int B) {
  if (int r = check_device(c)) return r;
  if (B < 0 || B > c->cfg.max_batch)
    return fail(c, ENT_E_INVAL, "B must be in [0, max_batch]");
  return ENT_OK;
}

size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

namespace ent {
std::string config_error(const ent_config* cfg, int* code) { return check_config(cfg, code); }
void set_free_error(const std::string& msg) { g_init_error = msg; }
}  // namespace ent

extern "C" {

void ent_default_config(ent_config* out) {
  if (!out) return;
  memset(out, 0, sizeof(*out));
  out->max_batch = 64;
  out->num_q_heads = 32;
  out->num_kv_heads = 8;
  out->head_dim = 128;
  out->block_size = ENT_BLOCK_SIZE;
  out->max_blocks_per_seq = 512;
  out->num_pool_blocks = 1;
  out->vocab = 128256;
  out->kv_dtype = ENT_BF16;
  out->scale = static_cast<float>(1.0 / sqrt(128.0));
  out->eta = -0.05f;
  out->h_target = 2.5f;
  out->t_min = 0.05f;
  out->t_max = 5.0f;
  out->eps_h = 0.0f;
  out->h_min = 2.5f;
  out->kappa_min = 0.05f;
  out->b_min = 4;
  out->log_v = static_cast<float>(log(128256.0));
  out->estimator = ENT_EST_EXACT;
  out->est_k = 256;
  out->t_cal = 1.0f;
  out->rho_t = INFINITY;
  out->dkappa = 1.0f;
  out->h_bias = 0.0f;
  out->scoring = ENT_SCORE_MEANKEY;
  out->keep_first = 0;
  out->keep_last = 0;
}

int ent_check_config(const ent_config* cfg, char* msg, int msg_len) {
  int code;
  const std::string m = check_config(cfg, &code);
  if (msg && msg_len > 0) snprintf(msg, static_cast<size_t>(msg_len), "%s", m.c_str());
  return code;
}

int ent_row_stats_chunks(int vocab) { return vocab <= 0 ? 0 : (vocab + ENT_ROW_CHUNK - 1) / ENT_ROW_CHUNK; }

int ent_init(const ent_config* cfg, ent_ctx** out) {
  if (!out) {
    g_init_error = "out is NULL";
    return ENT_E_INVAL;
  }
  *out = nullptr;
  int code;
  const std::string m = check_config(cfg, &code);
  if (code != ENT_OK) {
    g_init_error = m;
    return code;
  }
  ent_ctx* c = new (std::nothrow) ent_ctx();
  if (!c) {
    g_init_error = "host allocation failed";
    return ENT_E_NOMEM;
  }
  c->cfg = *cfg;
  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&c->num_cu, hipDeviceAttributeMultiprocessorCount, c->device);
  if (e != hipSuccess) {
    g_init_error = std::string("no usable HIP device: ") + hipGetErrorString(e);
    delete c;
    return ENT_E_HIP;
  }
  const ent_config& f = c->cfg;
  c->group = f.num_q_heads / f.num_kv_heads;
  c->chunks = ent_row_stats_chunks(f.vocab);
  c->lse_chunks = (f.max_blocks_per_seq + ent::kMinScoreChunk - 1) / ent::kMinScoreChunk;
  c->decode_grid = ent::decode_grid_size(c);
  c->prologue_grid = ent::prologue_grid_size(c);
  ent::step_occupancy(c);

  const size_t Bm = static_cast<size_t>(f.max_batch);
  const size_t sz_ent_part = align_up(Bm * c->chunks * 3 * sizeof(float));
  const size_t sz_stats = align_up(Bm * c->chunks * 2 * sizeof(float));
  const size_t sz_z = align_up(Bm * f.max_blocks_per_seq * f.num_q_heads * sizeof(float));
  const size_t sz_lse = align_up(Bm * c->lse_chunks * f.num_q_heads * 2 * sizeof(float));
  const size_t sz_lrow = align_up(Bm * f.num_q_heads * sizeof(float));
  const size_t sz_isc = align_up(Bm * f.max_blocks_per_seq * sizeof(float));
  const size_t sz_kphys = align_up(Bm * f.max_blocks_per_seq * sizeof(int));
  const size_t nslots = static_cast<size_t>(
      ent::decode_partial_slots(c->decode_grid, f.max_batch, f.num_kv_heads));
  const size_t sz_acc = align_up(nslots * c->group * f.head_dim * sizeof(float));
  const size_t sz_ml = align_up(nslots * c->group * 2 * sizeof(float));
  const size_t sz_rec = align_up(static_cast<size_t>(c->decode_grid) * 4 * sizeof(int4));
  const size_t sz_tmax = f.estimator == ENT_EST_EXACT
                             ? 0
                             : align_up(Bm * c->chunks * ent::kEstChunkThreads * sizeof(float));
  const size_t sz_ex = f.scoring == ENT_SCORE_EXACT
                           ? align_up(Bm * f.max_blocks_per_seq * f.num_q_heads * 2 * sizeof(float))
                           : 0;
  const size_t sz_tick = align_up(Bm * sizeof(unsigned));
  const size_t sz_flags = align_up(sizeof(unsigned));
  c->ws_bytes = sz_ent_part + sz_stats + sz_z + sz_lse + sz_lrow + sz_isc + sz_kphys + sz_acc + sz_ml +
                sz_rec + sz_tmax + sz_ex + sz_tick + sz_flags;
  e = hipMalloc(&c->ws, c->ws_bytes);
  if (e != hipSuccess) {
    g_init_error = std::string("workspace allocation failed: ") + hipGetErrorString(e);
    delete c;
    return ENT_E_NOMEM;
  }
  e = hipMemset(c->ws, 0, c->ws_bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    g_init_error = std::string("workspace clear failed: ") + hipGetErrorString(e);
    (void)hipFree(c->ws);
    delete c;
    return ENT_E_HIP;
  }
  char* p = static_cast<char*>(c->ws);
  auto take = [&p](size_t n) { char* r = p; p += n; return r; };
  c->ent_part = reinterpret_cast<float*>(take(sz_ent_part));
  c->stats_tmp = reinterpret_cast<float*>(take(sz_stats));
  c->zbuf = reinterpret_cast<float*>(take(sz_z));
  c->lse_part = reinterpret_cast<float*>(take(sz_lse));
  c->lrow = reinterpret_cast<float*>(take(sz_lrow));
  c->iscores = reinterpret_cast<float*>(take(sz_isc));
  c->kept_phys = reinterpret_cast<int*>(take(sz_kphys));
  c->dec_acc = reinterpret_cast<float*>(take(sz_acc));
  c->dec_ml = reinterpret_cast<float*>(take(sz_ml));
  c->dec_rec = reinterpret_cast<int4*>(take(sz_rec));
  c->tmax = sz_tmax ? reinterpret_cast<float*>(take(sz_tmax)) : nullptr;
  c->exbuf = sz_ex ? reinterpret_cast<float2*>(take(sz_ex)) : nullptr;
  c->tickets = reinterpret_cast<unsigned*>(take(sz_tick));
  c->dev_flags = reinterpret_cast<unsigned*>(take(sz_flags));
  *out = c;
  return ENT_OK;
}

int ent_destroy(ent_ctx* c) {
  if (!c) return ENT_E_INVAL;
  // The context's device is synchronised and freed on, whichever is current.
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  const bool other = e == hipSuccess && cur != c->device;
  if (other) e = hipSetDevice(c->device);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  const hipError_t e2 = hipFree(c->ws);
  const hipError_t e3 = other ? hipSetDevice(cur) : hipSuccess;
  delete c;
  return (e == hipSuccess && e2 == hipSuccess && e3 == hipSuccess) ? ENT_OK : ENT_E_HIP;
}

const char* ent_last_error(const ent_ctx* c) {
  return c ? c->err.c_str() : g_init_error.c_str();
}

int ent_device_status(ent_ctx* c, void* stream, unsigned* flags) {
  if (!c || !flags) return c ? fail(c, ENT_E_INVAL, "flags is NULL") : ENT_E_INVAL;
  if (int r = check_device(c)) return r;
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "stream synchronise");
  unsigned v = 0;
  e = hipMemcpy(&v, c->dev_flags, sizeof(unsigned), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(c->dev_flags, 0, sizeof(unsigned));
  if (e != hipSuccess) return hip_fail(c, e, "device status read");
  *flags = v;
  c->err.clear();
  return ENT_OK;
}

int ent_entropy_temperature(ent_ctx* c, int B, const float* logits, long long ld, ent_state st,
                            float* h_out, float* temp_used, float* row_stats, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  if (!logits || !st.h_prev || !st.tau || !st.temp || !h_out || !temp_used)
    return fail(c, ENT_E_INVAL, "ent_entropy_temperature: NULL required pointer");
  if (ld < c->cfg.vocab) return fail(c, ENT_E_INVAL, "ent_entropy_temperature: ld < vocab");
  if (h_out == st.h_prev) return fail(c, ENT_E_INVAL, "ent_entropy_temperature: h_out aliases h_prev");
  if (temp_used == st.temp) return fail(c, ENT_E_INVAL, "ent_entropy_temperature: temp_used aliases temp");
  const hipError_t e = ent::launch_entropy(c, B, logits, ld, st, h_out, temp_used, row_stats, true,
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_entropy_temperature launch");
  c->err.clear();
  return ENT_OK;
}

int ent_block_summary(ent_ctx* c, int B, const void* k_cache, const int* block_tables,
                      const int* ctx_lens, float* ksum, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  if (!k_cache || !block_tables || !ctx_lens || !ksum)
    return fail(c, ENT_E_INVAL, "ent_block_summary: NULL required pointer");
  if (!aligned(k_cache, 16))
    return fail(c, ENT_E_INVAL, "ent_block_summary: k_cache needs 16-byte alignment");
  const hipError_t e = ent::launch_block_summary(c, B, k_cache, block_tables, ctx_lens, ksum,
                                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_block_summary launch");
  c->err.clear();
  return ENT_OK;
}

int ent_block_select(ent_ctx* c, int B, const void* q, const float* ksum, const void* k_cache,
                     const int* block_tables, const int* ctx_lens, const float* h, int* kept,
                     int* n_kept, float* scores, float* theta, float* kappa, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  const bool exact = c->cfg.scoring == ENT_SCORE_EXACT;
  if (!q || !block_tables || !ctx_lens || !h || !kept || !n_kept)
    return fail(c, ENT_E_INVAL, "ent_block_select: NULL required pointer");
  if (exact ? !k_cache : !ksum)
    return fail(c, ENT_E_INVAL, exact ? "ent_block_select: exact scoring needs k_cache"
                                      : "ent_block_select: mean-key scoring needs ksum");
  if (!aligned(q, 16) || (exact ? !aligned(k_cache, 16) : !aligned(ksum, 16)))
    return fail(c, ENT_E_INVAL, "ent_block_select: q, ksum or k_cache misaligned");
  const hipError_t e = ent::launch_block_select(c, B, q, ksum, k_cache, block_tables, ctx_lens, h,
                                                kept, n_kept, scores, theta, kappa,
                                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_block_select launch");
  c->err.clear();
  return ENT_OK;
}

int ent_sparse_paged_decode(ent_ctx* c, int B, const void* q, const void* k_cache,
                            const void* v_cache, const int* block_tables, const int* ctx_lens,
                            const int* kept, const int* n_kept, float* out, float* lse,
                            void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  if (!q || !k_cache || !v_cache || !block_tables || !ctx_lens || !kept || !n_kept || !out)
    return fail(c, ENT_E_INVAL, "ent_sparse_paged_decode: NULL required pointer");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16))
    return fail(c, ENT_E_INVAL, "ent_sparse_paged_decode: q, caches and out need 16-byte alignment");
  const hipError_t e = ent::launch_decode(c, B, q, k_cache, v_cache, block_tables, ctx_lens, kept,
                                          n_kept, out, lse, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_sparse_paged_decode launch");
  c->err.clear();
  return ENT_OK;
}

int ent_sample(ent_ctx* c, int B, const float* logits, long long ld, const float* row_stats,
               const float* temp_used, const float* uniforms, int* tokens, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  if (!logits || !temp_used || !uniforms || !tokens)
    return fail(c, ENT_E_INVAL, "ent_sample: NULL required pointer");
  if (ld < c->cfg.vocab) return fail(c, ENT_E_INVAL, "ent_sample: ld < vocab");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float* stats = row_stats;
  if (!stats) {
    ent_state none{nullptr, nullptr, nullptr};
    const hipError_t e = ent::launch_entropy(c, B, logits, ld, none, nullptr, const_cast<float*>(temp_used),
                                             c->stats_tmp, false, s);
    if (e != hipSuccess) return hip_fail(c, e, "ent_sample statistics launch");
    stats = c->stats_tmp;
  }
  const hipError_t e = ent::launch_sample(c, B, logits, ld, stats, temp_used, uniforms, tokens, s);
  if (e != hipSuccess) return hip_fail(c, e, "ent_sample launch");
  c->err.clear();
  return ENT_OK;
}

int ent_decode_step(ent_ctx* c, int B, const float* logits, long long ld, ent_state st,
                    const void* q, const void* k_cache, const void* v_cache, const float* ksum,
                    const int* block_tables, const int* ctx_lens, const float* uniforms,
                    float* h_out, float* temp_used, float* row_stats, int* kept, int* n_kept,
                    float* out, float* lse, int* tokens, float* scores, float* theta,
                    void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  const bool exact = c->cfg.scoring == ENT_SCORE_EXACT;   // ksum unused in exact mode
  if (!logits || !st.h_prev || !st.tau || !st.temp || !q || !k_cache || !v_cache ||
      (!exact && !ksum) || !block_tables || !ctx_lens || !uniforms || !h_out || !temp_used ||
      !kept || !n_kept || !out || !tokens)
    return fail(c, ENT_E_INVAL, "ent_decode_step: NULL required pointer");
  if (ld < c->cfg.vocab) return fail(c, ENT_E_INVAL, "ent_decode_step: ld < vocab");
  if (h_out == st.h_prev) return fail(c, ENT_E_INVAL, "ent_decode_step: h_out aliases h_prev");
  if (temp_used == st.temp) return fail(c, ENT_E_INVAL, "ent_decode_step: temp_used aliases temp");
  if (!aligned(q, 16) || (!exact && !aligned(ksum, 16)) || !aligned(k_cache, 16) ||
      !aligned(v_cache, 16) || !aligned(out, 16))
    return fail(c, ENT_E_INVAL, "ent_decode_step: q, ksum, caches and out need 16-byte alignment");
  if (exact) {
    // The conservative scoring mode: the staged calls in order (every
    // argument they check was checked above, so none fails part-way).  The
    // sampler reuses the entropy pass's row statistics.
    float* stats = row_stats ? row_stats : c->stats_tmp;
    if (int r = ent_entropy_temperature(c, B, logits, ld, st, h_out, temp_used, stats, stream))
      return r;
    if (int r = ent_block_select(c, B, q, ksum, k_cache, block_tables, ctx_lens, h_out, kept,
                                 n_kept, scores, theta, st.kappa, stream))
      return r;
    if (int r = ent_sparse_paged_decode(c, B, q, k_cache, v_cache, block_tables, ctx_lens, kept,
                                        n_kept, out, lse, stream))
      return r;
    return ent_sample(c, B, logits, ld, stats, temp_used, uniforms, tokens, stream);
  }
  const hipError_t e = ent::launch_decode_step(c, B, logits, ld, st, q, k_cache, v_cache, ksum,
                                               block_tables, ctx_lens, uniforms, h_out,
                                               temp_used, row_stats, kept, n_kept, out, lse,
                                               tokens, scores, theta,
                                               static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_decode_step launch");
  c->err.clear();
  return ENT_OK;
}

int ent_decode_step_append(ent_ctx* c, int B, const float* logits, long long ld, ent_state st,
                           const void* q, void* k_cache, void* v_cache, float* ksum,
                           const int* block_tables, int* ctx_lens, const float* uniforms,
                           const void* k_new, const void* v_new, float* h_out, float* temp_used,
                           float* row_stats, int* kept, int* n_kept, float* out, float* lse,
                           int* tokens, float* scores, float* theta, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  const bool exact = c->cfg.scoring == ENT_SCORE_EXACT;
  if (!k_new || !v_new)
    return fail(c, ENT_E_INVAL, "ent_decode_step_append: NULL required pointer");
  if (!aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(c, ENT_E_INVAL, "ent_decode_step_append: k_new and v_new need 16-byte alignment");
  if (exact) {
    // The staged step, then the append.
    if (int r = ent_decode_step(c, B, logits, ld, st, q, k_cache, v_cache, ksum, block_tables,
                                ctx_lens, uniforms, h_out, temp_used, row_stats, kept, n_kept, out,
                                lse, tokens, scores, theta, stream))
      return r;
    return ent_kv_append(c, B, k_new, v_new, block_tables, ctx_lens, k_cache, v_cache, ksum,
                         stream);
  }
  if (!logits || !st.h_prev || !st.tau || !st.temp || !q || !k_cache || !v_cache || !ksum ||
      !block_tables || !ctx_lens || !uniforms || !h_out || !temp_used || !kept || !n_kept || !out ||
      !tokens)
    return fail(c, ENT_E_INVAL, "ent_decode_step_append: NULL required pointer");
  if (ld < c->cfg.vocab) return fail(c, ENT_E_INVAL, "ent_decode_step_append: ld < vocab");
  if (h_out == st.h_prev) return fail(c, ENT_E_INVAL, "ent_decode_step_append: h_out aliases h_prev");
  if (temp_used == st.temp)
    return fail(c, ENT_E_INVAL, "ent_decode_step_append: temp_used aliases temp");
  if (!aligned(q, 16) || !aligned(ksum, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
      !aligned(out, 16))
    return fail(c, ENT_E_INVAL,
                "ent_decode_step_append: q, ksum, caches and out need 16-byte alignment");
  const ent::AppendArgs ap =
      ent::make_append_args(c, k_new, v_new, block_tables, ctx_lens, k_cache, v_cache, ksum);
  const hipError_t e = ent::launch_decode_step(c, B, logits, ld, st, q, k_cache, v_cache, ksum,
                                               block_tables, ctx_lens, uniforms, h_out, temp_used,
                                               row_stats, kept, n_kept, out, lse, tokens, scores,
                                               theta, static_cast<hipStream_t>(stream), &ap);
  if (e != hipSuccess) return hip_fail(c, e, "ent_decode_step_append launch");
  c->err.clear();
  return ENT_OK;
}

int ent_kv_append(ent_ctx* c, int B, const void* k_new, const void* v_new, const int* block_tables,
                  int* ctx_lens, void* k_cache, void* v_cache, float* ksum, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_batch(c, B)) return r;
  if (B == 0) return ENT_OK;
  if (!k_new || !v_new || !block_tables || !ctx_lens || !k_cache || !v_cache ||
      (!ksum && c->cfg.scoring != ENT_SCORE_EXACT))
    return fail(c, ENT_E_INVAL, "ent_kv_append: NULL required pointer");
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16))
    return fail(c, ENT_E_INVAL, "ent_kv_append: k_new, v_new and k_cache need 16-byte alignment");
  const hipError_t e = ent::launch_kv_append(c, B, k_new, v_new, block_tables, ctx_lens, k_cache,
                                             v_cache, ksum, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_kv_append launch");
  c->err.clear();
  return ENT_OK;
}

int ent_schedule(ent_ctx* c, int N, const ent_sched_params* prm, const float* tau,
                 const int* n_kept, const int* ctx_lens, float* tau_last, float* gain, int* age,
                 int b_sel, int* selected, int* n_selected, float* priority, void* stream) {
  if (!c) return ENT_E_INVAL;
  if (int r = check_device(c)) return r;
  if (N < 0 || N > ENT_SCHED_MAX_POOL)
    return fail(c, ENT_E_INVAL, "ent_schedule: N must be in [0, ENT_SCHED_MAX_POOL]");
  if (!prm) return fail(c, ENT_E_INVAL, "ent_schedule: params is NULL");
  const ent_sched_params& p = *prm;
  if (!(p.alpha >= 0.f) || !(p.beta >= 0.f) || !(p.gamma >= 0.f) || !isfinite(p.alpha) ||
      !isfinite(p.beta) || !isfinite(p.gamma))
    return fail(c, ENT_E_INVAL, "ent_schedule: alpha, beta and gamma must be finite and >= 0");
  if (!isfinite(p.slo)) return fail(c, ENT_E_INVAL, "ent_schedule: slo must be finite");
  if (!(p.slack_floor > 0.f) || !isfinite(p.slack_floor))
    return fail(c, ENT_E_INVAL, "ent_schedule: slack_floor must be finite and > 0");
  if (!(p.gain_floor > 0.f) || !isfinite(p.gain_floor))
    return fail(c, ENT_E_INVAL, "ent_schedule: gain_floor must be finite and > 0");
  if (!(p.ewma_rate >= 0.f && p.ewma_rate <= 1.f))
    return fail(c, ENT_E_INVAL, "ent_schedule: ewma_rate must be in [0, 1]");
  if (N == 0) {
    c->err.clear();
    return ENT_OK;
  }
  if (!tau || !n_kept || !ctx_lens || !tau_last || !gain || !age || !selected || !n_selected)
    return fail(c, ENT_E_INVAL, "ent_schedule: NULL required pointer");
  const hipError_t e = ent::launch_schedule(N, p, tau, n_kept, ctx_lens, tau_last, gain, age, b_sel,
                                            selected, n_selected, priority,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "ent_schedule launch");
  c->err.clear();
  return ENT_OK;
}

}  // extern "C"
