/*
 * ent.h -- C ABI of the entropic-time decode step on MI355X (gfx950).
 *
 * One batched decode step of entropic-time inference (arXiv 2603.03310):
 * per sequence, the exact Shannon entropy of the next-token distribution,
 * entropic time and the temperature control law, entropy-driven pruning of
 * the paged KV cache, decode attention over the kept blocks, and sampling at
 * the controlled temperature.
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers owned by the caller, unless a parameter says
 *    "host".  The context owns only its workspace, allocated once by ent_init.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL is
 *    the default stream).  They allocate nothing and never synchronise, except
 *    ent_init, ent_destroy and ent_device_status.
 *  - Arguments are validated on the host before anything is launched.  A bad
 *    argument returns ENT_E_INVAL (or ENT_E_UNSUPPORTED) with nothing launched,
 *    and a message for ent_last_error.  A HIP failure returns ENT_E_HIP.
 *    Outputs are undefined after an error.
 *  - Device-side checks: a block table entry outside [0, num_pool_blocks) or a
 *    context length outside [0, max_blocks_per_seq * 16] is never
 *    dereferenced; the kernel skips it and raises a flag that
 *    ent_device_status reports.
 *  - A context is not thread-safe; calls that share a context must be ordered
 *    on one stream (the workspace is reused by every call).
 *  - A context belongs to the HIP device current at ent_init; every call on it
 *    must be made with that device current (else ENT_E_INVAL, nothing
 *    launched).  ent_destroy accepts any current device.
 *  - Batch sizes: 0 <= B <= max_batch.  B == 0 launches nothing.
 *
 * Paged KV cache layout (block size 16 tokens, P = num_pool_blocks):
 *    k_cache [P, H_kv, 16, d]   token-major tile per (physical block, KV head)
 *    v_cache [P, H_kv, d, 16]   dim-major tile per (physical block, KV head)
 *  element type kv_dtype (bf16 or fp32); queries have the same type.  Logical
 *  token i of sequence b is slot i % 16 of physical block
 *  block_tables[b * max_blocks_per_seq + i / 16].  A sequence of N tokens
 *  occupies nb = ceil(N / 16) logical blocks; the last holds N - 16 (nb - 1).
 */
#ifndef ENT_H
#define ENT_H

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ent_ctx ent_ctx;

enum {
  ENT_OK = 0,
  ENT_E_INVAL = -1,        /* bad argument: nothing launched */
  ENT_E_NOMEM = -2,        /* workspace allocation failed (ent_init) */
  ENT_E_HIP = -3,          /* a HIP runtime call or launch failed */
  ENT_E_UNSUPPORTED = -4   /* shape outside what the kernels implement */
};

enum { ENT_F32 = 0, ENT_BF16 = 1 };

/* Entropy the controller acts on (Section 2.1 and Section 3.3, "Entropy
 * estimator in the control loop"): the exact entropy, the top-k truncated
 * entropy H~ of the renormalised top-k distribution, or the tail-corrected
 * estimate H^ = H~ + h(mbar) + mbar ln(|V| - k) (mbar = probability mass
 * outside the top-k set, h the binary entropy).  With k >= |V| both
 * estimates equal the exact entropy. */
enum { ENT_EST_EXACT = 0, ENT_EST_TOPK = 1, ENT_EST_TAIL = 2 };
#define ENT_EST_MAX_K 512

/* Block scoring (Section 3.2: I_b is the attention-weighted surprisal of
 * block b's tokens).  MEANKEY: the weights of the current query when every
 * token carries its block's mean key (one summary per block and KV head is
 * read).  EXACT: the token-level softmax of the current query over every
 * valid key of the sequence (every key is read: the conservative mode). */
enum { ENT_SCORE_MEANKEY = 0, ENT_SCORE_EXACT = 1 };

/* Tokens per logical row chunk of the entropy reduction; row statistics hold
 * one (max, sum) pair per chunk: ent_row_stats_chunks(vocab) chunks per row. */
#define ENT_ROW_CHUNK 4096
#define ENT_BLOCK_SIZE 16

/* Device-status flags (ent_device_status). */
#define ENT_DEV_BAD_TABLE 1u     /* a block table entry was out of range */
#define ENT_DEV_BAD_CTXLEN 2u    /* a context length was out of range */
#define ENT_DEV_CACHE_FULL 4u    /* append found no room in the block table */

/* Shapes and control parameters; host values, copied by ent_init.
 * The paper names the control symbols but gives no values (Section 3.3, the
 * temperature law and the estimator error bound; Section 3.3 "Conservative
 * pruning under uncertainty bounds" and Section 5 for H_min and B_min). */
typedef struct {
  int max_batch;           /* largest B any call will pass, >= 1 */
  int num_q_heads;         /* H_q */
  int num_kv_heads;        /* H_kv; H_q % H_kv == 0, G = H_q / H_kv in {1,2,4,8,16},
                              H_q <= 128, H_kv * head_dim <= 2048 */
  int head_dim;            /* d: 64 or 128 */
  int block_size;          /* tokens per KV block: must be 16 */
  int max_blocks_per_seq;  /* MAXB: row length of block_tables, <= 16384;
                              max_batch * MAXB * H_kv < 2^31 */
  int num_pool_blocks;     /* P: physical blocks in k_cache / v_cache, < 2^30 */
  int vocab;               /* |V|: logits per row */
  int kv_dtype;            /* ENT_BF16 or ENT_F32 (K, V and queries) */
  float scale;             /* softmax scale of scoring and attention, e.g. 1/sqrt(d) */
  float eta;               /* SIGNED gain of the temperature law; < 0 stabilises */
  float h_target;          /* target entropy H* (nats) */
  float t_min, t_max;      /* temperature clip bounds, 0 < t_min <= t_max */
  float eps_h;             /* entropy estimator error bound (0 for exact entropy) */
  float h_min;             /* entropy floor for pruning decisions */
  float kappa_min;         /* smallest kept fraction of blocks, in [0, 1] */
  int b_min;               /* smallest number of kept blocks, >= 0 */
  float log_v;             /* log |V| as float32; must exceed h_min */
  int estimator;           /* ENT_EST_EXACT, ENT_EST_TOPK or ENT_EST_TAIL; with an estimate,
                              eps_h is its error bound and enters the block budget */
  int est_k;               /* k of the estimators, 1 <= k <= ENT_EST_MAX_K (ignored when exact) */
  /* Calibration and safe control (Section 5).  Neutral values leave the
   * step unchanged: t_cal = 1, rho_t = INFINITY, dkappa = 1, h_bias = 0. */
  float t_cal;             /* calibration temperature, > 0: every softmax over the vocabulary
                              (entropy, estimates, sampling) uses z / (t_cal * T_t) */
  float rho_t;             /* bound on |ln T_{t+1} - ln T_t|: the temperature step
                              exp(eta (H - H*)) is clipped to [e^-rho_t, e^rho_t]; >= 0 or INFINITY */
  float dkappa;            /* largest decrease of a sequence's kept fraction per step, in [0, 1];
                              needs the kept-fraction state (ent_state.kappa) */
  float h_bias;            /* offset added to the entropy the controller and budget act on
                              (miscalibration stress tests); finite */
  int scoring;             /* ENT_SCORE_MEANKEY (default) or ENT_SCORE_EXACT */
  int keep_first;          /* leading logical blocks always kept, >= 0 (0 = none) */
  int keep_last;           /* trailing logical blocks always kept, >= 0 (0 = none); forced
                              blocks count toward the budget k (it becomes max(k, forced)) */
} ent_config;

/* Per-sequence controller state, device arrays of B floats each, read and
 * updated in place by ent_entropy_temperature: the previous step's entropy
 * H_{t-1} (NaN = no previous step), entropic time tau, and temperature T_t.
 * kappa (nullable): the previous step's kept fraction of blocks (NaN = none),
 * read and updated by the block selection; the rate guard dkappa applies
 * only when it is given. */
typedef struct {
  float* h_prev;
  float* tau;
  float* temp;
  float* kappa;
} ent_state;

/* Defaults: Llama-3-8B decode shapes (32/8 heads, d = 128, bf16, |V| = 128256),
 * eta = -0.05, H* = 2.5, T in [0.05, 5], eps_H = 0, H_min = H*, kappa_min = 0.05,
 * B_min = 4, exact entropy (est_k = 256 for the estimators), no calibration or
 * rate guards, no bias.  max_batch, max_blocks_per_seq and num_pool_blocks
 * must be set. */
void ent_default_config(ent_config* out);

/* Host-only check of a configuration (no HIP call).  Returns ENT_OK, or
 * ENT_E_INVAL / ENT_E_UNSUPPORTED and writes a message into msg (host buffer
 * of msg_len bytes; may be NULL). */
int ent_check_config(const ent_config* cfg, char* msg, int msg_len);

/* Number of row-statistics chunks per logit row: ceil(vocab / ENT_ROW_CHUNK). */
int ent_row_stats_chunks(int vocab);

/* Create a context on the current HIP device: validates cfg, allocates and
 * zeroes the workspace (size grows with max_batch, H_q, MAXB).  *out receives
 * the context (host pointer) or NULL on error. */
int ent_init(const ent_config* cfg, ent_ctx** out);

/* Free the workspace and the context.  Synchronises the device first. */
int ent_destroy(ent_ctx* c);

/* Message of the last error on this context ("" if none).  The string is
 * owned by the context and valid until its next call.  ent_last_error(NULL)
 * returns the message of the last failed ent_init. */
const char* ent_last_error(const ent_ctx* c);

/* Synchronise `stream`, then return in *flags (host) the ENT_DEV_* flags
 * raised by kernels since the last call, and clear them. */
int ent_device_status(ent_ctx* c, void* stream, unsigned* flags);

/* Entropy and controller (Section 2: H_t, Delta H_t, entropic time tau;
 * Section 2.1: exact entropy of the tempered softmax and its top-k and
 * tail-corrected estimates; Section 3.3: the temperature law
 * T_{t+1} = clip(T_t exp(eta (H_t - H*)), T_min, T_max)).
 *
 * For each row b < B of logits (fp32, row stride ld >= vocab elements):
 *   H_t      = -sum_x p(x) ln p(x),  p = softmax(z / T_t),  T_t = st.temp[b]
 *              (or the configured estimate of it, cfg.estimator)
 *   h_out[b] = H_t;  temp_used[b] = T_t
 *   st.tau[b]   += max(0, st.h_prev[b] - H_t)   (unchanged if h_prev is NaN)
 *   st.h_prev[b] = H_t;  st.temp[b] = T_{t+1}
 * row_stats (nullable): float [B, ent_row_stats_chunks(vocab), 2] chunk
 * statistics of the same pass at T_t, reused by ent_sample.
 * Preconditions: >= 1 finite logit per row, temp > 0.  h_out must not alias
 * st.h_prev; temp_used must not alias st.temp. */
int ent_entropy_temperature(ent_ctx* c, int B, const float* logits, long long ld,
                            ent_state st, float* h_out, float* temp_used, float* row_stats,
                            void* stream);

/* ent_entropy_temperature for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Needs no context and allocates nothing: the configuration
 * is passed directly (host pointer, checked as by ent_init; only vocab,
 * max_batch, the controller and estimator fields and head_dim matter), and
 * the kernels' scratch (the chunk partials of the entropy pass, and with an
 * estimator the chunk threads' logit maxima) is a static device array of
 * ENT_NOALLOC_SCRATCH_BYTES that each GPU holds until the process ends.
 * Arguments and results as in ent_entropy_temperature, bit-identical to it.
 * Limit: 12 B ceil(vocab / 4096) bytes (+ 1024 B ceil(vocab / 4096) with an
 * estimator) + 256, each term rounded up to 256, must fit the array, else
 * ENT_E_UNSUPPORTED with nothing launched (e.g. B <= 4096 rows of 128256
 * logits with the exact entropy, B <= 63 with an estimator).  Every call on
 * a GPU shares that GPU's array: calls that overlap on one GPU (two streams,
 * two threads) race and give undefined results.  Errors: ent_last_error(NULL). */
#define ENT_NOALLOC_SCRATCH_BYTES (2u << 20)
int ent_entropy_temperature_noalloc(const ent_config* cfg, int B, const float* logits,
                                    long long ld, ent_state st, float* h_out, float* temp_used,
                                    float* row_stats, void* stream);

/* Per-block mean keys (the summaries block scoring reads).  For each
 * sequence b < B and logical block j < nb_b, with p = block_tables[b][j]:
 *   ksum[p, g, :] = (1/n_j) sum over the n_j valid slots of k_cache[p, g, slot, :]
 * ksum: float [P, H_kv, d], indexed by physical block.  Entries of blocks not
 * listed are left untouched.  ctx_lens: int [B].  k_cache: 16-byte aligned.
 * Each mean sums the slots in slot order, as ent_kv_append's refresh does,
 * so both give the same bits. */
int ent_block_summary(ent_ctx* c, int B, const void* k_cache, const int* block_tables,
                      const int* ctx_lens, float* ksum, void* stream);

/* Block scores and kept-block selection (Section 3.2: block entropic
 * contribution I_b and the kept set B_t = {b : I_b >= theta_t}; Section 3.3
 * and Section 5: the safety floor, the minimum block budget and the bounded
 * rate of change of the threshold).
 *   ENT_SCORE_MEANKEY:
 *   z_bh  = scale <q_h, ksum[p_b, h / G]>,  weights a_bh = e^{z_bh} / sum_b' n_b' e^{z_b'h}
 *   I_b   = (1/H_q) sum_h n_b a_bh (-ln a_bh)
 *   ENT_SCORE_EXACT (reads k_cache; ksum unused):
 *   s_ih  = scale <q_h, k_i>,  a_ih = softmax over the valid tokens i of s_.h
 *   I_b   = (1/H_q) sum_h sum_{i in b} a_ih (-ln a_ih)
 *   H_g   = max(h[b] + eps_H, H_min);  u = clip((H_g - H_min)/(log_v - H_min), 0, 1)
 *   kappa = kappa_min + (1 - kappa_min) u, then max(kappa, kappa[b] - dkappa) when the
 *           state kappa is given and kappa[b] is not NaN
 *   k     = min(nb, max(min(B_min, nb), ceil(kappa nb)))
 *           (float32, in exactly this order, no fused multiply-add)
 *   F     = the first keep_first and the last keep_last blocks (forced keeps)
 *   theta = max(k, |F|)-th largest of I_b, with +inf for the blocks of F;
 *   kept  = F + {b : I_b >= theta} in ascending order
 * kappa (nullable, in/out): the kept-fraction state; receives this step's
 * fraction for every sequence with blocks.
 * q: [B, H_q, d] (kv_dtype); ksum from ent_block_summary (mean-key mode);
 * k_cache (exact mode; may be NULL otherwise); h: float [B] (the entropy
 * from ent_entropy_temperature).  Outputs: kept int [B, MAXB] (first
 * n_kept[b] entries valid, logical block ids), n_kept int [B]; scores
 * (nullable) float [B, MAXB] (I_b for b < nb, forced blocks included);
 * theta (nullable) float [B] (+inf when nothing is kept, or when the forced
 * blocks fill the budget). */
int ent_block_select(ent_ctx* c, int B, const void* q, const float* ksum, const void* k_cache,
                     const int* block_tables, const int* ctx_lens, const float* h, int* kept,
                     int* n_kept, float* scores, float* theta, float* kappa, void* stream);

/* Decode attention over the kept blocks only (Section 3.2: attention is
 * restricted to B_t).  For query head h (KV head g = h / G), over the valid
 * tokens i of the kept blocks of sequence b:
 *   s_i = scale <q_h, k_i>;  out[b, h, :] = sum_i softmax(s)_i v_i;
 *   lse[b, h] = ln sum_i e^{s_i}
 * The softmax is renormalised over the kept tokens.  An empty kept set gives
 * out = 0 and lse = -inf.  out: float [B, H_q, d]; lse (nullable) float [B, H_q]. */
int ent_sparse_paged_decode(ent_ctx* c, int B, const void* q, const void* k_cache,
                            const void* v_cache, const int* block_tables, const int* ctx_lens,
                            const int* kept, const int* n_kept, float* out, float* lse,
                            void* stream);

/* Sampling at the controlled temperature (Sections 2.1 and 3.3).  Token of
 * row b = inverse CDF of softmax(z / temp_used[b]) in index order at the
 * uniform uniforms[b] in [0, 1): the smallest x with C_x > u S (C the running
 * sum of e^{z/T - max}, S its total), or the last token of positive mass if
 * rounding leaves none.  row_stats (nullable) must come from
 * ent_entropy_temperature on the same logits and temperatures; when NULL the
 * statistics are recomputed (one more pass over the logits).  tokens: int [B]. */
int ent_sample(ent_ctx* c, int B, const float* logits, long long ld, const float* row_stats,
               const float* temp_used, const float* uniforms, int* tokens, void* stream);

/* The whole decode step of Sections 2 to 3.3 in one call, bit-identical to
 * ent_entropy_temperature, ent_block_select, ent_sparse_paged_decode and
 * ent_sample called in that order on the same arguments (row_stats and
 * temp_used passed from the first to the last).  The entropy passes and the
 * block scoring share one launch; the per-sequence entropy, controller and
 * selection share a second; decode attention follows, and sampling shares
 * the launch that merges the split attention segments.  In the exact
 * scoring mode the step is the four staged calls in order and ksum may be
 * NULL.
 * Arguments as in those calls: st is updated in place (tau, h_prev, temp
 * for the next step); h_out, temp_used, tokens: [B]; kept, n_kept, out as
 * in ent_sparse_paged_decode; row_stats, lse, scores, theta nullable.
 * Alignment: q and ksum 16 bytes (and the caches and out, as for decode). */
int ent_decode_step(ent_ctx* c, int B, const float* logits, long long ld, ent_state st,
                    const void* q, const void* k_cache, const void* v_cache, const float* ksum,
                    const int* block_tables, const int* ctx_lens, const float* uniforms,
                    float* h_out, float* temp_used, float* row_stats, int* kept, int* n_kept,
                    float* out, float* lse, int* tokens, float* scores, float* theta,
                    void* stream);

/* Append one token per sequence to the paged cache (the memory part of the
 * step's state, Section 3).  With N = ctx_lens[b] and p = block_tables[b][N/16]:
 * write k_new[b, g, :] to k_cache[p, g, N%16, :] and v_new[b, g, :] to
 * v_cache[p, g, :, N%16], recompute ksum[p, g, :] over the block's N%16 + 1
 * valid slots (bit-identical to ent_block_summary), and set ctx_lens[b] = N+1.
 * k_new, v_new: [B, H_kv, d] (kv_dtype).  ksum may be NULL in the exact
 * scoring mode, which does not read summaries (then none is maintained).
 * Alignment: k_new, v_new and k_cache 16 bytes. */
int ent_kv_append(ent_ctx* c, int B, const void* k_new, const void* v_new,
                  const int* block_tables, int* ctx_lens, void* k_cache, void* v_cache,
                  float* ksum, void* stream);

/* One step of the closed loop (Section 3.4: the step's outputs, then the
 * state's memory grows by the new token): ent_decode_step followed by
 * ent_kv_append of this step's new token, bit-identical to the two calls in
 * that order.  k_new, v_new: [B, H_kv, d] (kv_dtype, 16-byte aligned).  The
 * append runs on workgroups of its own inside the step's last launch, the
 * merge of split attention segments, which reads nothing the append writes
 * (in the exact scoring mode: the staged calls, then the append).
 * Arguments as in the two calls: ctx_lens is incremented, k_cache, v_cache
 * and ksum receive the new token. */
int ent_decode_step_append(ent_ctx* c, int B, const float* logits, long long ld, ent_state st,
                           const void* q, void* k_cache, void* v_cache, float* ksum,
                           const int* block_tables, int* ctx_lens, const float* uniforms,
                           const void* k_new, const void* v_new, float* h_out, float* temp_used,
                           float* row_stats, int* kept, int* n_kept, float* out, float* lse,
                           int* tokens, float* scores, float* theta, void* stream);

/* Entropy-aware scheduling over a pool of N active sequences (Section 3.1:
 * the priority pi(s) = E[Delta H_s] / (alpha C_s + beta M_s + gamma L_s);
 * Section 7: nonnegative bounded terms, no starvation).  Readings: the
 * expected gain is a running mean g of the sequence's entropy drops (its
 * entropic time increments), C_s the blocks it kept at its last step, M_s
 * the blocks it holds, ceil(N_s / 16), and L_s its slack against a service
 * objective of slo steps, which shrinks while it waits. */
typedef struct {
  float alpha, beta, gamma;  /* cost weights, finite and >= 0 */
  float slo;                 /* service objective, in steps, finite */
  float slack_floor;         /* smallest slack, finite and > 0 */
  float gain_floor;          /* smallest expected gain, finite and > 0 */
  float ewma_rate;           /* weight lam of the newest drop, in [0, 1] */
} ent_sched_params;
#define ENT_SCHED_MAX_POOL 8192

/* One scheduling call (one workgroup; N <= ENT_SCHED_MAX_POOL).  For each
 * sequence s < N, with a_s = age[s] on entry:
 *   if a_s == 0 (it ran since the last call):
 *       gain[s] = (1 - lam) gain[s] + lam (tau[s] - tau_last[s]);  tau_last[s] = tau[s]
 *   pi_s = max(gain[s], gain_floor) /
 *          (alpha max(n_kept[s], 0) + beta ceil(max(ctx_lens[s], 0) / 16)
 *           + gamma max(slo - a_s, slack_floor))
 *   (float32, in exactly this order, no fused multiply-add)
 * The min(b_sel, N) largest pi are selected, equal priorities to the lower
 * index; selected[0 .. n_selected) receives their indices in ascending order
 * (int [N] of room), *n_selected (device int) their number; age[s] becomes 0
 * when selected and a_s + 1 otherwise.  tau: float [N], entropic time (as
 * updated by the decode step); n_kept, ctx_lens: int [N]; tau_last, gain
 * (float [N]) and age (int [N]) are the scheduler state, updated in place
 * (start: tau_last = tau, gain = 0 or a prior, age = 0).  priority
 * (nullable): float [N], receives pi.  b_sel < 0 selects none.  N == 0
 * launches nothing (n_selected is not written).  c serves for error
 * messages only. */
int ent_schedule(ent_ctx* c, int N, const ent_sched_params* prm, const float* tau,
                 const int* n_kept, const int* ctx_lens, float* tau_last, float* gain, int* age,
                 int b_sel, int* selected, int* n_selected, float* priority, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ENT_H */
