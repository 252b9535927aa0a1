// Exact entropy of the tempered next-token distribution, the entropic-time
// and temperature controller, and inverse-CDF sampling.
//
// Entropy (Section 2 and Section 2.1 of the paper): H = -sum_x p(x) ln p(x)
// with p = softmax(z / T).  One pass over each logit row: the row is cut into
// chunks of ENT_ROW_CHUNK logits, one 256-thread workgroup per (chunk, row);
// each thread holds 16 logits in registers, so the chunk's maximum and the
// sums   S = sum 2^(t - M),  W = sum 2^(t - M) (t - M)   (t = z log2(e) / T)
// come from one read of HBM.  A second kernel (one wave per row) merges the
// chunk triples and runs the controller:
//   H = ln 2 (log2 S - W / S)
//   tau += max(0, H_prev - H)                    (Section 2, entropic time)
//   T'  = clip(T exp(eta (H - H*)), T_min, T_max)  (Section 3.3, signed eta)
// Chunk (max, sum) pairs double as the row statistics the sampler reuses.

#include "ent_internal.h"

#include <math.h>

namespace ent {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = kRowChunk / kThreads;   // 16 logits per thread
static_assert(kPerThread == 16, "chunk layout");

__device__ __forceinline__ float block_max_256(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}

__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// Loads the thread's 16 logits of chunk `c`, scaled to log2 units: t = z * c2.
// Positions past the vocabulary read as -inf (zero probability).
template <bool VEC>
__device__ __forceinline__ void load_chunk(const float* __restrict__ row, int V, int c,
                                           float c2, float (&v)[kPerThread]) {
  const int base = c * kRowChunk;
  if (VEC) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = base + (i * kThreads + threadIdx.x) * 4;
      if (idx + 3 < V) {
        const float4 x = *reinterpret_cast<const float4*>(row + idx);
        v[4 * i + 0] = x.x * c2;
        v[4 * i + 1] = x.y * c2;
        v[4 * i + 2] = x.z * c2;
        v[4 * i + 3] = x.w * c2;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          v[4 * i + k] = (idx + k < V) ? row[idx + k] * c2 : -INFINITY;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int idx = base + i * kThreads + threadIdx.x;
      v[i] = idx < V ? row[idx] * c2 : -INFINITY;
    }
  }
}

// Chunk pass: per (chunk, row) the maximum M, S = sum 2^(t - M) and
// W = sum 2^(t - M) (t - M).  Writes the triple to `part` (when non-null) and
// (M, S) to `row_stats` (when non-null).
template <bool VEC>
__global__ __launch_bounds__(kThreads) void entropy_chunk_kernel(
    const float* __restrict__ logits, long long ld, int V, int C,
    const float* __restrict__ temp,    // T_t [B]
    float* __restrict__ part,          // nullable [B, C, 3]
    float* __restrict__ row_stats) {   // nullable [B, C, 2]
  __shared__ float red[4];
  const int c = blockIdx.x;
  const int b = blockIdx.y;
  const float T = temp[b];
  const float c2 = __fdiv_rn(kLog2e, T);
  const float* row = logits + static_cast<long long>(b) * ld;

  float v[kPerThread];
  load_chunk<VEC>(row, V, c, c2, v);
  float m = v[0];
#pragma unroll
  for (int i = 1; i < kPerThread; ++i) m = fmaxf(m, v[i]);
  const float M = block_max_256(m, red);

  float S = 0.f, W = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const float d = v[i] - M;
      const float e = exp2f(d);
      S += e;
      W += (e > 0.f) ? e * d : 0.f;
    }
  }
  S = block_sum_256(S, red);
  W = block_sum_256(W, red);

  if (threadIdx.x == 0) {
    const long long o = static_cast<long long>(b) * C + c;
    if (row_stats) {
      row_stats[2 * o + 0] = M;
      row_stats[2 * o + 1] = S;
    }
    if (part) {
      part[3 * o + 0] = M;
      part[3 * o + 1] = S;
      part[3 * o + 2] = W;
    }
  }
}

// Merge of a row's C chunk triples (one wave per row) and the controller.
__global__ __launch_bounds__(kThreads) void entropy_finalize_kernel(
    int B, int C, const float* __restrict__ part, float* __restrict__ temp,
    float* __restrict__ h_prev, float* __restrict__ tau, float* __restrict__ h_out,
    float* __restrict__ temp_used, float eta, float h_target, float t_min, float t_max) {
  const int b = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (b >= B) return;
  const float* pr = part + static_cast<long long>(b) * C * 3;
  float mloc = -INFINITY;
  for (int i = lane; i < C; i += 64) mloc = fmaxf(mloc, pr[3 * i]);
  const float MG = wave_max(mloc);
  float s = 0.f, w = 0.f;
  for (int i = lane; i < C; i += 64) {
    const float mc = pr[3 * i];
    const float sc = pr[3 * i + 1];
    const float wc = pr[3 * i + 2];
    if (sc > 0.f) {
      const float dm = mc - MG;
      const float f = exp2f(dm);
      s += sc * f;
      w += f * (wc + sc * dm);
    }
  }
  s = wave_sum(s);
  w = wave_sum(w);
  if (lane == 0) {
    const float T = temp[b];
    const float H = (log2f(s) - w / s) * kLn2;
    h_out[b] = H;
    temp_used[b] = T;
    const float hp = h_prev[b];
    float ta = tau[b];
    if (!isnan(hp)) ta += fmaxf(0.f, hp - H);
    float tn = T * expf(eta * (H - h_target));
    tn = fminf(fmaxf(tn, t_min), t_max);
    tau[b] = ta;
    h_prev[b] = H;
    temp[b] = tn;
  }
}

// ---------------------------------------------------------------------------
// Inverse-CDF sampling.  One workgroup per row.  The chunk masses
// S_c 2^(M_c - M) (from the row statistics) locate the chunk that holds the
// target u S; that chunk is re-read and scanned in index order with float64
// running sums.
// ---------------------------------------------------------------------------
constexpr int kMaxChunks = kThreads;   // vocab <= 256 * 4096

__device__ __forceinline__ double block_excl_scan_d(double v, double* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(incl, o);
    if (lane >= o) incl += n;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  double before = 0.0;
  for (int i = 0; i < w; ++i) before += wsum[i];
  __syncthreads();
  return before + incl - v;
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void sample_kernel(
    const float* __restrict__ logits, long long ld, int V, int C,
    const float* __restrict__ row_stats, const float* __restrict__ temp_used,
    const float* __restrict__ uniforms, int* __restrict__ tokens) {
  __shared__ double s_w[kMaxChunks];
  __shared__ double wsum[4];
  __shared__ float red[4];
  __shared__ int s_chunk, s_idx, s_lastpos;
  __shared__ double s_before, s_target;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const float T = temp_used[b];
  const float c2 = __fdiv_rn(kLog2e, T);
  const float* row = logits + static_cast<long long>(b) * ld;
  const float* st = row_stats + static_cast<long long>(b) * C * 2;

  const float mc = t < C ? st[2 * t] : -INFINITY;
  const float sc = t < C ? st[2 * t + 1] : 0.f;
  const float M = block_max_256(mc, red);
  s_w[t] = (t < C && sc > 0.f) ? static_cast<double>(sc) *
                                     exp2(static_cast<double>(mc) - static_cast<double>(M))
                               : 0.0;
  if (t == 0) {
    s_idx = 0x7fffffff;
    s_lastpos = -1;
  }
  __syncthreads();
  if (t == 0) {
    double tot = 0.0;
    for (int i = 0; i < C; ++i) tot += s_w[i];
    const double target = static_cast<double>(uniforms[b]) * tot;
    double cum = 0.0;
    int chunk = -1, lastpos = 0;
    double before = 0.0;
    for (int i = 0; i < C; ++i) {
      if (s_w[i] > 0.0) lastpos = i;
      if (chunk < 0 && cum + s_w[i] > target) {
        chunk = i;
        before = cum;
      }
      cum += s_w[i];
    }
    double tgt = target;
    if (chunk < 0) {            // rounding put the target at the very top:
      chunk = lastpos;          // take the last token of positive mass
      before = 0.0;
      tgt = HUGE_VAL;
    }
    s_chunk = chunk;
    s_before = before;
    s_target = tgt;
  }
  __syncthreads();
  const int chunk = s_chunk;
  const int base = chunk * kRowChunk + t * kPerThread;
  float e[kPerThread];
  if (VEC && base + kPerThread <= V) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 x = *reinterpret_cast<const float4*>(row + base + 4 * i);
      e[4 * i + 0] = exp2f(x.x * c2 - M);
      e[4 * i + 1] = exp2f(x.y * c2 - M);
      e[4 * i + 2] = exp2f(x.z * c2 - M);
      e[4 * i + 3] = exp2f(x.w * c2 - M);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i)
      e[i] = (base + i < V) ? exp2f(row[base + i] * c2 - M) : 0.f;
  }
  double local = 0.0;
  int lastpos = -1;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    local += static_cast<double>(e[i]);
    if (e[i] > 0.f) lastpos = base + i;
  }
  double pos = s_before + block_excl_scan_d(local, wsum);
  const double target = s_target;
  int found = 0x7fffffff;
  for (int i = 0; i < kPerThread; ++i) {
    pos += static_cast<double>(e[i]);
    if (pos > target) {
      found = base + i;
      break;
    }
  }
  if (found != 0x7fffffff) atomicMin(&s_idx, found);
  if (lastpos >= 0) atomicMax(&s_lastpos, lastpos);
  __syncthreads();
  if (t == 0) tokens[b] = (s_idx != 0x7fffffff) ? s_idx : s_lastpos;
}

bool row_vec_ok(const float* p, long long ld) {
  return (reinterpret_cast<uintptr_t>(p) % 16 == 0) && (ld % 4 == 0);
}

}  // namespace

hipError_t launch_entropy(const ent_ctx* c, int B, const float* logits, long long ld,
                          ent_state st, float* h_out, float* temp_used, float* row_stats,
                          bool controller, hipStream_t s) {
  const ent_config& cf = c->cfg;
  const dim3 grid(c->chunks, B);
  const bool vec = row_vec_ok(logits, ld);
  auto k = vec ? entropy_chunk_kernel<true> : entropy_chunk_kernel<false>;
  // Without the controller (statistics for the sampler) the temperatures are
  // the ones passed in temp_used.
  const float* T = controller ? st.temp : temp_used;
  hipLaunchKernelGGL(k, grid, dim3(kThreads), 0, s, logits, ld, cf.vocab, c->chunks, T,
                     controller ? c->ent_part : nullptr, row_stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !controller) return e;
  const int rows_per_wg = kThreads / 64;
  hipLaunchKernelGGL(entropy_finalize_kernel, dim3((B + rows_per_wg - 1) / rows_per_wg),
                     dim3(kThreads), 0, s, B, c->chunks, c->ent_part, st.temp, st.h_prev, st.tau,
                     h_out, temp_used, cf.eta, cf.h_target, cf.t_min, cf.t_max);
  return hipGetLastError();
}

hipError_t launch_sample(const ent_ctx* c, int B, const float* logits, long long ld,
                         const float* row_stats, const float* temp_used, const float* uniforms,
                         int* tokens, hipStream_t s) {
  const bool vec = row_vec_ok(logits, ld);
  auto k = vec ? sample_kernel<true> : sample_kernel<false>;
  hipLaunchKernelGGL(k, dim3(B), dim3(kThreads), 0, s, logits, ld, c->cfg.vocab, c->chunks,
                     row_stats, temp_used, uniforms, tokens);
  return hipGetLastError();
}

}  // namespace ent
