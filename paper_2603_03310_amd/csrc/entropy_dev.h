// Device bodies of the entropy, controller and sampling stages, shared by
// the per-stage kernels (entropy.hip, prologue.hip) and the fused step
// kernels (step.hip, decode.hip).
//
// Entropy (Section 2 and Section 2.1 of the paper): H = -sum_x p(x) ln p(x)
// with p = softmax(z / T).  One pass over each logit row: the row is cut into
// chunks of ENT_ROW_CHUNK logits, one 256-thread workgroup per (chunk, row);
// each thread holds 16 logits in registers, so the chunk's maximum and the sums
//   S = sum 2^(t - M),  W = sum 2^(t - M) (t - M)   (t = z log2(e) / T)
// come from one read of HBM.  One wave per row then merges the chunk triples:
//   H = ln 2 (log2 S - W / S)
// and the controller updates the sequence's state:
//   tau += max(0, H_prev - H)                      (Section 2, entropic time)
//   T'  = clip(T exp(eta (H - H*)), T_min, T_max)    (Section 3.3, signed eta)
// Chunk (max, sum) pairs double as the row statistics the sampler reuses.
//
// Sampling: the chunk masses S_c 2^(M_c - M) locate the chunk holding the
// target u S; that chunk is re-read and scanned in index order with float64
// running sums.
#pragma once

#include "ent_internal.h"

#include <math.h>

namespace ent {
namespace {

constexpr int kChunkThreads = 256;
constexpr int kPerThread = kRowChunk / kChunkThreads;   // 16 logits per thread
static_assert(kPerThread == 16, "chunk layout");
constexpr int kSampleThreads = 256;                     // threads that scan a chunk
constexpr int kMaxChunks = 256;                         // vocab <= 256 * 4096

// Reductions over the first NT threads of the workgroup (NT a multiple of
// 64); every thread of the workgroup must call them.
template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0 && w < NT / 64) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, red[i]);
  __syncthreads();
  return r;
}

template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0 && w < NT / 64) red[w] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; i += 2) r += (i + 1 < NT / 64) ? (red[i] + red[i + 1]) : red[i];
  __syncthreads();
  return r;
}

// The thread's 16 logits of chunk c (unscaled).  Positions past the
// vocabulary read as -inf (zero probability).
template <bool VEC>
__device__ __forceinline__ void load_chunk(const float* __restrict__ row, int V, int c,
                                           float (&v)[kPerThread]) {
  const int base = c * kRowChunk;
  if (VEC && base + kRowChunk <= V) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 x = *reinterpret_cast<const float4*>(row + base + (i * kChunkThreads + threadIdx.x) * 4);
      v[4 * i + 0] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
  } else {
    // Ragged or unaligned: every load from an index clamped into the row,
    // so all sixteen are in flight together (no branch per load).
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int idx = base + (i * kChunkThreads + threadIdx.x) * 4 + k;
        const float x = row[min(idx, V - 1)];
        v[4 * i + k] = idx < V ? x : -INFINITY;
      }
  }
}

// Chunk pass of (chunk c, row b) by a 256-thread workgroup: writes the triple
// (M, S, W) to part (when non-null), (M, S) to row_stats (when non-null) and
// each thread's largest scaled logit to tmax[b, c, thread] (when non-null:
// the top-k estimators select from these).
template <bool VEC>
__device__ __forceinline__ void entropy_chunk_body(const float* __restrict__ logits, long long ld,
                                                   int V, int C, const float* __restrict__ temp,
                                                   float t_cal, float* __restrict__ part,
                                                   float* __restrict__ row_stats,
                                                   float* __restrict__ tmax, int c, int b,
                                                   float* red) {
  static_assert(kChunkThreads == kEstChunkThreads, "thread maxima per chunk");
  const float* row = logits + static_cast<long long>(b) * ld;
  float v[kPerThread];
  load_chunk<VEC>(row, V, c, v);
  // The logits are in flight before the temperature is waited for.
  __builtin_amdgcn_sched_barrier(0);
  const float T = temp[b] * t_cal;          // effective temperature (calibration wrapper)
  const float c2 = __fdiv_rn(kLog2e, T);
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) v[i] *= c2;   // log2 units: t = z * c2
  float m = v[0];
#pragma unroll
  for (int i = 1; i < kPerThread; ++i) m = fmaxf(m, v[i]);
  if (tmax) tmax[(static_cast<long long>(b) * C + c) * kChunkThreads + threadIdx.x] = m;
  const float M = block_max<kChunkThreads>(m, red);
  float S = 0.f, W = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      // d <= 0: the hardware exp2 (no denormal-range fix-up; terms below
      // 2^-126 of the chunk maximum do not change S or W).
      const float d = v[i] - M;
      const float e = __builtin_amdgcn_exp2f(d);
      S += e;
      W += (e > 0.f) ? e * d : 0.f;
    }
  }
  S = block_sum<kChunkThreads>(S, red);
  W = block_sum<kChunkThreads>(W, red);
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

// Entropy of row b from its C chunk triples, by one wave (result in every lane).
__device__ __forceinline__ float row_entropy(const float* __restrict__ part, int C, int b) {
  const int lane = threadIdx.x & 63;
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
  {
    // No contraction here or in the controller: the entropy must be the same
    // rounded float whether a caller keeps it in a register or reloads it.
#pragma clang fp contract(off)
    return (log2f(s) - w / s) * kLn2;
  }
}

// Controller update of sequence b given its entropy H (or estimate) at its
// controlled temperature T (temp_used nullable: the fused step records T_t
// earlier).  The controller acts on H + h_bias (0 outside stress tests); the
// temperature's multiplicative step exp(eta (H - H*)) is clipped to
// [e^-rho_t, e^rho_t] (no-op for rho_t = inf) before the clip to
// [T_min, T_max].  Returns the entropy acted on (the budget's input).
__device__ __forceinline__ float controller_update(int b, float H, float T, float* h_prev,
                                                   float* tau, float* temp, float* h_out,
                                                   float* temp_used, const Control& ct) {
#pragma clang fp contract(off)
  H = H + ct.h_bias;
  h_out[b] = H;
  if (temp_used) temp_used[b] = T;
  const float hp = h_prev[b];
  float ta = tau[b];
  if (!isnan(hp)) ta += fmaxf(0.f, hp - H);
  float step = expf(ct.eta * (H - ct.h_target));
  step = fminf(fmaxf(step, expf(-ct.rho_t)), expf(ct.rho_t));
  float tn = T * step;
  tn = fminf(fmaxf(tn, ct.t_min), ct.t_max);
  tau[b] = ta;
  h_prev[b] = H;
  temp[b] = tn;
  return H;
}

// Exclusive prefix sum (float64) over the first kSampleThreads threads.
__device__ __forceinline__ double block_excl_scan_d(double v, double* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(incl, o);
    if (lane >= o) incl += n;
  }
  if (lane == 63 && w < kSampleThreads / 64) wsum[w] = incl;
  __syncthreads();
  double before = 0.0;
  for (int i = 0; i < w && i < kSampleThreads / 64; ++i) before += wsum[i];
  __syncthreads();
  const double excl = __shfl_up(incl, 1);
  return before + (lane == 0 ? 0.0 : excl);
}

struct SampleShared {
  double wsum[kSampleThreads / 64];
  int chunk, idx, lastpos;
  float M;
  double before, target;
};

// Inverse-CDF sample of row b at temperature T and uniform u.  Every thread
// of the workgroup calls it; the first kSampleThreads threads do the work.
// Returns the token (meaningful in thread 0).  The first wave picks the
// chunk: lane l holds chunks 4 l .. 4 l + 3 (kMaxChunks = 256), their masses
// 2^(M_c - M) S_c in double, a wave scan of the lanes' sums, the lane where
// the running mass first exceeds u times the total by a ballot, then the
// chunk within that lane by a sequential walk.
template <bool VEC>
__device__ __forceinline__ int sample_body(const float* __restrict__ logits, long long ld, int V,
                                           int C, const float* __restrict__ stats, float T,
                                           float u, int b, SampleShared& sh) {
  static_assert(kMaxChunks == 4 * 64, "four chunks per lane of one wave");
  const int t = threadIdx.x;
  const bool worker = t < kSampleThreads;
  const float c2 = __fdiv_rn(kLog2e, T);
  const float* row = logits + static_cast<long long>(b) * ld;
  const float* st = stats + static_cast<long long>(b) * C * 2;
  if (t < 64) {
    constexpr int PER = kMaxChunks / 64;
    float mc[PER], sc[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = PER * t + k;
      mc[k] = i < C ? st[2 * i] : -INFINITY;
      sc[k] = i < C ? st[2 * i + 1] : 0.f;
    }
    float ml = mc[0];
#pragma unroll
    for (int k = 1; k < PER; ++k) ml = fmaxf(ml, mc[k]);
    const float M = wave_max(ml);
    double wl[PER];
    int lastk = -1;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      wl[k] = (PER * t + k < C && sc[k] > 0.f)
                  ? static_cast<double>(sc[k]) * exp2(static_cast<double>(mc[k]) - static_cast<double>(M))
                  : 0.0;
      if (wl[k] > 0.0) lastk = k;
    }
    double loc = 0.0;
#pragma unroll
    for (int k = 0; k < PER; ++k) loc += wl[k];
    double incl = loc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double n = __shfl_up(incl, o);
      if (t >= o) incl += n;
    }
    const double tot = __shfl(incl, 63);
    const double target = static_cast<double>(u) * tot;
    // The lane's running mass, stepped chunk by chunk from its exclusive prefix.
    double cum = incl - loc, run = cum;
#pragma unroll
    for (int k = 0; k < PER; ++k) run += wl[k];
    const unsigned long long hit = __ballot(run > target);
    if (hit != 0ull) {
      if (t == __ffsll(static_cast<long long>(hit)) - 1) {
        int chunk = PER * t + PER - 1;
        double before = cum;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          if (cum + wl[k] > target) {
            chunk = PER * t + k;
            before = cum;
            break;
          }
          cum += wl[k];
        }
        sh.chunk = chunk;
        sh.before = before;
        sh.target = target;
      }
    } else {
      // Rounding put the target at the very top: the last chunk of positive
      // mass (chunk 0 when there is none), its last token of positive mass.
      const unsigned long long pos = __ballot(lastk >= 0);
      const int L = pos ? 63 - __clzll(static_cast<long long>(pos)) : 0;
      if (t == L) {
        sh.chunk = pos ? PER * t + lastk : 0;
        sh.before = 0.0;
        sh.target = HUGE_VAL;
      }
    }
    if (t == 0) {
      sh.M = M;
      sh.idx = 0x7fffffff;
      sh.lastpos = -1;
    }
  }
  __syncthreads();
  const float M = sh.M;
  const int base = sh.chunk * kRowChunk + t * kPerThread;
  float e[kPerThread];
  if (!worker) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) e[i] = 0.f;
  } else if (VEC && base + kPerThread <= V) {
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
    for (int i = 0; i < kPerThread; ++i) {
      const float x = row[min(base + i, V - 1)];   // clamped: loads issue together
      e[i] = (base + i < V) ? exp2f(x * c2 - M) : 0.f;
    }
  }
  double local = 0.0;
  int lastpos = -1;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    local += static_cast<double>(e[i]);
    if (e[i] > 0.f) lastpos = base + i;
  }
  double pos = sh.before + block_excl_scan_d(local, sh.wsum);
  const double target = sh.target;
  int found = 0x7fffffff;
  if (worker) {
    for (int i = 0; i < kPerThread; ++i) {
      pos += static_cast<double>(e[i]);
      if (pos > target) {
        found = base + i;
        break;
      }
    }
  }
  // The smallest index found and the largest of positive mass: per wave by
  // shuffles, then one shared-memory atomic per wave (one per thread made
  // the threads' atomics on one address serialise: 4 us per row).
  const unsigned fmin = wave_min_u(static_cast<unsigned>(found));
  const unsigned lmax = wave_max_u(static_cast<unsigned>(lastpos + 1));
  if (worker && (t & 63) == 0) {
    if (fmin != 0x7fffffffu) atomicMin(&sh.idx, static_cast<int>(fmin));
    if (lmax != 0u) atomicMax(&sh.lastpos, static_cast<int>(lmax) - 1);
  }
  __syncthreads();
  return (sh.idx != 0x7fffffff) ? sh.idx : sh.lastpos;
}

inline bool row_vec_ok(const float* p, long long ld) {
  return (reinterpret_cast<uintptr_t>(p) % 16 == 0) && (ld % 4 == 0);
}

}  // namespace
}  // namespace ent
