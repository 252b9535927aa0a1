// Top-k and tail-corrected entropy estimates of one logit row (Section 2.1
// of the paper: the top-k entropy approximation and the tail-corrected
// estimator; Section 3.3: the controller acting on the estimate).
//
//   K    = the k most probable tokens of p = softmax(z / T)
//   H~   = entropy of p restricted to K and renormalised
//   mbar = probability mass outside K
//   H^   = H~ + h(mbar) + mbar ln(|V| - k),   h the binary entropy
//
// In the log2-scaled units of the chunk pass (t = z log2(e) / T, row maximum
// M, S = sum over the row of 2^(t - M)):
//   S_K = sum_K 2^(t - M),  W_K = sum_K 2^(t - M) (t - M),
//   H~  = ln 2 (log2 S_K - W_K / S_K),  mbar = (S - S_K) / S.
// Only the multiset of the k largest t matters, so tokens tied at the k-th
// value are interchangeable.
//
// Finding K exactly without a second pass over the row: the chunk pass
// records each chunk thread's largest t (16 logits per thread).  theta1, the
// k-th largest of those maxima, is a lower bound of the row's k-th largest t
// (k distinct tokens reach it).  A token with t > theta1 lies in a thread
// whose maximum exceeds theta1, and fewer than k threads qualify.  Their
// logits are re-read (under 16 k values):
//   * if at least k of those values exceed theta1, the row's k-th largest is
//     the k-th largest of them, and every token at or above it was re-read;
//   * otherwise the row's k-th largest is theta1 itself and K is the values
//     above theta1 plus copies of theta1.
// Both selections are exact radix selects (8-bit digits over the bits in
// which the keys differ, as in the block selection).  The first kEstThreads
// threads of the workgroup do all the arithmetic, in a fixed order, so every
// caller (the per-stage kernel, the fused step) gets the same float.
#pragma once

#include "entropy_dev.h"

namespace ent {
namespace {

constexpr int kEstThreads = 256;
constexpr int kEstWaves = kEstThreads / 64;
constexpr int kEstLds1 = 8192;     // thread maxima staged in LDS (more: read from memory)

struct EstShared {
  unsigned hist[256];
  unsigned red[2 * kEstWaves];
  float fred[3 * kEstWaves];        // three independent block sums
  int ired[kEstWaves];
  float M, S;
  int digit, krem;
};

__device__ __forceinline__ unsigned est_key(float f) {
  const unsigned u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float est_key_value(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Dynamic LDS of the estimator: keys (stage 1 maxima or stage 2 values),
// then the qualifying thread list.
__host__ __device__ inline int est_key_slots(int C, int k) {
  const int n1 = C * kEstChunkThreads;
  const int s1 = n1 <= kEstLds1 ? n1 : 0;
  return s1 > 16 * k ? s1 : 16 * k;
}
__host__ __device__ inline size_t est_lds_bytes(int C, int k) {
  return static_cast<size_t>(est_key_slots(C, k) + k) * 4;
}

// Sum over the first kEstThreads threads (result in every thread).
__device__ __forceinline__ float est_block_sum(float v, EstShared& sh, int slot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum(v);
  if (lane == 0 && wave < kEstWaves) sh.fred[slot * kEstWaves + wave] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int w = 0; w < kEstWaves; ++w) r += sh.fred[slot * kEstWaves + w];
  return r;
}

// k-th largest (1 <= k <= n) of the n keys get(0 .. n-1); n_gt receives the
// number of keys strictly above it.  Every thread of the workgroup calls it.
template <class Get>
__device__ unsigned est_kth_largest(Get get, int n, int k, EstShared& sh, int& n_gt) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const bool worker = t < kEstThreads;
  unsigned kmin = 0xFFFFFFFFu, kmax = 0u;
  if (worker)
    for (int i = t; i < n; i += kEstThreads) {
      const unsigned x = get(i);
      kmin = min(kmin, x);
      kmax = max(kmax, x);
    }
  kmin = wave_min_u(kmin);
  kmax = wave_max_u(kmax);
  if (worker && lane == 0) {
    sh.red[wave] = kmin;
    sh.red[kEstWaves + wave] = kmax;
  }
  if (t == 0) sh.krem = k;
  __syncthreads();
  kmin = sh.red[0];
  kmax = sh.red[kEstWaves];
#pragma unroll
  for (int w = 1; w < kEstWaves; ++w) {
    kmin = min(kmin, sh.red[w]);
    kmax = max(kmax, sh.red[kEstWaves + w]);
  }
  const unsigned diff = kmin ^ kmax;
  unsigned prefix = kmax;
  if (diff) {
    const int top = 31 - __clz(diff);
    unsigned mask = top == 31 ? 0u : ~((2u << top) - 1u);
    prefix = kmax & mask;
    for (int hi = top; hi >= 0; hi -= 8) {
      const int shift = max(hi - 7, 0);
      const int width = hi - shift + 1;
      const unsigned dmask = (1u << width) - 1u;
      if (t < 256) sh.hist[t] = 0u;
      __syncthreads();
      if (worker)
        for (int i = t; i < n; i += kEstThreads) {
          const unsigned x = get(i);
          if ((x & mask) == prefix) atomicAdd(&sh.hist[(x >> shift) & dmask], 1u);
        }
      __syncthreads();
      if (wave == 0) {
        // Bins 4 lane .. 4 lane + 3; suffix sums over lanes find the digit
        // holding the krem-th largest remaining key.
        const unsigned c0 = sh.hist[4 * lane], c1 = sh.hist[4 * lane + 1],
                       c2 = sh.hist[4 * lane + 2], c3 = sh.hist[4 * lane + 3];
        const unsigned cl = c0 + c1 + c2 + c3;
        unsigned suf = cl;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const unsigned nx = __shfl_down(suf, o);
          if (lane + o < 64) suf += nx;
        }
        const unsigned krem = static_cast<unsigned>(sh.krem);
        const unsigned above = suf - cl;
        if (above < krem && suf >= krem) {
          unsigned run = above;
          const unsigned cs[4] = {c0, c1, c2, c3};
          int d = 4 * lane;
          for (int x = 3; x >= 0; --x) {
            if (run + cs[x] >= krem) {
              d = 4 * lane + x;
              break;
            }
            run += cs[x];
          }
          sh.digit = d;
          sh.krem = static_cast<int>(krem - run);
        }
      }
      __syncthreads();
      prefix |= static_cast<unsigned>(sh.digit) << shift;
      mask |= dmask << shift;
    }
  }
  n_gt = k - sh.krem;
  __syncthreads();
  return prefix;
}

// Estimate of row b: ENT_EST_TOPK gives H~, ENT_EST_TAIL gives H^ (k < |V|;
// the caller takes the exact entropy when k >= |V|).  part: the chunk
// triples; tmax: the chunk threads' maxima [B, C, 256]; T: the row's
// temperature (the chunk pass's); lds: est_lds_bytes(C, k) of dynamic LDS.
// Every thread of the workgroup (>= kEstThreads threads) calls it; the
// result is returned in every thread.
__device__ float row_estimate(int est, int k, const float* __restrict__ part,
                              const float* __restrict__ tmax, const float* __restrict__ logits,
                              long long ld, int V, int C, float T, int b, unsigned* lds,
                              EstShared& sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const bool worker = t < kEstThreads;
  const int n1 = C * kEstChunkThreads;
  const float* tm = tmax + static_cast<long long>(b) * n1;
  const float* row = logits + static_cast<long long>(b) * ld;
  unsigned* keys = lds;
  int* qual = reinterpret_cast<int*>(lds + est_key_slots(C, k));

  // Row maximum and mass from the chunk triples (as the exact entropy does).
  if (wave == 0) {
    const float* pr = part + static_cast<long long>(b) * C * 3;
    float mloc = -INFINITY;
    for (int i = lane; i < C; i += 64) mloc = fmaxf(mloc, pr[3 * i]);
    const float MG = wave_max(mloc);
    float s = 0.f;
    for (int i = lane; i < C; i += 64) {
      const float sc = pr[3 * i + 1];
      if (sc > 0.f) s += sc * exp2f(pr[3 * i] - MG);
    }
    s = wave_sum(s);
    if (lane == 0) {
      sh.M = MG;
      sh.S = s;
    }
  }

  // Stage 1: theta1 = k-th largest thread maximum.
  const bool in_lds = n1 <= kEstLds1;
  if (in_lds && worker)
    for (int i = t; i < n1; i += kEstThreads) keys[i] = est_key(tm[i]);
  __syncthreads();
  unsigned th1;
  int unused;
  if (k > n1)
    th1 = est_key(-INFINITY);          // fewer maxima than k: every thread with a value qualifies
  else if (in_lds)
    th1 = est_kth_largest([&](int i) { return keys[i]; }, n1, k, sh, unused);
  else
    th1 = est_kth_largest([&](int i) { return est_key(tm[i]); }, n1, k, sh, unused);

  // Qualifying threads (maximum > theta1), in index order: each worker scans
  // a contiguous run of maxima, then an exclusive scan of the counts.
  const int per = (n1 + kEstThreads - 1) / kEstThreads;
  int cnt = 0;
  if (worker)
    for (int i = t * per; i < min(n1, (t + 1) * per); ++i)
      cnt += (in_lds ? keys[i] : est_key(tm[i])) > th1;
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int nx = __shfl_up(incl, o);
    if (lane >= o) incl += nx;
  }
  if (worker && lane == 63) sh.ired[wave] = incl;
  __syncthreads();
  int before = incl - cnt, nq = 0;
#pragma unroll
  for (int w = 0; w < kEstWaves; ++w) {
    if (w < wave) before += sh.ired[w];
    nq += sh.ired[w];
  }
  nq = min(nq, k);                     // < k by construction
  if (worker)
    for (int i = t * per, o = before; i < min(n1, (t + 1) * per); ++i)
      if ((in_lds ? keys[i] : est_key(tm[i])) > th1 && o < nq) qual[o++] = i;
  __syncthreads();

  // Stage 2: re-read the qualifying threads' logits (the chunk pass's
  // element mapping and scaling), 16 values each.
  const float c2 = __fdiv_rn(kLog2e, T);
  if (worker)
    for (int q = t; q < nq; q += kEstThreads) {
      const int j = qual[q];
      const int base = (j / kEstChunkThreads) * kRowChunk + (j % kEstChunkThreads) * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int pos = base + i * kEstChunkThreads * 4 + kk;
          const float v = pos < V ? row[pos] * c2 : -INFINITY;
          keys[q * 16 + 4 * i + kk] = est_key(v);
        }
    }
  __syncthreads();
  const int n2 = nq * 16;
  int a = 0;
  if (worker)
    for (int i = t; i < n2; i += kEstThreads) a += keys[i] > th1;
  a = static_cast<int>(est_block_sum(static_cast<float>(a), sh, 0) + 0.5f);   // exact below 2^24
  unsigned theta = th1;
  int n_gt = a;
  if (a >= k) theta = est_kth_largest([&](int i) { return keys[i]; }, n2, k, sh, n_gt);

  // Sums over the top-k multiset: values above theta, plus k - n_gt copies of theta.
  const float M = sh.M, S = sh.S;
  float s = 0.f, w = 0.f;
  if (worker)
    for (int i = t; i < n2; i += kEstThreads) {
      const unsigned x = keys[i];
      if (x > theta) {
        const float d = est_key_value(x) - M;
        const float e = __builtin_amdgcn_exp2f(d);
        s += e;
        w += (e > 0.f) ? e * d : 0.f;
      }
    }
  s = est_block_sum(s, sh, 1);
  w = est_block_sum(w, sh, 2);
  {
#pragma clang fp contract(off)
    const float dt = est_key_value(theta) - M;
    const float et = __builtin_amdgcn_exp2f(dt);
    const float nt = static_cast<float>(k - n_gt);
    const float SK = s + nt * et;
    const float WK = w + ((et > 0.f) ? nt * (et * dt) : 0.f);
    const float Ht = (log2f(SK) - WK / SK) * kLn2;
    float H = Ht;
    if (est == ENT_EST_TAIL) {
      float mbar = (S - SK) / S;
      mbar = fminf(fmaxf(mbar, 0.f), 1.f);
      const float hb = (mbar > 0.f && mbar < 1.f) ? -mbar * logf(mbar) - (1.f - mbar) * log1pf(-mbar)
                                                  : 0.f;
      H = Ht + hb + mbar * logf(static_cast<float>(V - k));
    }
    __syncthreads();
    return H;
  }
}

}  // namespace
}  // namespace ent
