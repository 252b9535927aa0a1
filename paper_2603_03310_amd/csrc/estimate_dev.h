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
// Both selections are exact radix selects (11-bit digits over the bits in
// which the keys differ); the second counts only the values above theta1.
// Every thread of the workgroup takes part in the selections, whose results
// do not depend on the workgroup size; the qualifying threads are listed in
// ascending order and the first kEstThreads threads form the sums in a fixed
// order, so every caller (the per-stage kernel, the fused step in either
// form) gets the same float.
#pragma once

#include "entropy_dev.h"

namespace ent {
namespace {

constexpr int kEstThreads = 256;   // threads that form the sums (every caller has them)
constexpr int kEstWaves = kEstThreads / 64;
constexpr int kEstMaxWaves = 16;   // workgroups of up to 1024 threads
constexpr int kEstLds1 = 8192;     // thread maxima staged in LDS (more: read from memory)
constexpr int kEstDigit = 11;      // radix digit bits
constexpr int kEstBins = 1 << kEstDigit;
constexpr int kEstMaxRuns = kMaxChunks * kEstChunkThreads / 64;   // runs of 64 maxima
static_assert(kEstMaxRuns <= kEstBins, "run counts reuse the histogram");

constexpr int kEstRankMax = 64;    // prefix groups this small are finished by counting ranks
static_assert(kEstRankMax <= kEstBins, "candidates reuse the histogram");

struct EstShared {
  alignas(16) unsigned hist[kEstBins];   // radix histogram, then candidates or run offsets
  unsigned red[2 * kEstMaxWaves];
  float fred[2 * kEstWaves];
  int ired[kEstMaxWaves];
  float M, S;
  int digit, krem, nq, ncand, rgt;
  unsigned rv;
};

__device__ __forceinline__ unsigned est_key(float f) {
  const unsigned u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float est_key_value(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Dynamic LDS of the estimator: keys (stage 1 maxima or stage 2 values,
// 16-byte aligned), then the qualifying thread list.
__host__ __device__ inline int est_key_slots(int C, int k) {
  const int n1 = C * kEstChunkThreads;
  const int s1 = n1 <= kEstLds1 ? n1 : 0;
  return s1 > 16 * k ? s1 : 16 * k;
}
__host__ __device__ inline size_t est_lds_bytes(int C, int k) {
  return static_cast<size_t>(est_key_slots(C, k) + k) * 4;
}
// Offset (in 4-byte words, a multiple of 4) of the estimator's area after
// `words` words of other dynamic LDS.
__host__ __device__ inline int est_lds_offset(int words) { return (words + 3) & ~3; }

// Key sources for the selections, four keys per read.
struct EstLdsKeys {
  const unsigned* p;
  __device__ __forceinline__ uint4 load4(int i4) const { return reinterpret_cast<const uint4*>(p)[i4]; }
  __device__ __forceinline__ unsigned load(int i) const { return p[i]; }
};
struct EstMaxKeys {   // thread maxima read from memory
  const float* p;
  __device__ __forceinline__ uint4 load4(int i4) const {
    const float4 v = reinterpret_cast<const float4*>(p)[i4];
    return make_uint4(est_key(v.x), est_key(v.y), est_key(v.z), est_key(v.w));
  }
  __device__ __forceinline__ unsigned load(int i) const { return est_key(p[i]); }
};

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

// Integer sum over the whole workgroup (result in every thread).
__device__ __forceinline__ int est_block_count(int v, EstShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) sh.ired[wave] = v;
  __syncthreads();
  int r = 0;
  for (int w = 0; w < nw; ++w) r += sh.ired[w];
  __syncthreads();
  return r;
}

// One histogram update per active lane.  Lanes whose bin equals the first
// active lane's bin add together (one atomic for all of them): equal keys
// (ties) would otherwise serialise on one LDS address.
__device__ __forceinline__ void est_hist_add(unsigned* hist, bool act, unsigned bin) {
  const unsigned long long am = __ballot(act);
  if (am == 0ull) return;
  const int leader = __ffsll(static_cast<long long>(am)) - 1;
  const unsigned lb = __builtin_amdgcn_readlane(bin, leader);
  const bool same = act && bin == lb;
  const unsigned long long sm = __ballot(same);
  if ((threadIdx.x & 63) == leader) atomicAdd(&hist[lb], static_cast<unsigned>(__popcll(sm)));
  if (act && !same) atomicAdd(&hist[bin], 1u);
}

// k-th largest among the keys >= lo of src (4 n4 keys); requires
// 1 <= k <= their number.  n_gt receives how many of them lie strictly
// above it.  Radix select over the bits in which those keys differ,
// kEstDigit bits per pass from the top; once the keys that share the
// selected prefix are few (at most kEstRankMax) they are gathered into LDS
// and the answer is found among them by counting ranks, instead of further
// passes over every key.  Every thread of the workgroup calls it and takes
// part (the result does not depend on the workgroup size).  Ties: callers
// whose keys often repeat aggregate equal bins per wave.
template <class Src, bool kTies = false>
__device__ __forceinline__ unsigned est_kth_largest(const Src& src, int n4, unsigned lo, int k,
                                                    EstShared& sh, int& n_gt) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int NT = blockDim.x, nw = NT >> 6;
  unsigned kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll 4
  for (int i = t; i < n4; i += NT) {
    const uint4 x = src.load4(i);
    const unsigned e[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (e[j] >= lo) {
        kmin = min(kmin, e[j]);
        kmax = max(kmax, e[j]);
      }
  }
  kmin = wave_min_u(kmin);
  kmax = wave_max_u(kmax);
  if (lane == 0) {
    sh.red[wave] = kmin;
    sh.red[kEstMaxWaves + wave] = kmax;
  }
  if (t == 0) sh.krem = k;
  __syncthreads();
  kmin = sh.red[0];
  kmax = sh.red[kEstMaxWaves];
  for (int w = 1; w < nw; ++w) {
    kmin = min(kmin, sh.red[w]);
    kmax = max(kmax, sh.red[kEstMaxWaves + w]);
  }
  const unsigned diff = kmin ^ kmax;
  unsigned prefix = kmax;
  if (diff) {
    const int top = 31 - __clz(diff);
    unsigned mask = top == 31 ? 0u : ~((2u << top) - 1u);
    prefix = kmax & mask;
    for (int hi = top; hi >= 0; hi -= kEstDigit) {
      const int shift = max(hi - (kEstDigit - 1), 0);
      const int width = hi - shift + 1;
      const unsigned dmask = (1u << width) - 1u;
      for (int i = t; i < kEstBins; i += NT) sh.hist[i] = 0u;
      __syncthreads();
      // (The ballots of the tie-aware form are convergent: that loop cannot
      // be unrolled over its run-time trip count.)
      constexpr int kUnroll = kTies ? 1 : 4;
#pragma unroll kUnroll
      for (int i = t; i < n4; i += NT) {
        const uint4 x = src.load4(i);
        const unsigned e[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool act = e[j] >= lo && (e[j] & mask) == prefix;
          if (kTies) est_hist_add(sh.hist, act, (e[j] >> shift) & dmask);
          else if (act) atomicAdd(&sh.hist[(e[j] >> shift) & dmask], 1u);
        }
      }
      __syncthreads();
      if (wave == 0) {
        // Lane l holds bins BPL l .. BPL l + BPL - 1; suffix sums over lanes
        // find the digit holding the krem-th largest remaining key.
        constexpr int BPL = kEstBins / 64;
        unsigned c[BPL];
        unsigned cl = 0;
#pragma unroll
        for (int j = 0; j < BPL; j += 4) {
          const uint4 h = *reinterpret_cast<const uint4*>(&sh.hist[BPL * lane + j]);
          c[j] = h.x;
          c[j + 1] = h.y;
          c[j + 2] = h.z;
          c[j + 3] = h.w;
          cl += h.x + h.y + h.z + h.w;
        }
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
          int d = BPL * lane;
#pragma unroll
          for (int j = BPL - 1; j >= 0; --j) {
            if (run + c[j] >= krem) {
              d = BPL * lane + j;
              break;
            }
            run += c[j];
          }
          sh.digit = d;
          sh.krem = static_cast<int>(krem - run);
        }
      }
      __syncthreads();
      prefix |= static_cast<unsigned>(sh.digit) << shift;
      mask |= dmask << shift;
      const int c = static_cast<int>(sh.hist[sh.digit]);   // keys sharing the new prefix
      const int krem = sh.krem;
      __syncthreads();                       // every thread has read both before reuse
      if (shift > 0 && c <= kEstRankMax) {
        // The krem-th largest of those c keys: gather them (any order),
        // then each counts the keys above it and at or above it.
        if (t == 0) sh.ncand = 0;
        __syncthreads();
        unsigned* cand = sh.hist;
#pragma unroll 4
        for (int i = t; i < n4; i += NT) {
          const uint4 x = src.load4(i);
          const unsigned e[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (e[j] >= lo && (e[j] & mask) == prefix) cand[atomicAdd(&sh.ncand, 1)] = e[j];
        }
        __syncthreads();
        for (int i = t; i < c; i += NT) {
          const unsigned v = cand[i];
          int gt = 0, ge = 0;
          for (int j = 0; j < c; ++j) {
            const unsigned x = cand[j];
            gt += x > v;
            ge += x >= v;
          }
          if (gt < krem && ge >= krem) {     // equal keys write the same values
            sh.rv = v;
            sh.rgt = gt;
          }
        }
        __syncthreads();
        n_gt = k - krem + sh.rgt;
        const unsigned r = sh.rv;
        __syncthreads();
        return r;
      }
    }
  }
  n_gt = k - sh.krem;
  __syncthreads();
  return prefix;
}

// Qualifying threads (maximum > th1) in ascending index order, into qual
// (at most cap entries); returns their number.  Wave ballots count each run
// of 64 maxima, one wave scans the run counts, and every qualifying index is
// written at its run's offset plus its rank within the run.
template <class Src>
__device__ __forceinline__ int est_qualifying(const Src& src, int n1, unsigned th1, int* qual,
                                              int cap, EstShared& sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, nw = blockDim.x >> 6;
  const int nrun = n1 / 64;
  for (int r = wave; r < nrun; r += nw) {
    const unsigned long long bal = __ballot(src.load(64 * r + lane) > th1);
    if (lane == 0) sh.hist[r] = static_cast<unsigned>(__popcll(bal));
  }
  __syncthreads();
  if (wave == 0) {
    const int per = (nrun + 63) / 64;
    unsigned loc = 0;
    for (int i = 0; i < per; ++i) {
      const int r = lane * per + i;
      if (r < nrun) loc += sh.hist[r];
    }
    unsigned incl = loc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned nx = __shfl_up(incl, o);
      if (lane >= o) incl += nx;
    }
    unsigned run = incl - loc;
    for (int i = 0; i < per; ++i) {
      const int r = lane * per + i;
      if (r < nrun) {
        const unsigned c = sh.hist[r];
        sh.hist[r] = run;
        run += c;
      }
    }
    if (lane == 63) sh.nq = static_cast<int>(incl);
  }
  __syncthreads();
  for (int r = wave; r < nrun; r += nw) {
    const int j = 64 * r + lane;
    const bool f = src.load(j) > th1;
    const unsigned long long bal = __ballot(f);
    const int o = static_cast<int>(sh.hist[r]) + __popcll(bal & ((1ull << lane) - 1ull));
    if (f && o < cap) qual[o] = j;
  }
  const int nq = min(sh.nq, cap);
  __syncthreads();
  return nq;
}

// Estimate of row b: ENT_EST_TOPK gives H~, ENT_EST_TAIL gives H^ (k < |V|;
// the caller takes the exact entropy when k >= |V|).  part: the chunk
// triples; tmax: the chunk threads' maxima [B, C, 256]; T: the row's
// temperature (the chunk pass's); lds: est_lds_bytes(C, k) of dynamic LDS,
// 16-byte aligned.  Every thread of the workgroup (a multiple of 64, from
// kEstThreads to 1024) calls it; the result, in every thread, does not
// depend on the workgroup size.
__device__ __forceinline__ float row_estimate(int est, int k, const float* __restrict__ part,
                                              const float* __restrict__ tmax,
                                              const float* __restrict__ logits, long long ld,
                                              int V, int C, float T, int b, unsigned* lds,
                                              EstShared& sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int NT = blockDim.x;
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

  // Stage 1: theta1 = k-th largest thread maximum (staged in LDS when the
  // maxima fit, all of a thread's loads issued before its stores).
  const bool in_lds = n1 <= kEstLds1;
  if (in_lds) {
    constexpr int P4 = kEstLds1 / 4 / kEstThreads;   // float4 per thread, at most
    float4 v[P4];
#pragma unroll
    for (int u = 0; u < P4; ++u) {
      const int i4 = t + u * NT;
      v[u] = i4 < n1 / 4 ? reinterpret_cast<const float4*>(tm)[i4] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < P4; ++u) {
      const int i4 = t + u * NT;
      if (i4 < n1 / 4)
        reinterpret_cast<uint4*>(keys)[i4] =
            make_uint4(est_key(v[u].x), est_key(v[u].y), est_key(v[u].z), est_key(v[u].w));
    }
  }
  __syncthreads();
  unsigned th1;
  int unused, nq;
  if (k > n1) {
    th1 = est_key(-INFINITY);        // fewer maxima than k: every thread with a value qualifies
  } else if (in_lds) {
    th1 = est_kth_largest(EstLdsKeys{keys}, n1 / 4, 0u, k, sh, unused);
  } else {
    th1 = est_kth_largest(EstMaxKeys{tm}, n1 / 4, 0u, k, sh, unused);
  }
  if (in_lds) nq = est_qualifying(EstLdsKeys{keys}, n1, th1, qual, k, sh);
  else nq = est_qualifying(EstMaxKeys{tm}, n1, th1, qual, k, sh);

  // Stage 2: re-read the qualifying threads' logits (the chunk pass's
  // element mapping and scaling), 16 values each.
  const float c2 = __fdiv_rn(kLog2e, T);
  for (int q = t; q < nq; q += NT) {
    const int j = qual[q];
    const int base = (j / kEstChunkThreads) * kRowChunk + (j % kEstChunkThreads) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int pos = base + i * kEstChunkThreads * 4 + kk;
        const float x = row[min(pos, V - 1)];   // clamped: loads issue together
        const float v = pos < V ? x * c2 : -INFINITY;
        keys[q * 16 + 4 * i + kk] = est_key(v);
      }
  }
  __syncthreads();
  const int n2 = nq * 16;
  int a = 0;
  for (int i = t; i < n2 / 4; i += NT) {
    const uint4 x = reinterpret_cast<const uint4*>(keys)[i];
    a += (x.x > th1) + (x.y > th1) + (x.z > th1) + (x.w > th1);
  }
  a = est_block_count(a, sh);
  unsigned theta = th1;
  int n_gt = a;
  if (a >= k) theta = est_kth_largest(EstLdsKeys{keys}, n2 / 4, th1 + 1u, k, sh, n_gt);

  // Sums over the top-k multiset: values above theta, plus k - n_gt copies
  // of theta, formed by the first kEstThreads threads in a fixed order.
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
  s = est_block_sum(s, sh, 0);
  w = est_block_sum(w, sh, 1);
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
