// Decode attention over the kept blocks only (Section 3.2 of the paper:
// attention computation is restricted to the kept block set).
//
// Work decomposition (stream-K).  A unit is one kept block of one sequence
// for one KV head (its G query heads together).  Units are laid end to end,
// sequence-major, then KV head, then kept-list order; the (sequence, KV head)
// runs are "segments".  Every wave of the persistent grid takes one
// contiguous range of units (of equal length, or for bf16 weighted by the
// XCD its workgroup runs on), so the waves finish together and the pipeline
// never drains between work items.  A wave walks its range with a
// 64-unit metadata window (kept id and physical block per lane, gathered in
// parallel) and a one-block-ahead register prefetch of the K and V tiles.
// Where its range covers a whole segment it writes the output directly;
// where it covers part of one it writes an unnormalised partial
// (max, sum, output) to slot (range + segment), which is unique because both
// partitions are ordered intervals.  The range in which a cut segment begins
// also writes a record (segment, last range holding it, total units), so a
// second kernel merges the partials of every cut segment from that record
// alone, without rebuilding the plan.  The kept counts stay on the device.
//
// bf16 path (MFMA, gfx950).  Per kept block of 16 tokens:
//   S^T[16 tok x 16 heads] = K[16 x d] . Q^T[d x 16]   v_mfma_f32_16x16x32_bf16,
//     A = K rows from the token-major K tile (16 B per lane per step), the
//         tile loaded 1 KB whole per instruction (non-temporal) and passed
//         through the wave's LDS rows into this layout,
//     B = the G query heads (zero-padded to 16 columns), held in registers;
//   online softmax per head column (log2 domain, fp32); the cross-lane max is
//   taken only when some score exceeds a head's running max;
//   O^T[d x 16] += V^T[d x 16 tok] . P^T[16 tok x 16]   v_mfma_f32_16x16x16_bf16,
//     A = rows of the dim-major V tile (8 B per lane per 16-dim tile, each
//         load instruction a whole 512 B span; non-temporal),
//     B = P^T taken straight from the S^T accumulator registers, split into
//         a bf16 high part and a bf16 remainder (two MFMAs), so P keeps
//         about 16 bits.
// fp32 path (VALU): the same decomposition with scalar dot products.

#include "blocks_dev.h"
#include "entropy_dev.h"

#include <math.h>

#include <algorithm>

namespace ent {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kWindow = 64;                  // units of metadata per window

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4_t __attribute__((__vector_size__(4 * sizeof(short))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const int* tables;
  const int* ctx_lens;
  const int* kept;
  const int* kept_phys;   // nullable: encoded physical blocks of the kept lists
  const int* n_kept;
  float* out;
  float* lse;
  float* part_acc;    // [W + S, G, D]
  float* part_ml;     // [W + S, G, 2]
  int4* rec;          // [R] cut-segment record of each range: (segment or -1, last range, U, 0)
  unsigned* flags;
  int B, Hkv, G, MAXB, P;
  int W;              // waves of the decode grid
  int R;              // ranges that write partials (workgroups for bf16, waves for fp32)
  int xw;             // 1: ranges weighted by XCD (bf16, wv_begin / wg_begin), 0: equal wave ranges
  int nsl;            // merge workgroups per segment
  float scale_log2;   // softmax scale times log2(e)
};

// Plan in LDS: s_pref[b] = first unit of sequence b (s_pref[B] = total),
// s_nk[b] = kept blocks of b (0 when its context length is invalid),
// s_N[b] = context length.
__device__ void build_plan(const DecodeArgs& a, int* s_pref, int* s_nk, int* s_N, int* s_red) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = (a.B + kThreads - 1) / kThreads;
  int loc = 0;
  for (int i = 0; i < per; ++i) {
    const int b = t * per + i;
    if (b < a.B) {
      const int N = a.ctx_lens[b];
      const bool ok = N >= 0 && N <= a.MAXB * kBlock;
      const int nk = ok ? min(max(a.n_kept[b], 0), a.MAXB) : 0;
      s_nk[b] = nk;
      s_N[b] = ok ? N : 0;
      loc += nk * a.Hkv;
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
    if (b < a.B) {
      s_pref[b] = run;
      run += s_nk[b] * a.Hkv;
    }
  }
  if (t == kThreads - 1) s_pref[a.B] = run;
  __syncthreads();
}

// Sequences with nothing kept (or an invalid context length) get out = 0 and
// lse = -inf, written by workgroup b % gridDim.x.  s_nk is in LDS (uniform).
template <int D>
__device__ __forceinline__ void zero_empty(const DecodeArgs& a, const int* s_nk) {
  const int Hq = a.Hkv * a.G;
  for (int b = blockIdx.x; b < a.B; b += gridDim.x) {
    if (s_nk[b] != 0) continue;
    float* o = a.out + static_cast<long long>(b) * Hq * D;
    for (int e = threadIdx.x; e < Hq * D; e += blockDim.x) o[e] = 0.f;
    if (a.lse)
      for (int h = threadIdx.x; h < Hq; h += blockDim.x) a.lse[static_cast<long long>(b) * Hq + h] = -INFINITY;
  }
}

__device__ __forceinline__ int range_begin(int w, int U, int W) {
  return static_cast<int>(static_cast<long long>(w) * U / W);
}
// The wave whose range holds unit x (U > 0); the product in 64 bits, since
// (x + 1) W passes 2^31 once the kept units do 2^31 / W.
__device__ __forceinline__ int wave_of(int x, int U, int W) {
  return static_cast<int>((static_cast<long long>(x + 1) * W - 1) / U);
}

// The bf16 decode's ranges, weighted by XCD: workgroups are dealt to the
// eight XCDs in turn (workgroup x on XCD x mod 8), and waves on the odd XCDs
// were measured streaming their units 10-15% slower than those on the even
// ones (per-wave timestamps, the same in every range); an odd workgroup
// therefore takes kOddW / kEvenW of an even one's units, its four waves
// alike (10:9 measured best against 20:19, 7:6 and 5:4).  Each workgroup's
// range is the union of its waves' ranges.
constexpr int kEvenW = 10, kOddW = 9;
__device__ __forceinline__ long long wg_weight(int x) {
  return static_cast<long long>(x >> 1) * (kEvenW + kOddW) + ((x & 1) ? kEvenW : 0);
}
__device__ __forceinline__ int wg_begin(int x, int U, int R) {
  return static_cast<int>(wg_weight(x) * U / wg_weight(R));
}
__device__ __forceinline__ int wv_begin(int w, int U, int R) {
  const int x = w / kWaves, i = w - x * kWaves;
  const long long c = kWaves * wg_weight(x) + static_cast<long long>(i) * ((x & 1) ? kOddW : kEvenW);
  return static_cast<int>(c * U / (kWaves * wg_weight(R)));
}
// The workgroup whose range holds unit u (U > 0).
__device__ __forceinline__ int wg_of(int u, int U, int R) {
  int x = static_cast<int>(static_cast<long long>(u) * R / U);
  x = x < 0 ? 0 : (x >= R ? R - 1 : x);
  while (x > 0 && wg_begin(x, U, R) > u) --x;
  while (x + 1 < R && wg_begin(x + 1, U, R) <= u) ++x;
  return x;
}

// Sequence holding unit x: the largest b with s_pref[b] <= x.
__device__ __forceinline__ int seq_of(int x, const int* s_pref, int B) {
  int lo = 0, hi = B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_pref[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// Metadata of one unit, gathered by one lane.
struct UnitMeta {
  int seg;   // b * H_kv + g, or -1 past the end of the range
  int p;     // physical block, -1 to skip
  int nv;    // valid tokens of the block
};

__device__ __forceinline__ UnitMeta unit_meta(const DecodeArgs& a, int x, int u1,
                                              const int* s_pref, const int* s_nk, const int* s_N) {
  UnitMeta m{-1, -1, 0};
  if (x >= u1) return m;
  const int b = seq_of(x, s_pref, a.B);
  const int nk = s_nk[b];
  const int r = static_cast<int>(x - s_pref[b]);
  const int g = r / nk, j = r % nk;
  m.seg = b * a.Hkv + g;
  const int N = s_N[b];
  const int nb = (N + kBlock - 1) / kBlock;
  const long long row = static_cast<long long>(b) * a.MAXB;
  if (a.kept_phys) {
    // The selection's encoding: physical block, bit 30 = the sequence's last block.
    const int v = a.kept_phys[row + j];
    if (v >= 0) {
      m.p = v & ((1 << 30) - 1);
      m.nv = (v >> 30) ? N - kBlock * (nb - 1) : kBlock;
    } else if (g == 0) {
      raise_flag(a.flags, ENT_DEV_BAD_TABLE);
    }
    return m;
  }
  const int kid = a.kept[row + j];
  if (kid >= 0 && kid < nb) {
    const int p = a.tables[row + kid];
    if (p >= 0 && p < a.P) {
      m.p = p;
      m.nv = (kid == nb - 1) ? N - kBlock * (nb - 1) : kBlock;
    } else if (g == 0) {
      raise_flag(a.flags, ENT_DEV_BAD_TABLE);
    }
  } else if (g == 0) {
    raise_flag(a.flags, ENT_DEV_BAD_TABLE);
  }
  return m;
}

// K and V tiles are read once per step: non-temporal loads (the nt bit)
// measured 8% faster on the decode than plain loads (the queries, read by
// every wave of a segment, keep plain loads: 1 us better).  The exact
// scoring mode's whole-row K loads and the block-summary gather (both staged
// through LDS) use the bit too; it made loads straight into the MFMA layout
// slower, and the logit pass no faster, so those keep plain loads.
// Whole-row K loads staged through LDS measured 1-2% faster than loads
// straight into the MFMA layout.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x8_t load_bf16x8(const uint16_t* p) {
  const uint4 x = *reinterpret_cast<const uint4*>(p);
  return __builtin_bit_cast(bf16x8_t, x);
}
__device__ __forceinline__ bf16x8_t load_bf16x8_nt(const uint16_t* p) {
  const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return __builtin_bit_cast(bf16x8_t, x);
}
__device__ __forceinline__ s16x4_t load_s16x4(const uint16_t* p) {
  const u32x2_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  return __builtin_bit_cast(s16x4_t, x);
}

template <int D>
__global__ __launch_bounds__(kThreads, 3) void decode_bf16_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;      // QK k-steps (32 dims each)
  constexpr int MT = D / 16;      // PV output tiles (16 dims each)
  extern __shared__ __attribute__((aligned(16))) int s_mem[];
  __shared__ int s_red[kWaves];
  __shared__ int s_cseg[2 * kWaves];
  __shared__ int4 s_gd[2 * kWaves];         // merge groups: slots, segment, its record
  __shared__ int s_ng;
  // Each wave's K tile in the MFMA layout's source form, rows padded by 16 B.
  __shared__ __attribute__((aligned(16))) uint16_t s_kst[kWaves * kBlock * (D + 8)];
  // Dynamic LDS: cut partials first (16-byte aligned), then the plan.
  float* s_cacc = reinterpret_cast<float*>(s_mem);
  float* s_cml = s_cacc + 2 * kWaves * a.G * D;
  int* s_pref = reinterpret_cast<int*>(s_cml + 2 * kWaves * kMaxGroup * 2);
  int* s_nk = s_pref + a.B + 1;
  int* s_N = s_nk + a.B;
  build_plan(a, s_pref, s_nk, s_N, s_red);
  const int U = s_pref[a.B];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int w = blockIdx.x * kWaves + wave;
  zero_empty<D>(a, s_nk);
  if (U == 0) {
    if (threadIdx.x == 0) a.rec[blockIdx.x] = make_int4(-1, 0, 0, 0);
    return;
  }
  const int G = a.G;
  // Cut partials of this workgroup's waves, merged in LDS at the end:
  // slot 2 i (wave i's first segment, begun before its range) and 2 i + 1
  // (its last, continuing after it): G x D sums and (max, sum) per head.
  if (lane < 2) s_cseg[2 * wave + lane] = -1;
  const int u0 = wv_begin(w, U, a.R), u1 = wv_begin(w + 1, U, a.R);
  const int r16 = lane & 15, gq = lane >> 4;
  const int Hq = a.Hkv * G;
  const bool head_ok = r16 < G;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  const uint16_t* kc = static_cast<const uint16_t*>(a.kc);
  const uint16_t* vc = static_cast<const uint16_t*>(a.vc);

  int ubase = u0;
  UnitMeta win = unit_meta(a, ubase + lane, u1, s_pref, s_nk, s_N);
  const bool busy = u0 < u1;

  bf16x8_t kcur[KS], knxt[KS];
  s16x4_t vcur[MT], vnxt[MT];
  auto load_tiles = [&](int i, bf16x8_t (&kr)[KS], s16x4_t (&vr)[MT]) {
    const int seg = __shfl(win.seg, i);
    const int p = max(__shfl(win.p, i), 0);
    const int g = max(seg, 0) % a.Hkv;
    const long long tile = (static_cast<long long>(p) * a.Hkv + g) * kBlock * D;
    // K: load ks covers the tile's bytes [ks, ks + 1) * 4 KB / KS whole (lane
    // l its 16 bytes l), staged through LDS into the MFMA layout before use.
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kr[ks] = load_bf16x8_nt(kc + tile + ks * (kBlock * D / KS) + lane * 8);
#pragma unroll
    for (int m = 0; m < MT; ++m) vr[m] = load_s16x4(vc + tile + (16 * m + r16) * kBlock + 4 * gq);
  };
  if (busy) load_tiles(0, kcur, vcur);

  int cur_seg = -1;
  bf16x8_t qreg[KS];
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t oacc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) oacc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // The first segment's queries load together with the first tiles.
  if (busy) {
    cur_seg = __shfl(win.seg, 0);
    const int b = cur_seg / a.Hkv, g = cur_seg % a.Hkv;
    const long long qh = static_cast<long long>(b) * Hq + g * G + r16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (head_ok) qreg[ks] = load_bf16x8(q + qh * D + ks * 32 + gq * 8);
      else qreg[ks] = __builtin_bit_cast(bf16x8_t, make_uint4(0u, 0u, 0u, 0u));
    }
  }

  auto flush = [&]() {
    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    const int b = cur_seg / a.Hkv, g = cur_seg % a.Hkv;
    const int seg_start = s_pref[b] + g * s_nk[b];
    const int seg_end = seg_start + s_nk[b];
    if (!head_ok) return;
    if (seg_start >= u0 && seg_end <= u1) {
      const long long oh = static_cast<long long>(b) * Hq + g * G + r16;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const f32x4_t o = oacc[m] * inv;
        *reinterpret_cast<float4*>(a.out + oh * D + 16 * m + 4 * gq) = make_float4(o[0], o[1], o[2], o[3]);
      }
      if (gq == 0 && a.lse) a.lse[oh] = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    } else {
      // Cut by this wave's range: keep the partial for the workgroup merge.
      const int cs = 2 * wave + (seg_start < u0 ? 0 : 1);
      if (lane == 0) s_cseg[cs] = cur_seg;
      float* acc = s_cacc + (static_cast<long long>(cs) * G + r16) * D;
#pragma unroll
      for (int m = 0; m < MT; ++m)
        *reinterpret_cast<float4*>(acc + 16 * m + 4 * gq) =
            make_float4(oacc[m][0], oacc[m][1], oacc[m][2], oacc[m][3]);
      if (gq == 0) {
        s_cml[(cs * kMaxGroup + r16) * 2 + 0] = m_run;
        s_cml[(cs * kMaxGroup + r16) * 2 + 1] = l_tot;
      }
    }
  };

  // One unit: compute on the tiles in (kc, vc) while the next unit's tiles
  // stream into (kn, vn); the loop below alternates the two buffers.
  auto unit = [&](int u, bf16x8_t (&kc)[KS], s16x4_t (&vc)[MT], bf16x8_t (&kn)[KS],
                  s16x4_t (&vn)[MT]) {
    int i = static_cast<int>(u - ubase);
    if (i == kWindow) {
      ubase = u;
      i = 0;
      win = unit_meta(a, ubase + lane, u1, s_pref, s_nk, s_N);
      load_tiles(0, kc, vc);
    }
    const int seg = __shfl(win.seg, i);
    if (seg != cur_seg) {
      if (cur_seg >= 0) flush();
      cur_seg = seg;
      const int b = seg / a.Hkv, g = seg % a.Hkv;
      const long long qh = static_cast<long long>(b) * Hq + g * G + r16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (head_ok) qreg[ks] = load_bf16x8(q + qh * D + ks * 32 + gq * 8);
        else qreg[ks] = __builtin_bit_cast(bf16x8_t, make_uint4(0u, 0u, 0u, 0u));
      }
      m_run = -INFINITY;
      l_run = 0.f;
#pragma unroll
      for (int m = 0; m < MT; ++m) oacc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    // The next unit's tiles, issued unconditionally so that the wait below
    // covers only the current unit's loads; past the end of the window or of
    // the range the current tiles are re-read (cache hits) and discarded.
    load_tiles((i + 1 < kWindow && u + 1 < u1) ? i + 1 : i, kn, vn);
    const int p = __shfl(win.p, i);
    const int nv = __shfl(win.nv, i);
    if (p >= 0) {
      // The K tile through the wave's LDS rows: written as loaded (whole
      // rows per load), read back with lane (r16, gq) holding row r16, MFMA
      // k-slot (gq, e) of step ks = dim 32 ks + 8 gq + e (the queries' slots
      // too).  The rows are the wave's own, so wave-level barriers order the
      // exchange (and the previous unit's reads before this unit's writes).
      uint16_t* st = s_kst + wave * kBlock * (D + 8);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int e0 = ks * (kBlock * D / KS) + lane * 8;
        *reinterpret_cast<bf16x8_t*>(st + (e0 / D) * (D + 8) + (e0 % D)) = kc[ks];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      bf16x8_t kmf[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kmf[ks] = *reinterpret_cast<const bf16x8_t*>(st + r16 * (D + 8) + ks * 32 + gq * 8);
      f32x4_t sacc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kmf[ks], qreg[ks], sacc, 0, 0, 0);
      float sc[4];
      bool up = false;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sc[e] = (4 * gq + e < nv) ? sacc[e] * a.scale_log2 : -INFINITY;
        up |= sc[e] > m_run;
      }
      // The running max moves only when some score exceeds it.
      if (__any(up)) {
        float mloc = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        const float m_new = fmaxf(m_run, mloc);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int m = 0; m < MT; ++m) oacc[m] *= alpha;
        m_run = m_new;
      }
      // Arguments are <= 0; the hardware exp2 flushes results below 2^-126,
      // which are negligible next to the running maximum's weight of 1.
      bf16x2_t ph[2], pl[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const f32x2_t pe = {__builtin_amdgcn_exp2f(sc[2 * k] - m_run),
                            __builtin_amdgcn_exp2f(sc[2 * k + 1] - m_run)};
        l_run += pe.x + pe.y;
        // P = high bf16 part + bf16 remainder (both rounded to nearest).
        ph[k] = __builtin_convertvector(pe, bf16x2_t);
        pl[k] = __builtin_convertvector(pe - __builtin_convertvector(ph[k], f32x2_t), bf16x2_t);
      }
      const s16x4_t phi = __builtin_bit_cast(s16x4_t, make_uint2(__builtin_bit_cast(uint32_t, ph[0]),
                                                                 __builtin_bit_cast(uint32_t, ph[1])));
      const s16x4_t plo = __builtin_bit_cast(s16x4_t, make_uint2(__builtin_bit_cast(uint32_t, pl[0]),
                                                                 __builtin_bit_cast(uint32_t, pl[1])));
      if (nv < kBlock) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * gq + e >= nv) vc[m][e] = 0;
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        oacc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vc[m], phi, oacc[m], 0, 0, 0);
        oacc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vc[m], plo, oacc[m], 0, 0, 0);
      }
    }
  };
  for (int u = u0; u < u1;) {
    unit(u, kcur, vcur, knxt, vnxt);
    if (++u >= u1) break;
    unit(u, knxt, vnxt, kcur, vcur);
    ++u;
  }
  if (busy) flush();

  // Workgroup merge: consecutive slots of one segment (in unit order) are one
  // group; a group whose segment lies inside the workgroup's range is final,
  // else it becomes the workgroup's partial of that segment (slot wg + seg).
  // First, per (slot, head), the slot's weight 2^(m - M) in its group and the
  // group's (M, L), all slots' loads issued at once; then every output is one
  // weighted sum over its group's slots, in slot order, four consecutive
  // outputs per thread (16-byte LDS reads and stores: with one float each the
  // stores, issued while the other workgroups' loads fill the CU's memory
  // pipeline, made this loop the longest part of a workgroup's end).
  constexpr int kSlots = 2 * kWaves;
  static_assert(kSlots * kMaxGroup + kSlots <= kThreads, "one thread per (slot, head), then per slot");
  static_assert(3 * kSlots * kMaxGroup * sizeof(float) <= sizeof(s_kst), "merge weights in the K rows");
  // The K staging rows are dead once every wave has left its loop.
  float* s_wf = reinterpret_cast<float*>(s_kst);
  float* s_wm = s_wf + kSlots * kMaxGroup;
  float* s_wl = s_wm + kSlots * kMaxGroup;
  __syncthreads();
  if (threadIdx.x < kSlots * kMaxGroup) {
    const int k = threadIdx.x / kMaxGroup, r = threadIdx.x % kMaxGroup;
    const int seg = s_cseg[k];
    float f = 0.f, M = -INFINITY, L = 0.f;
    if (seg >= 0 && r < G) {
#pragma unroll
      for (int kk = 0; kk < kSlots; ++kk)
        if (s_cseg[kk] == seg && s_cml[(kk * kMaxGroup + r) * 2 + 1] > 0.f)
          M = fmaxf(M, s_cml[(kk * kMaxGroup + r) * 2]);
#pragma unroll
      for (int kk = 0; kk < kSlots; ++kk) {
        const float l = s_cml[(kk * kMaxGroup + r) * 2 + 1];
        if (s_cseg[kk] != seg || !(l > 0.f)) continue;
        const float fk = exp2f(s_cml[(kk * kMaxGroup + r) * 2] - M);
        L += l * fk;
        if (kk == k) f = fk;
      }
    }
    s_wf[threadIdx.x] = f;
    s_wm[threadIdx.x] = M;
    s_wl[threadIdx.x] = L;
  } else if (threadIdx.x < kSlots * kMaxGroup + kSlots) {
    // Meanwhile, one thread per slot: a slot heads a group when it holds a
    // segment other than that of the nearest earlier slot holding one; the
    // group runs to the next slot holding another segment (the empty slots
    // between weigh 0).  The heads, in slot order, get the group's slots,
    // whether the segment lies inside this workgroup's range, and the record
    // of a cut segment that begins in it.
    const int k = threadIdx.x - kSlots * kMaxGroup;
    int cs[kSlots];
#pragma unroll
    for (int kk = 0; kk < kSlots; ++kk) cs[kk] = s_cseg[kk];
    bool hd[kSlots];
    int prev = -1;
#pragma unroll
    for (int kk = 0; kk < kSlots; ++kk) {
      hd[kk] = cs[kk] >= 0 && cs[kk] != prev;
      if (cs[kk] >= 0) prev = cs[kk];
    }
    int seg = -1, rank = 0, ng = 0;
    bool head = false;
#pragma unroll
    for (int kk = 0; kk < kSlots; ++kk) {
      if (kk == k) {
        seg = cs[kk];
        head = hd[kk];
      }
      if (kk < k && hd[kk]) ++rank;
      if (hd[kk]) ++ng;
    }
    int j = kSlots;
#pragma unroll
    for (int kk = kSlots - 1; kk >= 0; --kk)
      if (kk > k && cs[kk] >= 0 && cs[kk] != seg) j = kk;
    if (head) {
      const int b = seg / a.Hkv, g = seg % a.Hkv;
      const int seg_start = s_pref[b] + g * s_nk[b];
      const int seg_end = seg_start + s_nk[b];
      const int wg = blockIdx.x;
      const int g0 = wg_begin(wg, U, a.R), g1 = wg_begin(wg + 1, U, a.R);
      const bool whole = seg_start >= g0 && seg_end <= g1;
      const bool own = !whole && seg_start >= g0;
      s_gd[rank] = make_int4(k | (j << 8) | (whole ? 1 << 16 : 0) | (own ? 1 << 17 : 0), seg,
                             own ? wg_of(seg_end - 1, U, a.R) : 0, 0);
    }
    if (k == 0) s_ng = ng;
  }
  __syncthreads();
  const int wg = blockIdx.x;
  int owner = -1, owner_last = 0;            // cut segment that begins in this range
  const int ng = s_ng;
  for (int gi = 0; gi < ng; ++gi) {
    const int4 gd = s_gd[gi];
    // Slots i .. j-1 with s_cseg == seg form the group (the others weigh 0).
    const int i = gd.x & 255, j = (gd.x >> 8) & 255;
    const bool whole = (gd.x >> 16) & 1;
    const int seg = gd.y;
    const long long slot = static_cast<long long>(wg) + seg;
    if ((gd.x >> 17) & 1) {
      owner = seg;
      owner_last = gd.z;
    }
    for (int o = threadIdx.x; o < G * D / 4; o += kThreads) {
      const int r = (4 * o) / D, d = 4 * o - r * D;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int k = 0; k < kSlots; ++k) {
        const float f = s_wf[k * kMaxGroup + r];
        const float4 v = *reinterpret_cast<const float4*>(s_cacc + (k * G + r) * D + d);
        if (k >= i && k < j && f != 0.f) {
          acc.x += f * v.x;
          acc.y += f * v.y;
          acc.z += f * v.z;
          acc.w += f * v.w;
        }
      }
      const float M = s_wm[i * kMaxGroup + r], L = s_wl[i * kMaxGroup + r];
      if (whole) {
        const long long oh = static_cast<long long>(seg) * G + r;    // b H_q + g G + r
        const float4 res = L > 0.f ? make_float4(acc.x / L, acc.y / L, acc.z / L, acc.w / L)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
        *reinterpret_cast<float4*>(a.out + oh * D + d) = res;
        if (d == 0 && a.lse) a.lse[oh] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
      } else {
        *reinterpret_cast<float4*>(a.part_acc + (slot * G + r) * D + d) = acc;
        if (d == 0) {
          a.part_ml[(slot * G + r) * 2 + 0] = M;
          a.part_ml[(slot * G + r) * 2 + 1] = L;
        }
      }
    }
  }
  if (threadIdx.x == 0) a.rec[wg] = make_int4(owner, owner_last, U, 0);
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_f32_kernel(DecodeArgs a) {
  constexpr int DPL = D / 64;     // dims per lane
  extern __shared__ int s_mem[];
  __shared__ int s_red[kWaves];
  int* s_pref = s_mem;
  int* s_nk = s_mem + a.B + 1;
  int* s_N = s_nk + a.B;
  build_plan(a, s_pref, s_nk, s_N, s_red);
  const int U = s_pref[a.B];
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * kWaves + (threadIdx.x >> 6);
  zero_empty<D>(a, s_nk);
  // This wave's record; replaced below (same lane, program order) when a
  // segment that begins in its range is cut.
  if (lane == 0) a.rec[w] = make_int4(-1, 0, 0, 0);
  if (U == 0) return;
  const int u0 = range_begin(w, U, a.W), u1 = range_begin(w + 1, U, a.W);
  if (u0 >= u1) return;
  const int t16 = lane & 15, hs = lane >> 4;
  const int G = a.G;
  const int Hq = a.Hkv * G;
  const float* q = static_cast<const float*>(a.q);
  const float* kc = static_cast<const float*>(a.kc);
  const float* vc = static_cast<const float*>(a.vc);

  int ubase = u0;
  UnitMeta win = unit_meta(a, ubase + lane, u1, s_pref, s_nk, s_N);
  int cur_seg = -1;
  long long qbase = 0;
  float m_run[kMaxGroup], l_run[kMaxGroup], o[kMaxGroup][DPL];

  auto flush = [&]() {
    const int b = cur_seg / a.Hkv, g = cur_seg % a.Hkv;
    const int seg_start = s_pref[b] + g * s_nk[b];
    const int seg_end = seg_start + s_nk[b];
    const bool whole = seg_start >= u0 && seg_end <= u1;
    const long long slot = static_cast<long long>(w) + cur_seg;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h >= G) continue;
      if (whole) {
        const long long oh = static_cast<long long>(b) * Hq + g * G + h;
        const float inv = l_run[h] > 0.f ? 1.f / l_run[h] : 0.f;
#pragma unroll
        for (int y = 0; y < DPL; ++y) a.out[oh * D + lane + 64 * y] = o[h][y] * inv;
        if (lane == 0 && a.lse)
          a.lse[oh] = l_run[h] > 0.f ? (m_run[h] + log2f(l_run[h])) * kLn2 : -INFINITY;
      } else {
        if (h == 0 && lane == 0 && seg_start >= u0)
          a.rec[w] = make_int4(cur_seg, wave_of(seg_end - 1, U, a.W), U, 0);
#pragma unroll
        for (int y = 0; y < DPL; ++y) a.part_acc[(slot * G + h) * D + lane + 64 * y] = o[h][y];
        if (lane == 0) {
          a.part_ml[(slot * G + h) * 2 + 0] = m_run[h];
          a.part_ml[(slot * G + h) * 2 + 1] = l_run[h];
        }
      }
    }
  };

  for (int u = u0; u < u1; ++u) {
    int i = static_cast<int>(u - ubase);
    if (i == kWindow) {
      ubase = u;
      i = 0;
      win = unit_meta(a, ubase + lane, u1, s_pref, s_nk, s_N);
    }
    const int seg = __shfl(win.seg, i);
    if (seg != cur_seg) {
      if (cur_seg >= 0) flush();
      cur_seg = seg;
      const int b = seg / a.Hkv, g = seg % a.Hkv;
      qbase = (static_cast<long long>(b) * Hq + g * G) * D;
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        m_run[h] = -INFINITY;
        l_run[h] = 0.f;
#pragma unroll
        for (int y = 0; y < DPL; ++y) o[h][y] = 0.f;
      }
    }
    const int p = __shfl(win.p, i);
    const int nv = __shfl(win.nv, i);
    if (p < 0) continue;
    const long long tile = (static_cast<long long>(p) * a.Hkv + (seg % a.Hkv)) * kBlock * D;
    // Scores: lane (t16, hs) takes token t16 for heads hs, hs+4, hs+8, hs+12.
    float sc[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int h = hs + 4 * x;
      float dot = 0.f;
      if (h < G && t16 < nv) {
        for (int d = 0; d < D; ++d) dot += q[qbase + h * D + d] * kc[tile + t16 * D + d];
        sc[x] = dot * a.scale_log2;
      } else {
        sc[x] = -INFINITY;
      }
    }
    float vv[DPL][kBlock];
#pragma unroll
    for (int y = 0; y < DPL; ++y)
#pragma unroll
      for (int tt = 0; tt < kBlock; ++tt)
        vv[y][tt] = (tt < nv) ? vc[tile + (lane + 64 * y) * kBlock + tt] : 0.f;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h >= G) continue;
      float st[kBlock];
      float mb = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < kBlock; ++tt) {
        st[tt] = __shfl(sc[h >> 2], 16 * (h & 3) + tt);
        mb = fmaxf(mb, st[tt]);
      }
      const float m_new = fmaxf(m_run[h], mb);
      const float alpha = exp2f(m_run[h] - m_new);
      float lsum = 0.f;
      float acc[DPL];
#pragma unroll
      for (int y = 0; y < DPL; ++y) acc[y] = 0.f;
#pragma unroll
      for (int tt = 0; tt < kBlock; ++tt) {
        const float pt = exp2f(st[tt] - m_new);
        lsum += pt;
#pragma unroll
        for (int y = 0; y < DPL; ++y) acc[y] += pt * vv[y][tt];
      }
      l_run[h] = l_run[h] * alpha + lsum;
#pragma unroll
      for (int y = 0; y < DPL; ++y) o[h][y] = o[h][y] * alpha + acc[y];
      m_run[h] = m_new;
    }
  }
  flush();
}

// Merge of the partials of every segment that the decode ranges cut.  One
// workgroup per (decode range, slice of the G x d outputs); the range's
// record names the cut segment that begins in it, if any, and the last range
// holding a piece of it; a.nsl slices of at most 256 groups of four outputs
// per segment.  Each thread merges four consecutive outputs of one head row
// on its own (a partial's max and sum loaded once, its four sums as one
// 16-byte load), in range order, with a running (max, sum, output) rescaled
// as the maximum grows; the loads of eight partials are issued together, so
// one memory round trip follows the record for segments cut into at most
// eight pieces.  Ranges with no units (fewer units than ranges) wrote no
// partial.
constexpr int kCombinePrefetch = 8;        // partials whose loads are issued together

template <int D>
__device__ __forceinline__ void combine_body(const DecodeArgs& a, int item) {
  const int range = item / a.nsl, slice = item - range * a.nsl;
  const int4 rec = a.rec[range];
  const int seg = rec.x;
  if (seg < 0) return;                       // no cut segment begins in this range
  const int U = rec.z;
  const int w0 = range, w1 = rec.y;
  const int G = a.G;
  const int b = seg / a.Hkv, g = seg % a.Hkv;
  const int Hq = a.Hkv * G;
  const int q4 = slice * kThreads + static_cast<int>(threadIdx.x);   // group of four outputs
  if (q4 >= G * D / 4) return;
  const int r = (4 * q4) / D, d = 4 * q4 - r * D;
  const long long ob = static_cast<long long>(b) * Hq + g * G;   // first output head row
  float M = -INFINITY, L = 0.f;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = w0; c0 <= w1; c0 += kCombinePrefetch) {
    float m[kCombinePrefetch], l[kCombinePrefetch];
    f32x4_t v[kCombinePrefetch];
#pragma unroll
    for (int k = 0; k < kCombinePrefetch; ++k) {
      const int wi = c0 + k;
      const bool ok = wi <= w1 && (a.xw ? wg_begin(wi + 1, U, a.R) > wg_begin(wi, U, a.R)
                                        : range_begin(wi + 1, U, a.R) > range_begin(wi, U, a.R));
      const long long slot = static_cast<long long>(wi) + seg;
      m[k] = ok ? a.part_ml[(slot * G + r) * 2 + 0] : -INFINITY;
      l[k] = ok ? a.part_ml[(slot * G + r) * 2 + 1] : 0.f;
      v[k] = ok ? *reinterpret_cast<const f32x4_t*>(a.part_acc + (slot * G + r) * D + d)
                : f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int k = 0; k < kCombinePrefetch; ++k) {
      if (!(l[k] > 0.f)) continue;
      const float Mn = fmaxf(M, m[k]);
      const float f_old = (M == -INFINITY) ? 0.f : exp2f(M - Mn);
      const float f_new = exp2f(m[k] - Mn);
      L = L * f_old + l[k] * f_new;
      acc = acc * f_old + v[k] * f_new;
      M = Mn;
    }
  }
  const f32x4_t res = L > 0.f ? acc / L : f32x4_t{0.f, 0.f, 0.f, 0.f};
  *reinterpret_cast<f32x4_t*>(a.out + (ob + r) * D + d) = res;
  if (d == 0 && a.lse) a.lse[ob + r] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
}

template <int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(DecodeArgs a) {
  combine_body<D>(a, blockIdx.x);
}

// The merge and, on workgroups of their own placed first (their chains of
// dependent loads then overlap the merge instead of following it), the
// append of one token per sequence (APP: ent_decode_step_append) and the
// sampling of every row (nS = B; the decode step with long block tables).
// The merge reads only partials and records and writes outputs; the appends
// write the caches, the summaries and the lengths; sampling reads the logits
// and their row statistics: none of them reads what another writes.
template <int D, typename T, bool APP, bool VEC>
__global__ __launch_bounds__(kThreads) void merge_kernel(DecodeArgs a, AppendArgs ap, SampleArgs sp,
                                                         int nS) {
  static_assert(kThreads == kAppendThreads && kThreads == kSampleThreads, "workgroup size");
  __shared__ SampleShared ssh;
  int id = blockIdx.x;
  if (APP) {
    if (id < a.B) {
      append_body<T>(ap, id);
      return;
    }
    id -= a.B;
  }
  if (id < nS) {
    const int tok = sample_body<VEC>(sp.logits, sp.ld, sp.V, sp.C, sp.stats,
                                     sp.temp_used[id] * sp.t_cal, sp.uniforms[id], id, ssh);
    if (threadIdx.x == 0) sp.tokens[id] = tok;
    return;
  }
  combine_body<D>(a, id - nS);
}

template <typename K>
int occupancy_blocks(K kernel, size_t lds) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kThreads, lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

size_t plan_lds_bytes(int B) { return static_cast<size_t>(3 * B + 1) * sizeof(int); }

// bf16 decode: the workgroup's cut partials, then the plan.
size_t decode_lds_bytes(int B, int G, int D) {
  return static_cast<size_t>(2 * kWaves) * (static_cast<size_t>(G) * D + kMaxGroup * 2) * sizeof(float) +
         plan_lds_bytes(B);
}

}  // namespace

// Resident decode workgroups per CU, at most: with two instead of the three
// the registers allow, each wave has half as many units again, and on the
// 70B-shaped loop the decode entry point took 118.0-118.8 us against
// 121.2-121.4 us (the 8B step unchanged).
constexpr int kDecodePerCu = 2;

int decode_grid_size(const ent_ctx* c) {
  const ent_config& cf = c->cfg;
  const size_t lds = plan_lds_bytes(cf.max_batch);
  const size_t lds16 = decode_lds_bytes(cf.max_batch, c->group, cf.head_dim);
  int per_cu = 1;
  if (cf.kv_dtype == ENT_BF16)
    per_cu = cf.head_dim == 128 ? occupancy_blocks(decode_bf16_kernel<128>, lds16)
                                : occupancy_blocks(decode_bf16_kernel<64>, lds16);
  else
    per_cu = cf.head_dim == 128 ? occupancy_blocks(decode_f32_kernel<128>, lds)
                                : occupancy_blocks(decode_f32_kernel<64>, lds);
  return c->num_cu * std::min(per_cu, kDecodePerCu);
}

long long decode_partial_slots(int decode_grid, int max_batch, int num_kv_heads) {
  return static_cast<long long>(decode_grid) * kWaves +
         static_cast<long long>(max_batch) * num_kv_heads;
}

hipError_t launch_decode(const ent_ctx* c, int B, const void* q, const void* k_cache,
                         const void* v_cache, const int* tables, const int* ctx_lens,
                         const int* kept, const int* n_kept, float* out, float* lse,
                         hipStream_t s, const int* kept_phys, const AppendArgs* ap,
                         const SampleArgs* sp) {
  const ent_config& cf = c->cfg;
  DecodeArgs a;
  a.q = q;
  a.kc = k_cache;
  a.vc = v_cache;
  a.tables = tables;
  a.ctx_lens = ctx_lens;
  a.kept = kept;
  a.kept_phys = kept_phys;
  a.n_kept = n_kept;
  a.out = out;
  a.lse = lse;
  a.part_acc = c->dec_acc;
  a.part_ml = c->dec_ml;
  a.rec = c->dec_rec;
  a.flags = c->dev_flags;
  a.B = B;
  a.Hkv = cf.num_kv_heads;
  a.G = c->group;
  a.MAXB = cf.max_blocks_per_seq;
  a.P = cf.num_pool_blocks;
  a.W = c->decode_grid * kWaves;
  a.R = cf.kv_dtype == ENT_BF16 ? c->decode_grid : a.W;
  a.xw = cf.kv_dtype == ENT_BF16 ? 1 : 0;
  a.scale_log2 = cf.scale * kLog2e;
  const size_t lds = plan_lds_bytes(B);
  const dim3 grid(c->decode_grid);
  if (cf.kv_dtype == ENT_BF16) {
    const size_t lds16 = decode_lds_bytes(B, c->group, cf.head_dim);
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(decode_bf16_kernel<128>, grid, dim3(kThreads), lds16, s, a);
    else
      hipLaunchKernelGGL(decode_bf16_kernel<64>, grid, dim3(kThreads), lds16, s, a);
  } else {
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(decode_f32_kernel<128>, grid, dim3(kThreads), lds, s, a);
    else
      hipLaunchKernelGGL(decode_f32_kernel<64>, grid, dim3(kThreads), lds, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Slices per segment: four outputs per merge thread.
  a.nsl = (c->group * cf.head_dim / 4 + kThreads - 1) / kThreads;
  const int n_combine = a.R * a.nsl;
  if (ap || sp) {
    const int nS = sp ? B : 0;
    const dim3 g2(n_combine + (ap ? B : 0) + nS);
    const bool vec = !sp || row_vec_ok(sp->logits, sp->ld);
    const AppendArgs an{};
    const SampleArgs sn{};
    const AppendArgs& aa = ap ? *ap : an;
    const SampleArgs& ss = sp ? *sp : sn;
#define ENT_MERGE(DD, TT, AP)                                                                  \
  do {                                                                                         \
    if (vec)                                                                                   \
      hipLaunchKernelGGL((merge_kernel<DD, TT, AP, true>), g2, dim3(kThreads), 0, s, a, aa, ss, nS); \
    else                                                                                       \
      hipLaunchKernelGGL((merge_kernel<DD, TT, AP, false>), g2, dim3(kThreads), 0, s, a, aa, ss, nS); \
  } while (0)
#define ENT_MERGE_D(DD)                                      \
  do {                                                       \
    if (!ap) ENT_MERGE(DD, uint16_t, false);                 \
    else if (ap->bf16) ENT_MERGE(DD, uint16_t, true);        \
    else ENT_MERGE(DD, float, true);                         \
  } while (0)
    if (cf.head_dim == 128) ENT_MERGE_D(128);
    else ENT_MERGE_D(64);
#undef ENT_MERGE_D
#undef ENT_MERGE
    return hipGetLastError();
  }
  const dim3 cgrid(n_combine);
  if (cf.head_dim == 128)
    hipLaunchKernelGGL(combine_kernel<128>, cgrid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(combine_kernel<64>, cgrid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ent
