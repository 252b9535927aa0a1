// Decode attention over the kept blocks only (Section 3.2 of the paper:
// attention computation is restricted to the kept block set).
//
// Work decomposition.  A work item is (sequence b, KV head g, split s): up to
// kSplitBlocks consecutive entries of b's kept list, for the G query heads
// that share KV head g.  Items are enumerated from the device-resident kept
// counts (sequences with nothing kept still get one item, which writes zeros),
// so the host never learns how much was pruned.  The grid is persistent: each
// wave walks items with a grid stride.  A (b, g) pair split over several items
// writes (max, sum, unnormalised output) partials, which a second kernel
// merges; a pair with one item writes its output directly.
//
// bf16 path (MFMA, gfx950).  Per kept block of 16 tokens:
//   S^T[16 tok x 16 heads] = K[16 x d] . Q^T[d x 16]   v_mfma_f32_16x16x32_bf16,
//     A = K rows straight from the token-major K tile (16 B per lane per step),
//     B = the G query heads (zero-padded to 16 columns), held in registers;
//   online softmax per head column (log2 domain, fp32);
//   O^T[d x 16] += V^T[d x 16 tok] . P^T[16 tok x 16]   v_mfma_f32_16x16x16_bf16,
//     A = rows of the dim-major V tile (8 B per lane per 16-dim tile),
//     B = P^T taken straight from the S^T accumulator registers, split into
//         a bf16 high part and a bf16 remainder (two MFMAs), so P keeps
//         about 16 bits.
// fp32 path (VALU): the same items and merge, scalar dot products.

#include "ent_internal.h"

#include <math.h>

namespace ent {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int CB = kSplitBlocks;

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4_t __attribute__((__vector_size__(4 * sizeof(short))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const int* tables;
  const int* ctx_lens;
  const int* kept;
  const int* n_kept;
  float* out;
  float* lse;
  float* part_acc;
  float* part_ml;
  unsigned* flags;
  int B, Hkv, G, MAXB, P, splits_max;
  float scale_log2;   // softmax scale times log2(e)
};

// Builds, in LDS, the first work item of each sequence (s_pref[0..B]) and its
// number of splits (s_ns[0..B-1]).
__device__ void build_items(const DecodeArgs& a, int* s_pref, int* s_ns, int* s_red) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = (a.B + kThreads - 1) / kThreads;
  int loc = 0;
  for (int i = 0; i < per; ++i) {
    const int b = t * per + i;
    if (b < a.B) {
      const int nk = min(max(a.n_kept[b], 0), a.MAXB);
      const int ns = max(1, (nk + CB - 1) / CB);
      s_ns[b] = ns;
      loc += ns * a.Hkv;
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
      run += s_ns[b] * a.Hkv;
    }
  }
  if (t == kThreads - 1) s_pref[a.B] = run;
  __syncthreads();
}

struct Item {
  int b, g, sp, ns, N, nb, cnt;
  int my_j, my_p;   // lane i < cnt: kept block id and its physical block (-1 = skip)
};

__device__ __forceinline__ Item locate_item(const DecodeArgs& a, int item, const int* s_pref,
                                            const int* s_ns) {
  Item it;
  int lo = 0, hi = a.B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_pref[mid] <= item) lo = mid; else hi = mid;
  }
  it.b = lo;
  it.ns = s_ns[lo];
  const int rr = item - s_pref[lo];
  it.g = rr / it.ns;
  it.sp = rr % it.ns;
  const int lane = threadIdx.x & 63;
  const int N = a.ctx_lens[it.b];
  const bool ok = N >= 0 && N <= a.MAXB * kBlock;
  it.N = ok ? N : 0;
  it.nb = (it.N + kBlock - 1) / kBlock;
  const int nk = min(max(a.n_kept[it.b], 0), a.MAXB);
  const int j0 = it.sp * CB;
  it.cnt = max(0, min(nk, j0 + CB) - j0);
  it.my_j = -1;
  it.my_p = -1;
  if (lane < it.cnt) {
    const long long row = static_cast<long long>(it.b) * a.MAXB;
    const int j = a.kept[row + j0 + lane];
    if (j >= 0 && j < it.nb) {
      const int p = a.tables[row + j];
      if (p >= 0 && p < a.P) {
        it.my_j = j;
        it.my_p = p;
      } else if (it.g == 0) {
        raise_flag(a.flags, ENT_DEV_BAD_TABLE);
      }
    } else if (it.g == 0) {
      raise_flag(a.flags, ENT_DEV_BAD_TABLE);
    }
  }
  return it;
}

// Merge of the split partials of each (b, g) pair that was split: one wave
// per pair; pairs with a single split were finalised by the decode kernel.
template <int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(DecodeArgs a) {
  const int pair = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (pair >= a.B * a.Hkv) return;
  const int b = pair / a.Hkv, g = pair % a.Hkv;
  const int nk = min(max(a.n_kept[b], 0), a.MAXB);
  const int ns = max(1, (nk + CB - 1) / CB);
  if (ns == 1) return;
  const int Hq = a.Hkv * a.G;
  const long long base = static_cast<long long>(pair) * a.splits_max;
  for (int idx = lane; idx < a.G * D; idx += 64) {
    const int r = idx / D, d = idx % D;
    float M = -INFINITY;
    for (int s = 0; s < ns; ++s) {
      const float* ml = a.part_ml + ((base + s) * a.G + r) * 2;
      if (ml[1] > 0.f) M = fmaxf(M, ml[0]);
    }
    float Ls = 0.f, O = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float* ml = a.part_ml + ((base + s) * a.G + r) * 2;
      const float ls = ml[1];
      if (ls > 0.f) {
        const float f = exp2f(ml[0] - M);
        Ls += ls * f;
        O += a.part_acc[((base + s) * a.G + r) * D + d] * f;
      }
    }
    const long long oh = static_cast<long long>(b) * Hq + g * a.G + r;
    a.out[oh * D + d] = Ls > 0.f ? O / Ls : 0.f;
    if (d == 0 && a.lse) a.lse[oh] = Ls > 0.f ? (M + log2f(Ls)) * kLn2 : -INFINITY;
  }
}

__device__ __forceinline__ bf16x8_t load_bf16x8(const uint16_t* p) {
  const uint4 x = *reinterpret_cast<const uint4*>(p);
  return __builtin_bit_cast(bf16x8_t, x);
}
__device__ __forceinline__ s16x4_t load_s16x4(const uint16_t* p) {
  const uint2 x = *reinterpret_cast<const uint2*>(p);
  return __builtin_bit_cast(s16x4_t, x);
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_bf16_kernel(DecodeArgs a) {
  constexpr int KS = D / 32;      // QK k-steps (32 dims each)
  constexpr int MT = D / 16;      // PV output tiles (16 dims each)
  constexpr int DL = D / 4;       // dims per lane group in QK
  extern __shared__ int s_mem[];
  __shared__ int s_red[kWaves];
  int* s_pref = s_mem;
  int* s_ns = s_mem + a.B + 1;
  build_items(a, s_pref, s_ns, s_red);
  const int total = s_pref[a.B];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, gq = lane >> 4;
  const int Hq = a.Hkv * a.G;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  const uint16_t* kc = static_cast<const uint16_t*>(a.kc);
  const uint16_t* vc = static_cast<const uint16_t*>(a.vc);

  for (int item = blockIdx.x * kWaves + wave; item < total; item += gridDim.x * kWaves) {
    const Item it = locate_item(a, item, s_pref, s_ns);
    const bool head_ok = r16 < a.G;
    const long long qh = static_cast<long long>(it.b) * Hq + it.g * a.G + r16;
    bf16x8_t qreg[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (head_ok) qreg[ks] = load_bf16x8(q + qh * D + gq * DL + ks * 8);
      else qreg[ks] = __builtin_bit_cast(bf16x8_t, make_uint4(0u, 0u, 0u, 0u));
    }
    float m_run = -INFINITY, l_run = 0.f;
    f32x4_t oacc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) oacc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int i = 0; i < it.cnt; ++i) {
      const int j = __shfl(it.my_j, i);
      const int p = __shfl(it.my_p, i);
      if (p < 0) continue;
      const int nv = (j == it.nb - 1) ? it.N - kBlock * (it.nb - 1) : kBlock;
      const long long tile = (static_cast<long long>(p) * a.Hkv + it.g) * kBlock * D;
      bf16x8_t kreg[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kreg[ks] = load_bf16x8(kc + tile + r16 * D + gq * DL + ks * 8);
      s16x4_t vreg[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) vreg[m] = load_s16x4(vc + tile + (16 * m + r16) * kBlock + 4 * gq);

      f32x4_t sacc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kreg[ks], qreg[ks], sacc, 0, 0, 0);
      float s[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] = (4 * gq + e < nv) ? sacc[e] * a.scale_log2 : -INFINITY;
      float mloc = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run, mloc);
      const float alpha = exp2f(m_run - m_new);
      float pe[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) pe[e] = exp2f(s[e] - m_new);
      l_run = l_run * alpha + ((pe[0] + pe[1]) + (pe[2] + pe[3]));
      s16x4_t phi, plo;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint16_t hb = f32_to_bf16_rne(pe[e]);
        phi[e] = static_cast<short>(hb);
        plo[e] = static_cast<short>(f32_to_bf16_rne(pe[e] - bf16_to_f32(hb)));
      }
      if (nv < kBlock) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * gq + e >= nv) vreg[m][e] = 0;
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        oacc[m] *= alpha;
        oacc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vreg[m], phi, oacc[m], 0, 0, 0);
        oacc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vreg[m], plo, oacc[m], 0, 0, 0);
      }
      m_run = m_new;
    }

    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (it.ns == 1) {
      if (head_ok) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const f32x4_t o = oacc[m] * inv;
          *reinterpret_cast<float4*>(a.out + qh * D + 16 * m + 4 * gq) =
              make_float4(o[0], o[1], o[2], o[3]);
        }
        if (gq == 0 && a.lse) a.lse[qh] = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
      }
    } else {
      const long long slot = (static_cast<long long>(it.b) * a.Hkv + it.g) * a.splits_max + it.sp;
      if (head_ok) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
          *reinterpret_cast<float4*>(a.part_acc + (slot * a.G + r16) * D + 16 * m + 4 * gq) =
              make_float4(oacc[m][0], oacc[m][1], oacc[m][2], oacc[m][3]);
        if (gq == 0) {
          a.part_ml[(slot * a.G + r16) * 2 + 0] = m_run;
          a.part_ml[(slot * a.G + r16) * 2 + 1] = l_tot;
        }
      }
    }
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_f32_kernel(DecodeArgs a) {
  constexpr int DPL = D / 64;     // dims per lane
  extern __shared__ int s_mem[];
  __shared__ int s_red[kWaves];
  int* s_pref = s_mem;
  int* s_ns = s_mem + a.B + 1;
  build_items(a, s_pref, s_ns, s_red);
  const int total = s_pref[a.B];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t16 = lane & 15, hs = lane >> 4;
  const int Hq = a.Hkv * a.G;
  const float* q = static_cast<const float*>(a.q);
  const float* kc = static_cast<const float*>(a.kc);
  const float* vc = static_cast<const float*>(a.vc);

  for (int item = blockIdx.x * kWaves + wave; item < total; item += gridDim.x * kWaves) {
    const Item it = locate_item(a, item, s_pref, s_ns);
    const long long qbase = (static_cast<long long>(it.b) * Hq + it.g * a.G) * D;
    float m_run[kMaxGroup], l_run[kMaxGroup], o[kMaxGroup][DPL];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      m_run[h] = -INFINITY;
      l_run[h] = 0.f;
#pragma unroll
      for (int y = 0; y < DPL; ++y) o[h][y] = 0.f;
    }
    for (int i = 0; i < it.cnt; ++i) {
      const int j = __shfl(it.my_j, i);
      const int p = __shfl(it.my_p, i);
      if (p < 0) continue;
      const int nv = (j == it.nb - 1) ? it.N - kBlock * (it.nb - 1) : kBlock;
      const long long tile = (static_cast<long long>(p) * a.Hkv + it.g) * kBlock * D;
      // Scores: lane (t16, hs) takes token t16 for heads hs, hs+4, hs+8, hs+12.
      float sc[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int h = hs + 4 * x;
        float dot = 0.f;
        if (h < a.G && t16 < nv) {
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
        if (h >= a.G) continue;
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
    if (it.ns == 1) {
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h >= a.G) continue;
        const long long oh = static_cast<long long>(it.b) * Hq + it.g * a.G + h;
        const float inv = l_run[h] > 0.f ? 1.f / l_run[h] : 0.f;
#pragma unroll
        for (int y = 0; y < DPL; ++y) a.out[oh * D + lane + 64 * y] = o[h][y] * inv;
        if (lane == 0 && a.lse)
          a.lse[oh] = l_run[h] > 0.f ? (m_run[h] + log2f(l_run[h])) * kLn2 : -INFINITY;
      }
    } else {
      const long long slot = (static_cast<long long>(it.b) * a.Hkv + it.g) * a.splits_max + it.sp;
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h >= a.G) continue;
#pragma unroll
        for (int y = 0; y < DPL; ++y) a.part_acc[(slot * a.G + h) * D + lane + 64 * y] = o[h][y];
        if (lane == 0) {
          a.part_ml[(slot * a.G + h) * 2 + 0] = m_run[h];
          a.part_ml[(slot * a.G + h) * 2 + 1] = l_run[h];
        }
      }
    }
  }
}

template <typename K>
int occupancy_blocks(K kernel, size_t lds) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kThreads, lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

}  // namespace

int decode_grid_size(const ent_ctx* c) {
  const ent_config& cf = c->cfg;
  const size_t lds = static_cast<size_t>(2 * cf.max_batch + 1) * sizeof(int);
  int per_cu = 1;
  if (cf.kv_dtype == ENT_BF16)
    per_cu = cf.head_dim == 128 ? occupancy_blocks(decode_bf16_kernel<128>, lds)
                                : occupancy_blocks(decode_bf16_kernel<64>, lds);
  else
    per_cu = cf.head_dim == 128 ? occupancy_blocks(decode_f32_kernel<128>, lds)
                                : occupancy_blocks(decode_f32_kernel<64>, lds);
  return c->num_cu * per_cu;
}

hipError_t launch_decode(const ent_ctx* c, int B, const void* q, const void* k_cache,
                         const void* v_cache, const int* tables, const int* ctx_lens,
                         const int* kept, const int* n_kept, float* out, float* lse,
                         hipStream_t s) {
  const ent_config& cf = c->cfg;
  DecodeArgs a;
  a.q = q;
  a.kc = k_cache;
  a.vc = v_cache;
  a.tables = tables;
  a.ctx_lens = ctx_lens;
  a.kept = kept;
  a.n_kept = n_kept;
  a.out = out;
  a.lse = lse;
  a.part_acc = c->dec_acc;
  a.part_ml = c->dec_ml;
  a.flags = c->dev_flags;
  a.B = B;
  a.Hkv = cf.num_kv_heads;
  a.G = c->group;
  a.MAXB = cf.max_blocks_per_seq;
  a.P = cf.num_pool_blocks;
  a.splits_max = c->splits_max;
  a.scale_log2 = cf.scale * kLog2e;
  const size_t lds = static_cast<size_t>(2 * B + 1) * sizeof(int);
  const dim3 grid(c->decode_grid);
  if (cf.kv_dtype == ENT_BF16) {
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(decode_bf16_kernel<128>, grid, dim3(kThreads), lds, s, a);
    else
      hipLaunchKernelGGL(decode_bf16_kernel<64>, grid, dim3(kThreads), lds, s, a);
  } else {
    if (cf.head_dim == 128)
      hipLaunchKernelGGL(decode_f32_kernel<128>, grid, dim3(kThreads), lds, s, a);
    else
      hipLaunchKernelGGL(decode_f32_kernel<64>, grid, dim3(kThreads), lds, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 cgrid((B * cf.num_kv_heads + kWaves - 1) / kWaves);
  if (cf.head_dim == 128)
    hipLaunchKernelGGL(combine_kernel<128>, cgrid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(combine_kernel<64>, cgrid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ent
