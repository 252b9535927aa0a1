// The two streaming passes that open a decode step, as one persistent grid:
//
//   * entropy chunk passes: item (row b, chunk c) = 4096 logits, one wave
//     (chunk_load_wave / chunk_reduce_wave, Section 2.1);
//   * block scoring (bf16 queries): item (sequence b, tile of 16 blocks,
//     KV heads g0 and g0 + 1), one wave (score_pair_load /
//     score_pair_compute, Section 3.2).
//
// Both read HBM once (logits, block summaries) at a few flops per byte and
// do not depend on each other.  Items are numbered scoring first (sequence-
// major, then tile, then head pair), then entropy (row-major, then chunk);
// wave w of the grid takes items w, w + NW, ...  Each wave keeps the next
// item's loads in flight while it reduces the current one, and the grid is
// sized to the resident capacity, so no workgroup waits for a slot.  The
// per-stage entry points run the same kernel with only one kind of item,
// which keeps their results bit-identical to the fused step's.

#include "blocks_dev.h"
#include "entropy_dev.h"

#include <algorithm>

namespace ent {
namespace {

constexpr int kProThreads = 256;
constexpr int kProWaves = kProThreads / 64;

// Tile plan in LDS: s_pref[b] = first tile of sequence b (s_pref[B] = all
// tiles), s_nb[b] = blocks of b (0 when its context length is invalid; the
// selection stage flags those), s_N[b] = its context length.
__device__ void tile_plan(const int* __restrict__ ctx_lens, int B, int MAXB, int* s_pref,
                          int* s_nb, int* s_N, int* s_red) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = (B + kProThreads - 1) / kProThreads;
  int loc = 0;
  for (int i = 0; i < per; ++i) {
    const int b = t * per + i;
    if (b < B) {
      const int N = ctx_lens[b];
      const int nb = (N >= 0 && N <= MAXB * kBlock) ? (N + kBlock - 1) / kBlock : 0;
      s_nb[b] = nb;
      s_N[b] = N;
      loc += (nb + kMfmaChunk - 1) / kMfmaChunk;
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
      run += (s_nb[b] + kMfmaChunk - 1) / kMfmaChunk;
    }
  }
  if (t == kProThreads - 1) s_pref[B] = run;
  __syncthreads();
}

struct Item {
  int kind;     // 0 scoring, 1 entropy, -1 none
  int b;
  int x;        // tile (scoring) or chunk (entropy)
  int g0;       // first KV head (scoring)
};

template <bool VEC, int D>
__global__ __launch_bounds__(kProThreads) void prologue_kernel(PrologueArgs a) {
  extern __shared__ int s_mem[];
  __shared__ int s_red[kProWaves];
  int* s_pref = s_mem;
  int* s_nb = s_mem + a.B + 1;
  int* s_N = s_nb + a.B;
  long long n_score = 0;
  const int ngp = (a.Hkv + 1) / 2;
  if (a.do_score) {
    tile_plan(a.ctx_lens, a.B, a.MAXB, s_pref, s_nb, s_N, s_red);
    n_score = static_cast<long long>(s_pref[a.B]) * ngp;
  }
  const long long n_ent = a.do_entropy ? static_cast<long long>(a.B) * a.C : 0;
  const long long n = n_score + n_ent;
  const long long NW = static_cast<long long>(gridDim.x) * kProWaves;
  const long long w = static_cast<long long>(blockIdx.x) * kProWaves + (threadIdx.x >> 6);

  auto item_of = [&](long long idx) {
    Item it{-1, 0, 0, 0};
    if (idx >= n) return it;
    if (idx < n_score) {
      const int i = static_cast<int>(idx);       // < 2^31 under the configuration limits
      const int t = i / ngp;
      int lo = 0, hi = a.B;               // largest b with s_pref[b] <= t
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_pref[mid] <= t) lo = mid; else hi = mid;
      }
      it.kind = 0;
      it.b = lo;
      it.x = t - s_pref[lo];
      it.g0 = 2 * (i - t * ngp);
    } else {
      const int e = static_cast<int>(idx - n_score);   // B C < 2^31
      it.kind = 1;
      it.b = e / a.C;
      it.x = e - it.b * a.C;
    }
    return it;
  };
  // Issue the item's loads into buf (and its temperature into T).
  auto load_item = [&](const Item& it, float4 (&buf)[kWaveSlots], float& T) {
    if (it.kind == 0) {
      const int p = score_tile_block(a.tables, it.b, it.x, a.MAXB, s_nb[it.b], a.P, a.flags);
      score_pair_load<D>(a.ksum, p, a.Hkv, it.g0, min(2, a.Hkv - it.g0), buf);
    } else if (it.kind == 1) {
      T = a.temp[it.b];
      chunk_load_wave<VEC>(a.logits + static_cast<long long>(it.b) * a.ld, a.V, it.x, buf);
    }
  };
  auto compute_item = [&](const Item& it, const float4 (&buf)[kWaveSlots], float T) {
    if (it.kind == 0) {
      const int nb = s_nb[it.b];
      const int N = s_N[it.b];
      score_pair_compute<D>(a.q, buf, a.zbuf, a.lse_part, it.b, it.x, it.g0,
                            min(2, a.Hkv - it.g0), N, nb, a.Hkv, a.G, a.MAXB, a.nch_max,
                            a.scale);
    } else if (it.kind == 1) {
      chunk_reduce_wave(buf, T, a.part, a.row_stats,
                        static_cast<long long>(it.b) * a.C + it.x);
    }
  };

  static_assert(kScorePairSlots == kWaveSlots, "one register buffer serves both item kinds");
  float4 cur[kWaveSlots], nxt[kWaveSlots];
  float Tc = 1.f, Tn = 1.f;
  Item it = item_of(w);
  load_item(it, cur, Tc);
  for (long long idx = w; idx < n; idx += NW) {
    const Item nit = item_of(idx + NW);
    load_item(nit, nxt, Tn);
    compute_item(it, cur, Tc);
    it = nit;
    Tc = Tn;
#pragma unroll
    for (int i = 0; i < kWaveSlots; ++i) cur[i] = nxt[i];
  }
}

template <bool VEC, int D>
int prologue_per_cu() {
  int n = 0;
  const size_t lds = 0;     // the plan's dynamic LDS is small next to the limit
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, prologue_kernel<VEC, D>, kProThreads,
                                                   lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

}  // namespace

int prologue_grid_size(const ent_ctx* c) {
  const int d = c->cfg.head_dim;
  const int n = d == 128 ? std::min(prologue_per_cu<true, 128>(), prologue_per_cu<false, 128>())
                         : std::min(prologue_per_cu<true, 64>(), prologue_per_cu<false, 64>());
  return c->num_cu * n;
}

hipError_t launch_prologue(const ent_ctx* c, const PrologueArgs& a, hipStream_t s) {
  const ent_config& cf = c->cfg;
  // Upper bound of the items: no more workgroups than can have work.
  long long items = 0;
  if (a.do_entropy) items += static_cast<long long>(a.B) * a.C;
  if (a.do_score)
    items += static_cast<long long>(a.B) * ((cf.max_blocks_per_seq + kMfmaChunk - 1) / kMfmaChunk) *
             ((cf.num_kv_heads + 1) / 2);
  if (items == 0) return hipSuccess;
  const long long want = (items + kProWaves - 1) / kProWaves;
  const int grid = static_cast<int>(std::min<long long>(c->prologue_grid, want));
  const size_t lds = static_cast<size_t>(3 * a.B + 1) * sizeof(int);
  const bool vec = !a.do_entropy || row_vec_ok(a.logits, a.ld);
  if (cf.head_dim == 128) {
    if (vec)
      hipLaunchKernelGGL((prologue_kernel<true, 128>), dim3(grid), dim3(kProThreads), lds, s, a);
    else
      hipLaunchKernelGGL((prologue_kernel<false, 128>), dim3(grid), dim3(kProThreads), lds, s, a);
  } else {
    if (vec)
      hipLaunchKernelGGL((prologue_kernel<true, 64>), dim3(grid), dim3(kProThreads), lds, s, a);
    else
      hipLaunchKernelGGL((prologue_kernel<false, 64>), dim3(grid), dim3(kProThreads), lds, s, a);
  }
  return hipGetLastError();
}

}  // namespace ent
