// The two streaming passes that open a decode step, as one grid of
// independent 256-thread workgroups with two roles:
//
//   * block scoring (bf16 queries): workgroup (sequence b, tile of 16
//     blocks, group of four KV heads); wave w takes KV head 4 hg + w
//     (score_head_load / score_head_compute, Section 3.2);
//   * entropy chunk passes: workgroup (row b, chunk c) of 4096 logits
//     (entropy_chunk_body, Section 2.1).
//
// Both read HBM once (block summaries, logits) at a few flops per byte and
// do not depend on each other.  Scoring workgroups come first (they run
// longer).  Every workgroup keeps few registers, so many are resident at
// once and their loads overlap.  Tiles past a sequence's last block exit at
// once.  The per-stage entry points launch the same kernel with one role
// only, which keeps their results bit-identical to the fused step's.

#include "blocks_dev.h"
#include "entropy_dev.h"

namespace ent {
namespace {

constexpr int kProThreads = 256;
constexpr int kProWaves = kProThreads / 64;

__host__ __device__ inline int score_tiles(int MAXB) { return (MAXB + kMfmaChunk - 1) / kMfmaChunk; }
__host__ __device__ inline int head_groups(int Hkv) { return (Hkv + kProWaves - 1) / kProWaves; }

template <bool VEC, int D>
__global__ __launch_bounds__(kProThreads) void prologue_kernel(PrologueArgs a) {
  __shared__ float red[16];
  const int id = blockIdx.x;
  const int nhg = head_groups(a.Hkv);
  const int nsc = a.do_score ? a.B * score_tiles(a.MAXB) * nhg : 0;
  if (id < nsc) {
    const int per_b = score_tiles(a.MAXB) * nhg;
    const int b = id / per_b;
    const int r = id - b * per_b;
    const int ch = r / nhg;
    const int g = (r - ch * nhg) * kProWaves + (threadIdx.x >> 6);
    const int N = a.ctx_lens[b];
    if (N < 0 || N > a.MAXB * kBlock) return;    // flagged by the selection stage
    const int nb = (N + kBlock - 1) / kBlock;
    if (ch * kMfmaChunk >= nb || g >= a.Hkv) return;
    const int p = score_tile_block(a.tables, b, ch, a.MAXB, nb, a.P, a.flags);
    float4 buf[kScoreSlots];
    score_head_load<D>(a.ksum, p, a.Hkv, g, buf);
    score_head_compute<D>(a.q, buf, a.zbuf, a.lse_part, b, ch, g, N, nb, a.Hkv, a.G, a.MAXB,
                          a.nch_max, a.scale);
    return;
  }
  const int e = id - nsc;
  const int b = e / a.C;
  entropy_chunk_body<VEC>(a.logits, a.ld, a.V, a.C, a.temp, a.part, a.row_stats, e - b * a.C, b,
                          red);
}

}  // namespace

hipError_t launch_prologue(const ent_ctx* c, const PrologueArgs& a, hipStream_t s) {
  const ent_config& cf = c->cfg;
  long long grid = 0;
  if (a.do_score) grid += static_cast<long long>(a.B) * score_tiles(a.MAXB) * head_groups(a.Hkv);
  if (a.do_entropy) grid += static_cast<long long>(a.B) * a.C;
  if (grid == 0) return hipSuccess;
  const bool vec = !a.do_entropy || row_vec_ok(a.logits, a.ld);
  const dim3 g(static_cast<unsigned>(grid));
  if (cf.head_dim == 128) {
    if (vec)
      hipLaunchKernelGGL((prologue_kernel<true, 128>), g, dim3(kProThreads), 0, s, a);
    else
      hipLaunchKernelGGL((prologue_kernel<false, 128>), g, dim3(kProThreads), 0, s, a);
  } else {
    if (vec)
      hipLaunchKernelGGL((prologue_kernel<true, 64>), g, dim3(kProThreads), 0, s, a);
    else
      hipLaunchKernelGGL((prologue_kernel<false, 64>), g, dim3(kProThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ent
