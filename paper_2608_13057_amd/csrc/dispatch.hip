// Stage 1 of one GPU's share of the EP MoE block: per-expert counts of the
// routed (token, k) pairs, application of the per-batch split plan, padding of
// every local slot to whole M-tiles and the stable permutation of the pairs'
// activation rows into those padded groups.
//
// Definition: the fixed-charge dispatch problem (Sec. 3.1) -- counts n_e,
// shares x_{e,g} over the replicas R(e) -- with the paper's integration rules
// (Sec. 4.4): counts are masked against graph-padding rows, plan rows are
// renormalised at use and a zero-sum row falls back to uniform over the
// replicas holding the expert; grouped GEMM works on M-tiles (Sec. 2.2,
// Eq. 2).  The paper's in-graph kernel samples a replica per pair; here the
// split is the deterministic integer reading documented in the header, so
// the outputs are reproducible bit for bit.
//
// Three launches, none of which needs zeroed memory:
//   k_count   -- blocks of 1024 pairs: per-block histogram in LDS and the
//                stable rank of each pair within (block, expert), from wave
//                ballots (lanes of one wave with equal expert ids are found
//                with one ballot per id bit; ranks = popcount of the lower
//                lanes), plus per-wave counts for the waves before it.
//   k_plan    -- one block: per-expert exclusive scan of the block counts,
//                n_e, the plan split of each expert over its slots, padded
//                sizes, slot offsets, the tile count, padding-row markers.
//   k_scatter -- blocks of 32 pairs: rank -> slot -> row, index outputs, and
//                the copy of the activation row (16-byte loads/stores, one
//                wavefront per row).
#include "internal.h"

namespace tempo {
namespace {

__global__ __launch_bounds__(kCountThreads) void k_count(const int32_t* __restrict__ ids, int Pv, int E, int ebits,
                                                          int32_t* __restrict__ blk_hist,
                                                          uint32_t* __restrict__ blk_err,
                                                          int32_t* __restrict__ local_rank) {
  extern __shared__ int32_t sm[];  // run[E] then wc[4][E]
  int32_t* run = sm;
  int32_t* wc = sm + E;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int i = tid; i < 5 * E; i += kCountThreads) sm[i] = 0;
  __syncthreads();
  int bad = 0;
  const int base = blockIdx.x * kCountChunk;
  for (int r = 0; r < kCountChunk / kCountThreads; r++) {
    const int p = base + r * kCountThreads + tid;
    int e = -1;
    if (p < Pv) {
      const int id = ids[p];
      if (id >= 0 && id < E) e = id;
      else if (id != -1) bad = 1;
    }
    // lanes of this wavefront that carry the same expert id
    uint64_t peers = __ballot(e >= 0);
    for (int b = 0; b < ebits; b++) {
      const int bit = (e >> b) & 1;
      const uint64_t m = __ballot(e >= 0 && bit);
      peers &= bit ? m : ~m;
    }
    int rank_w = 0;
    if (e >= 0) {
      rank_w = __popcll(peers & ((1ull << lane) - 1ull));
      if (rank_w == 0) wc[w * E + e] = __popcll(peers);
    }
    __syncthreads();
    if (e >= 0) {
      int rk = run[e] + rank_w;
      for (int w2 = 0; w2 < w; w2++) rk += wc[w2 * E + e];
      local_rank[p] = rk;
    }
    __syncthreads();
    for (int x = tid; x < E; x += kCountThreads) {
      int s = 0;
#pragma unroll
      for (int w2 = 0; w2 < kCountThreads / 64; w2++) {
        s += wc[w2 * E + x];
        wc[w2 * E + x] = 0;
      }
      run[x] += s;
    }
    __syncthreads();
  }
  for (int x = tid; x < E; x += kCountThreads) blk_hist[(size_t)blockIdx.x * E + x] = run[x];
  const int any_bad = __syncthreads_or(bad);
  if (tid == 0) blk_err[blockIdx.x] = any_bad ? TEMPO_DERR_BAD_ID : 0u;
}

__global__ __launch_bounds__(1024) void k_plan(int nblk, int E, int S, int M, int timing, int32_t* __restrict__ blk_hist,
                                               const uint32_t* __restrict__ blk_err,
                                               const int32_t* __restrict__ slot_expert,
                                               const uint32_t* __restrict__ slot_weight,
                                               const uint32_t* __restrict__ remote_weight,
                                               const int32_t* __restrict__ remote_replicas,
                                               int32_t* __restrict__ expert_counts, uint32_t* __restrict__ cum_counts,
                                               int32_t* __restrict__ slot_counts, int32_t* __restrict__ slot_offsets,
                                               int32_t* __restrict__ row_token, int32_t* __restrict__ slot_lo,
                                               uint64_t* __restrict__ t0, uint64_t* __restrict__ t1,
                                               uint32_t* __restrict__ hdr) {
  __shared__ int32_t s_n[kMaxE];
  __shared__ int32_t s_c[kMaxS];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ uint32_t s_err;
  const int tid = threadIdx.x, bd = blockDim.x;
  if (tid == 0) s_err = 0;
  __syncthreads();
  uint32_t eb = 0;
  for (int b = tid; b < nblk; b += bd) eb |= blk_err[b];
  if (eb) atomicOr(&s_err, eb);
  // n_e and the exclusive prefix of the block counts, in place
  for (int e = tid; e < E; e += bd) {
    int acc = 0;
    for (int b = 0; b < nblk; b++) {
      const size_t i = (size_t)b * E + e;
      const int v = blk_hist[i];
      blk_hist[i] = acc;
      acc += v;
    }
    s_n[e] = acc;
    expert_counts[e] = acc;
    if (cum_counts) cum_counts[e] = cum_counts[e] + (uint32_t)acc;
  }
  __syncthreads();
  // plan split: slot s is entry j of its expert; its ranks are
  // [floor(n C_{j-1} / W), floor(n C_j / W))
  for (int s = tid; s < S; s += bd) {
    const int e = slot_expert[s];
    int c = 0, lo = 0;
    if (e < 0 || e >= E) {
      atomicOr(&s_err, TEMPO_DERR_BAD_SLOT_EXPERT);
    } else {
      uint64_t W = 0, before = 0;
      int nloc = 0, nloc_before = 0;
      for (int s2 = 0; s2 < S; s2++)
        if (slot_expert[s2] == e) {
          W += slot_weight[s2];
          nloc++;
          if (s2 < s) {
            before += slot_weight[s2];
            nloc_before++;
          }
        }
      const int rr = remote_replicas[e];
      const bool has_remote = remote_weight[e] > 0u || rr > 0;
      if (has_remote) W += remote_weight[e];
      uint64_t mine = slot_weight[s];
      bool uniform = (W == 0);
      if (W >= (1ull << 32)) {
        uniform = true;
        atomicOr(&s_err, TEMPO_DERR_WEIGHT_OVERFLOW);
      }
      if (uniform) {
        W = (uint64_t)nloc + (has_remote && rr > 0 ? (uint64_t)rr : 0ull);
        before = (uint64_t)nloc_before;
        mine = 1;
      }
      const uint64_t n = (uint64_t)s_n[e];
      const uint64_t blo = n * before / W, bhi = n * (before + mine) / W;
      lo = (int)blo;
      c = (int)(bhi - blo);
    }
    s_c[s] = c;
    slot_lo[s] = lo;
    slot_counts[s] = c;
  }
  __syncthreads();
  if (tid == 0) {
    int off = 0, tiles = 0, G = 0, N = 0;
    for (int s = 0; s < S; s++) {
      s_off[s] = off;
      const int P = (s_c[s] + M - 1) / M * M;
      off += P;
      tiles += P / M;
      G += s_c[s] > 0;
      N += s_c[s];
    }
    s_off[S] = off;
    hdr[kHdrTiles] = (uint32_t)tiles;
    hdr[kHdrActive] = (uint32_t)G;
    hdr[kHdrPairs] = (uint32_t)N;
    hdr[kHdrLastErr] = s_err;
    hdr[kHdrSticky] = hdr[kHdrSticky] | s_err;
  }
  __syncthreads();
  for (int s = tid; s <= S; s += bd) slot_offsets[s] = s_off[s];
  for (int s = 0; s < S; s++) {
    const int c = s_c[s], P = s_off[s + 1] - s_off[s];
    for (int r = c + tid; r < P; r += bd) row_token[s_off[s] + r] = -1;
  }
  if (timing)
    for (int s = tid; s < S; s += bd) {
      t0[s] = ~0ull;
      t1[s] = 0ull;
    }
}

template <int ESIZE>
__global__ __launch_bounds__(256) void k_scatter(const int32_t* __restrict__ ids, int P, int Pv, int K, int E, int S,
                                                 int H, const int32_t* __restrict__ blk_prefix,
                                                 const int32_t* __restrict__ local_rank,
                                                 const int32_t* __restrict__ slot_expert,
                                                 const int32_t* __restrict__ slot_lo,
                                                 const int32_t* __restrict__ slot_counts,
                                                 const int32_t* __restrict__ slot_offsets,
                                                 const uint8_t* __restrict__ x, const float* __restrict__ x_scale,
                                                 int32_t* __restrict__ pair_row, int32_t* __restrict__ row_token,
                                                 uint8_t* __restrict__ x_perm, float* __restrict__ x_perm_scale) {
  __shared__ int32_t s_se[kMaxS], s_lo[kMaxS], s_c[kMaxS], s_off[kMaxS];
  __shared__ int32_t s_row[kScatterPairs], s_tok[kScatterPairs];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int s = tid; s < S; s += 256) {
    s_se[s] = slot_expert[s];
    s_lo[s] = slot_lo[s];
    s_c[s] = slot_counts[s];
    s_off[s] = slot_offsets[s];
  }
  __syncthreads();
  if (tid < kScatterPairs) {
    const int p = blockIdx.x * kScatterPairs + tid;
    int row = -1;
    if (p < P) {
      if (p < Pv) {
        const int e = ids[p];
        if (e >= 0 && e < E) {
          const int r = blk_prefix[(size_t)(p / kCountChunk) * E + e] + local_rank[p];
          for (int s = 0; s < S; s++)
            if (s_se[s] == e && r >= s_lo[s] && r < s_lo[s] + s_c[s]) {
              row = s_off[s] + (r - s_lo[s]);
              break;
            }
        }
      }
      pair_row[p] = row;
      if (row >= 0) row_token[row] = p / K;
    }
    s_row[tid] = row;
    s_tok[tid] = p / K;
  }
  __syncthreads();
  // copy the activation rows: one wavefront per placed pair
  const int nch = H * ESIZE / 16;
  for (int j = w; j < kScatterPairs; j += 4) {
    const int row = s_row[j];
    if (row < 0) continue;
    const uint4* __restrict__ src = reinterpret_cast<const uint4*>(x + (size_t)s_tok[j] * H * ESIZE);
    uint4* __restrict__ dst = reinterpret_cast<uint4*>(x_perm + (size_t)row * H * ESIZE);
    constexpr int U = 8;
    for (int i0 = lane; i0 < nch; i0 += 64 * U) {
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; u++)
        if (i0 + u * 64 < nch) v[u] = src[i0 + u * 64];
#pragma unroll
      for (int u = 0; u < U; u++)
        if (i0 + u * 64 < nch) dst[i0 + u * 64] = v[u];
    }
    if (ESIZE == 1) {
      const int ns = H / 128;
      for (int i = lane; i < ns; i += 64) x_perm_scale[(size_t)row * ns + i] = x_scale[(size_t)s_tok[j] * ns + i];
    }
  }
}

}  // namespace

hipError_t launch_dispatch(const tempo_moe_shape& s, const tempo_plan& plan, const int32_t* topk_ids, const void* x,
                           const float* x_scale, const tempo_dispatch_out& out, char* ws, const Layout& L,
                           bool timing, hipStream_t st) {
  const int P = s.T * s.K, Pv = s.T_valid * s.K;
  int ebits = 0;
  while ((1 << ebits) < s.E) ebits++;
  int32_t* blk_hist = reinterpret_cast<int32_t*>(ws + L.blk_hist);
  uint32_t* blk_err = reinterpret_cast<uint32_t*>(ws + L.blk_err);
  int32_t* local_rank = reinterpret_cast<int32_t*>(ws + L.local_rank);
  int32_t* slot_lo = reinterpret_cast<int32_t*>(ws + L.slot_lo);
  uint64_t* t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  uint64_t* t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  uint32_t* hdr = reinterpret_cast<uint32_t*>(ws + L.header);

  hipLaunchKernelGGL(k_count, dim3(L.nblk), dim3(kCountThreads), 5 * s.E * sizeof(int32_t), st, topk_ids, Pv, s.E,
                     ebits, blk_hist, blk_err, local_rank);
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(1024), 0, st, L.nblk, s.E, s.S, s.m_tile, timing ? 1 : 0, blk_hist,
                     blk_err, plan.slot_expert, plan.slot_weight, plan.remote_weight, plan.remote_replicas,
                     out.expert_counts, out.cum_counts, out.slot_counts, out.slot_offsets, out.row_token, slot_lo,
                     t0, t1, hdr);
  const int nb = ceil_div(P, kScatterPairs);
  if (s.dtype == TEMPO_BF16)
    hipLaunchKernelGGL(k_scatter<2>, dim3(nb), dim3(256), 0, st, topk_ids, P, Pv, s.K, s.E, s.S, s.H, blk_hist,
                       local_rank, plan.slot_expert, slot_lo, out.slot_counts, out.slot_offsets,
                       static_cast<const uint8_t*>(x), x_scale, out.pair_row, out.row_token,
                       static_cast<uint8_t*>(out.x_perm), out.x_perm_scale);
  else
    hipLaunchKernelGGL(k_scatter<1>, dim3(nb), dim3(256), 0, st, topk_ids, P, Pv, s.K, s.E, s.S, s.H, blk_hist,
                       local_rank, plan.slot_expert, slot_lo, out.slot_counts, out.slot_offsets,
                       static_cast<const uint8_t*>(x), x_scale, out.pair_row, out.row_token,
                       static_cast<uint8_t*>(out.x_perm), out.x_perm_scale);
  return hipGetLastError();
}

}  // namespace tempo
