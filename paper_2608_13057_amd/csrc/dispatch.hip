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
// Ranks.  The rank of a pair within its expert is the number of valid pairs
// of the same expert with a smaller index p = t*K + k.  Pairs are processed
// in rounds of one pair per thread; within a wavefront, lanes holding the same
// expert are found with one ballot per bit of the expert id and the lane's
// rank is the popcount of those lanes below it; per-wavefront counts in LDS
// give the offset of earlier wavefronts and a running count the offset of
// earlier rounds.  No atomics decide positions.
//
// Two paths, both free of zero-initialised memory:
//   small batches (T*K <= 16384): k_dispatch_fused -- one launch; every
//     block re-derives the counts and the plan from all ids (cheap at this
//     size) and places and gathers its own 64 pairs, so no block waits for
//     another.
//   large batches: k_count (blocks of 1024 pairs, per-block histograms and
//     in-block ranks) -> k_plan (one block: per-expert scan over blocks, split,
//     offsets) -> k_scatter (index outputs) -> k_gather (one wavefront per
//     pair).
#include "internal.h"

namespace tempo {
namespace {

constexpr int kSmallMaxPairs = 16384;

// ---------------------------------------------------------------------------
// shared pieces
// ---------------------------------------------------------------------------

// Rank one round of pairs (one per thread) within (expert); wc is
// [NW][E] of zeros on entry and is zero again on exit; run [E] holds the
// counts of earlier rounds and is advanced.  Returns the rank (or -1).
template <int NW>
__device__ __forceinline__ int rank_round(int e, int E, int ebits, int32_t* run, int32_t* wc) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
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
  int rk = -1;
  if (e >= 0) {
    rk = run[e] + rank_w;
    for (int w2 = 0; w2 < w; w2++) rk += wc[w2 * E + e];
  }
  __syncthreads();
  for (int x = tid; x < E; x += NW * 64) {
    int s = 0;
#pragma unroll
    for (int w2 = 0; w2 < NW; w2++) {
      s += wc[w2 * E + x];
      wc[w2 * E + x] = 0;
    }
    run[x] += s;
  }
  __syncthreads();
  return rk;
}

// Exclusive scan of v over the block (blockDim = 64 * NW <= 1024); one value
// per thread.  Returns the thread's exclusive prefix; *total gets the sum.
template <int NW>
__device__ __forceinline__ int block_exclusive_scan(int v, int* s_tmp, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_tmp[w] = x;
  __syncthreads();
  if (w == 0) {
    int t = lane < NW ? s_tmp[lane] : 0;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(t, d);
      if (lane >= d) t += y;
    }
    if (lane < NW) s_tmp[32 + lane] = t;  // inclusive wave totals
  }
  __syncthreads();
  const int before = (w == 0 ? 0 : s_tmp[32 + w - 1]);
  *total = s_tmp[32 + NW - 1];
  __syncthreads();
  return before + x - v;
}

// Slot tables in LDS (filled by plan_slots).
struct SlotLds {
  int32_t se[kMaxS];   // expert of slot
  int32_t lo[kMaxS];   // first rank (within the expert) taken by the slot
  int32_t c[kMaxS];    // c_s
  int32_t off[kMaxS + 1];
};

// Plan split, padded sizes, offsets, padding-row markers and header.  n_e is
// read from n (LDS or global); runs on one block of NW wavefronts with
// S <= 64 * NW.  WRITE = false computes the LDS tables only.
template <int NW, bool WRITE>
__device__ void plan_slots(const int32_t* n, int E, int S, int M, const int32_t* __restrict__ slot_expert,
                           const uint32_t* __restrict__ slot_weight, const uint32_t* __restrict__ remote_weight,
                           const int32_t* __restrict__ remote_replicas, int32_t* __restrict__ slot_counts,
                           int32_t* __restrict__ slot_offsets, int32_t* __restrict__ row_token,
                           int32_t* __restrict__ slot_lo_out, uint32_t* __restrict__ hdr, SlotLds& L, uint32_t* s_err,
                           uint32_t* s_w, int* s_tmp, int timing, uint64_t* __restrict__ t0,
                           uint64_t* __restrict__ t1) {
  const int tid = threadIdx.x, bd = NW * 64;
  for (int s = tid; s < S; s += bd) {
    L.se[s] = slot_expert[s];
    s_w[s] = slot_weight[s];
  }
  __syncthreads();
  int c = 0, P = 0;
  if (tid < S) {
    const int s = tid, e = L.se[s];
    int lo = 0;
    if (e < 0 || e >= E) {
      atomicOr(s_err, TEMPO_DERR_BAD_SLOT_EXPERT);
    } else {
      uint64_t W = 0, before = 0;
      int nloc = 0, nloc_before = 0;
      for (int s2 = 0; s2 < S; s2++)
        if (L.se[s2] == e) {
          W += s_w[s2];
          nloc++;
          if (s2 < s) {
            before += s_w[s2];
            nloc_before++;
          }
        }
      const int rr = remote_replicas[e];  // LDS or global
      const uint32_t rw = remote_weight[e];
      const bool has_remote = rw > 0u || rr > 0;
      if (has_remote) W += rw;
      uint64_t mine = s_w[s];
      bool uniform = (W == 0);
      if (W >= (1ull << 32)) {
        uniform = true;
        atomicOr(s_err, TEMPO_DERR_WEIGHT_OVERFLOW);
      }
      if (uniform) {
        W = (uint64_t)nloc + (has_remote && rr > 0 ? (uint64_t)rr : 0ull);
        before = (uint64_t)nloc_before;
        mine = 1;
      }
      const uint64_t ne = (uint64_t)n[e];
      const uint64_t blo = ne * before / W, bhi = ne * (before + mine) / W;
      lo = (int)blo;
      c = (int)(bhi - blo);
    }
    L.c[s] = c;
    L.lo[s] = lo;
    if (WRITE) {
      slot_counts[s] = c;
      if (slot_lo_out) slot_lo_out[s] = lo;
    }
    P = (c + M - 1) / M * M;
  }
  int total = 0;
  const int off = block_exclusive_scan<NW>(P, s_tmp, &total);
  if (tid < S) L.off[tid] = off;
  if (tid == 0) L.off[S] = total;
  if (!WRITE) {
    __syncthreads();
    return;
  }
  // tiles, G, N
  const int tiles = block_exclusive_scan<NW>(P / M, s_tmp, &total), ntiles = total;
  (void)tiles;
  block_exclusive_scan<NW>(c > 0 ? 1 : 0, s_tmp, &total);
  const int G = total;
  block_exclusive_scan<NW>(c, s_tmp, &total);
  const int N = total;
  if (tid == 0) {
    hdr[kHdrTiles] = (uint32_t)ntiles;
    hdr[kHdrActive] = (uint32_t)G;
    hdr[kHdrPairs] = (uint32_t)N;
    const uint32_t e = *s_err;
    hdr[kHdrLastErr] = e;
    hdr[kHdrSticky] = hdr[kHdrSticky] | e;
  }
  __syncthreads();
  for (int s = tid; s <= S; s += bd) slot_offsets[s] = L.off[s];
  // padding rows of every slot
  for (int s = 0; s < S; s++) {
    const int cs = L.c[s], Ps = L.off[s + 1] - L.off[s];
    for (int r = cs + tid; r < Ps; r += bd) row_token[L.off[s] + r] = -1;
  }
  if (timing)
    for (int s = tid; s < S; s += bd) {
      t0[s] = ~0ull;
      t1[s] = 0ull;
    }
}

// Row of pair p with expert e and rank r (or -1 when the rank falls on the
// remote share).
__device__ __forceinline__ int row_of(const SlotLds& L, int S, int e, int r) {
  for (int s = 0; s < S; s++)
    if (L.se[s] == e && r >= L.lo[s] && r < L.lo[s] + L.c[s]) return L.off[s] + (r - L.lo[s]);
  return -1;
}

// ---------------------------------------------------------------------------
// small batches: one launch, no grid-wide synchronisation
// ---------------------------------------------------------------------------

// Block b owns pairs [64 b, 64 b + 64).  Every block histograms all valid ids
// (from L2; 16K pairs at most) -- the total gives n_e, the part before its
// chunk the rank offset of its pairs -- then recomputes the small plan split
// and slot offsets itself, places and gathers its own pairs.  Block 0 alone
// writes the per-expert / per-slot outputs and the header.
constexpr int kFusedChunk = 64;

template <int ESIZE>
__global__ __launch_bounds__(256) void k_dispatch_fused(
    const int32_t* __restrict__ ids, int P, int Pv, int K, int E, int ebits, int S, int M, int H,
    const int32_t* __restrict__ slot_expert, const uint32_t* __restrict__ slot_weight,
    const uint32_t* __restrict__ remote_weight, const int32_t* __restrict__ remote_replicas,
    int32_t* __restrict__ expert_counts, uint32_t* __restrict__ cum_counts, int32_t* __restrict__ slot_counts,
    int32_t* __restrict__ slot_offsets, int32_t* __restrict__ row_token, int32_t* __restrict__ pair_row,
    const uint8_t* __restrict__ x, const float* __restrict__ x_scale, uint8_t* __restrict__ x_perm,
    float* __restrict__ x_perm_scale, int row_cap, uint32_t* __restrict__ hdr, int timing,
    uint64_t* __restrict__ t0, uint64_t* __restrict__ t1) {
  constexpr int NW = 4;
  constexpr int IDS_PER_THREAD = kSmallMaxPairs / 256;  // every id of the batch, 64 per thread at most
  constexpr int BATCH = 16;                              // id loads in flight per thread
  extern __shared__ int32_t dyn[];  // n_all[E], n_before[E], first_slot[E], rem_w[E], rem_r[E]
  int32_t* n_all = dyn;
  int32_t* n_before = dyn + E;
  int32_t* first_slot = dyn + 2 * E;
  uint32_t* rem_w = reinterpret_cast<uint32_t*>(dyn + 3 * E);
  int32_t* rem_r = dyn + 4 * E;
  __shared__ SlotLds L;
  __shared__ uint32_t s_w[kMaxS];
  __shared__ int32_t s_next[kMaxS];
  __shared__ int s_tmp[64];
  __shared__ uint32_t s_err;
  __shared__ int32_t s_rank[kFusedChunk];
  __shared__ int32_t s_prow[kFusedChunk], s_ptok[kFusedChunk];
  __shared__ int s_nplaced;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int base = blockIdx.x * kFusedChunk;

  // every global input this block needs is requested before anything waits
  for (int i = tid; i < E; i += 256) {
    rem_w[i] = remote_weight[i];
    rem_r[i] = remote_replicas[i];
    n_all[i] = 0;
    n_before[i] = 0;
    first_slot[i] = 0x7fffffff;
  }
  if (tid == 0) s_err = 0;

  // histogram of all valid ids; wavefronts aggregate equal ids with ballots
  int bad = 0;
  const int nq = (P + 255) / 256;
  for (int b0 = 0; b0 < nq; b0 += BATCH) {
    int idv[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; u++) {
      const int p = (b0 + u) * 256 + tid;
      idv[u] = (b0 + u < nq && p < Pv) ? ids[p] : -1;
    }
    __syncthreads();  // LDS initialisation done (first batch) / keeps batches in step
#pragma unroll
    for (int u = 0; u < BATCH; u++) {
      if (b0 + u >= nq) break;
      const int q0 = (b0 + u) * 256;
      int e = -1;
      const int id = idv[u];
      if (id >= 0 && id < E) e = id;
      else if (id != -1) bad = 1;
      uint64_t peers = __ballot(e >= 0);
      for (int b = 0; b < ebits; b++) {
        const int bit = (e >> b) & 1;
        const uint64_t m = __ballot(e >= 0 && bit);
        peers &= bit ? m : ~m;
      }
      // a wavefront's 64 pairs lie wholly before the block's chunk, on it, or after it
      const int wbase = q0 + w * 64;
      if (e >= 0) {
        const int below = __popcll(peers & ((1ull << lane) - 1ull));
        if (below == 0) {
          atomicAdd(&n_all[e], __popcll(peers));
          if (wbase < base) atomicAdd(&n_before[e], __popcll(peers));
        }
        if (wbase == base) s_rank[lane] = below;  // in-chunk rank of an own pair
      }
    }
  }
  (void)IDS_PER_THREAD;
  // own pairs' ids (L2 hits: just read above)
  int own_e = -1;
  if (tid < kFusedChunk && base + tid < Pv) own_e = ids[base + tid];
  const int any_bad = __syncthreads_or(bad);
  if (blockIdx.x == 0) {
    if (tid == 0 && any_bad) s_err = TEMPO_DERR_BAD_ID;
    for (int e = tid; e < E; e += 256) {
      expert_counts[e] = n_all[e];
      if (cum_counts) cum_counts[e] = cum_counts[e] + (uint32_t)n_all[e];
    }
  }
  // plan split and offsets (every block; outputs from block 0 only)
  if (blockIdx.x == 0) {
    plan_slots<NW, true>(n_all, E, S, M, slot_expert, slot_weight, rem_w, rem_r, slot_counts, slot_offsets,
                         row_token, nullptr, hdr, L, &s_err, s_w, s_tmp, timing, t0, t1);
  } else {
    plan_slots<NW, false>(n_all, E, S, M, slot_expert, slot_weight, rem_w, rem_r, slot_counts, slot_offsets,
                          row_token, nullptr, hdr, L, &s_err, s_w, s_tmp, timing, t0, t1);
  }
  // per-expert list of local slots in ascending order: first_slot[e], s_next[s]
  for (int s = tid; s < S; s += 256) {
    const int e = L.se[s];
    int nx = -1;
    if (e >= 0 && e < E) {
      atomicMin(&first_slot[e], s);
      for (int s2 = s + 1; s2 < S; s2++)
        if (L.se[s2] == e) {
          nx = s2;
          break;
        }
    }
    s_next[s] = nx;
  }
  __syncthreads();
  // own pairs: rank -> slot -> row
  if (tid < kFusedChunk) {
    const int p = base + tid;
    int row = -1;
    const int e = own_e;
    if (e >= 0 && e < E) {
      const int r = n_before[e] + s_rank[tid];
      for (int s = first_slot[e]; s >= 0 && s < S; s = s_next[s])
        if (r >= L.lo[s] && r < L.lo[s] + L.c[s]) {
          row = L.off[s] + (r - L.lo[s]);
          break;
        }
    }
    if (p < P) {
      pair_row[p] = row;
      if (row >= 0) row_token[row] = p / K;
    }
    const uint64_t m = __ballot(row >= 0);
    if (row >= 0) {
      const int pos = __popcll(m & ((1ull << lane) - 1ull));
      s_prow[pos] = row;
      s_ptok[pos] = p / K;
    }
    if (lane == 0) s_nplaced = __popcll(m);
  }
  __syncthreads();
  // gather the placed rows: one wavefront per row, every load of a row in flight
  const int R = s_nplaced;
  const int nch = H * ESIZE / 16;
  for (int j = w; j < R; j += NW) {
    const uint4* __restrict__ src = reinterpret_cast<const uint4*>(x) + (size_t)s_ptok[j] * nch;
    uint4* __restrict__ dst = reinterpret_cast<uint4*>(x_perm) + (size_t)s_prow[j] * nch;
    constexpr int U = 8;
    for (int c0 = lane; c0 < nch; c0 += 64 * U) {
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; u++) v[u] = src[min(c0 + u * 64, nch - 1)];
#pragma unroll
      for (int u = 0; u < U; u++)
        if (c0 + u * 64 < nch) dst[c0 + u * 64] = v[u];
    }
    if (ESIZE == 1) {  // scales are stored block-major: [H/128][row_cap]
      const int ns = H / 128;
      for (int i = lane; i < ns; i += 64)
        x_perm_scale[(size_t)i * row_cap + s_prow[j]] = x_scale[(size_t)s_ptok[j] * ns + i];
    }
  }
}

// ---------------------------------------------------------------------------
// large batches
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kCountThreads) void k_count(const int32_t* __restrict__ ids, int Pv, int E, int ebits,
                                                          int32_t* __restrict__ blk_hist,
                                                          uint32_t* __restrict__ blk_err,
                                                          int32_t* __restrict__ local_rank) {
  constexpr int NW = kCountThreads / 64;
  extern __shared__ int32_t sm[];  // run[E] then wc[NW][E]
  int32_t* run = sm;
  int32_t* wc = sm + E;
  const int tid = threadIdx.x;
  for (int i = tid; i < (NW + 1) * E; i += kCountThreads) sm[i] = 0;
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
    const int rk = rank_round<NW>(e, E, ebits, run, wc);
    if (e >= 0) local_rank[p] = rk;
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
  constexpr int NW = 16;
  __shared__ int32_t s_n[kMaxE];
  __shared__ SlotLds L;
  __shared__ uint32_t s_w[kMaxS];
  __shared__ int s_tmp[64];
  __shared__ uint32_t s_err;
  const int tid = threadIdx.x;
  if (tid == 0) s_err = 0;
  __syncthreads();
  uint32_t eb = 0;
  for (int b = tid; b < nblk; b += 1024) eb |= blk_err[b];
  if (eb) atomicOr(&s_err, eb);
  // n_e and the exclusive prefix of the block counts, in place; the loads of
  // one expert's column are independent and issued back to back
  for (int e = tid; e < E; e += 1024) {
    int acc = 0;
    int b = 0;
    for (; b + 8 <= nblk; b += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; u++) v[u] = blk_hist[(size_t)(b + u) * E + e];
#pragma unroll
      for (int u = 0; u < 8; u++) {
        blk_hist[(size_t)(b + u) * E + e] = acc;
        acc += v[u];
      }
    }
    for (; b < nblk; b++) {
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
  plan_slots<NW, true>(s_n, E, S, M, slot_expert, slot_weight, remote_weight, remote_replicas, slot_counts, slot_offsets,
                 row_token, slot_lo, hdr, L, &s_err, s_w, s_tmp, timing, t0, t1);
}

__global__ __launch_bounds__(256) void k_scatter(const int32_t* __restrict__ ids, int P, int Pv, int K, int E, int S,
                                                 const int32_t* __restrict__ blk_prefix,
                                                 const int32_t* __restrict__ local_rank,
                                                 const int32_t* __restrict__ slot_expert,
                                                 const int32_t* __restrict__ slot_lo,
                                                 const int32_t* __restrict__ slot_counts,
                                                 const int32_t* __restrict__ slot_offsets,
                                                 int32_t* __restrict__ pair_row, int32_t* __restrict__ row_token) {
  __shared__ SlotLds L;
  const int tid = threadIdx.x;
  for (int s = tid; s < S; s += 256) {
    L.se[s] = slot_expert[s];
    L.lo[s] = slot_lo[s];
    L.c[s] = slot_counts[s];
    L.off[s] = slot_offsets[s];
  }
  __syncthreads();
  const int p = blockIdx.x * 256 + tid;
  if (p >= P) return;
  int row = -1;
  if (p < Pv) {
    const int e = ids[p];
    if (e >= 0 && e < E) row = row_of(L, S, e, blk_prefix[(size_t)(p / kCountChunk) * E + e] + local_rank[p]);
  }
  pair_row[p] = row;
  if (row >= 0) row_token[row] = p / K;
}

// ---------------------------------------------------------------------------
// row copy: one wavefront per pair
// ---------------------------------------------------------------------------

template <int ESIZE>
__global__ __launch_bounds__(256) void k_gather(const int32_t* __restrict__ pair_row, int P, int K, int H,
                                                const uint8_t* __restrict__ x, const float* __restrict__ x_scale,
                                                uint8_t* __restrict__ x_perm, float* __restrict__ x_perm_scale,
                                                int row_cap) {
  const int lane = threadIdx.x & 63;
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= P) return;
  const int row = pair_row[p];
  if (row < 0) return;
  const int t = p / K;
  const int nch = H * ESIZE / 16;
  const uint4* __restrict__ src = reinterpret_cast<const uint4*>(x + (size_t)t * H * ESIZE);
  uint4* __restrict__ dst = reinterpret_cast<uint4*>(x_perm + (size_t)row * H * ESIZE);
  constexpr int U = 8;
  for (int i0 = lane; i0 < nch; i0 += 64 * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; u++) v[u] = src[min(i0 + u * 64, nch - 1)];
#pragma unroll
    for (int u = 0; u < U; u++)
      if (i0 + u * 64 < nch) dst[i0 + u * 64] = v[u];
  }
  if (ESIZE == 1) {  // scales are stored block-major: [H/128][row_cap]
    const int ns = H / 128;
    for (int i = lane; i < ns; i += 64) x_perm_scale[(size_t)i * row_cap + row] = x_scale[(size_t)t * ns + i];
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

  if (P <= kSmallMaxPairs && s.S <= 256) {
    const size_t lds = (size_t)5 * s.E * sizeof(int32_t);
    const int nb = ceil_div(P, kFusedChunk);
    if (s.dtype == TEMPO_BF16)
      hipLaunchKernelGGL(k_dispatch_fused<2>, dim3(nb), dim3(256), lds, st, topk_ids, P, Pv, s.K, s.E, ebits, s.S,
                         s.m_tile, s.H, plan.slot_expert, plan.slot_weight, plan.remote_weight, plan.remote_replicas,
                         out.expert_counts, out.cum_counts, out.slot_counts, out.slot_offsets, out.row_token,
                         out.pair_row, static_cast<const uint8_t*>(x), x_scale, static_cast<uint8_t*>(out.x_perm),
                         out.x_perm_scale, L.row_cap, hdr, timing ? 1 : 0, t0, t1);
    else
      hipLaunchKernelGGL(k_dispatch_fused<1>, dim3(nb), dim3(256), lds, st, topk_ids, P, Pv, s.K, s.E, ebits, s.S,
                         s.m_tile, s.H, plan.slot_expert, plan.slot_weight, plan.remote_weight, plan.remote_replicas,
                         out.expert_counts, out.cum_counts, out.slot_counts, out.slot_offsets, out.row_token,
                         out.pair_row, static_cast<const uint8_t*>(x), x_scale, static_cast<uint8_t*>(out.x_perm),
                         out.x_perm_scale, L.row_cap, hdr, timing ? 1 : 0, t0, t1);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_count, dim3(L.nblk), dim3(kCountThreads), (kCountThreads / 64 + 1) * s.E * sizeof(int32_t), st,
                     topk_ids, Pv, s.E, ebits, blk_hist, blk_err, local_rank);
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(1024), 0, st, L.nblk, s.E, s.S, s.m_tile, timing ? 1 : 0, blk_hist, blk_err,
                     plan.slot_expert, plan.slot_weight, plan.remote_weight, plan.remote_replicas, out.expert_counts,
                     out.cum_counts, out.slot_counts, out.slot_offsets, out.row_token, slot_lo, t0, t1, hdr);
  hipLaunchKernelGGL(k_scatter, dim3(ceil_div(P, 256)), dim3(256), 0, st, topk_ids, P, Pv, s.K, s.E, s.S, blk_hist,
                     local_rank, plan.slot_expert, slot_lo, out.slot_counts, out.slot_offsets, out.pair_row,
                     out.row_token);
  const int nb = ceil_div(P, 4);
  if (s.dtype == TEMPO_BF16)
    hipLaunchKernelGGL(k_gather<2>, dim3(nb), dim3(256), 0, st, out.pair_row, P, s.K, s.H,
                       static_cast<const uint8_t*>(x), x_scale, static_cast<uint8_t*>(out.x_perm), out.x_perm_scale,
                       L.row_cap);
  else
    hipLaunchKernelGGL(k_gather<1>, dim3(nb), dim3(256), 0, st, out.pair_row, P, s.K, s.H,
                       static_cast<const uint8_t*>(x), x_scale, static_cast<uint8_t*>(out.x_perm), out.x_perm_scale,
                       L.row_cap);
  return hipGetLastError();
}

}  // namespace tempo
