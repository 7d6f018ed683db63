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
// One launch for decode-sized batches whose rows (and fp8 scales) stage 2
// reads from the token rows (k_dispatch_small: one workgroup does all of it);
// otherwise two launches
// (three for large batches, see k_scan); no block ever waits for or signals
// another (device-scope fences write back L2 on this multi-XCD chip and cost
// more than the work):
//   k_count  blocks of 256 pairs: in-block stable ranks and per-block expert
//            histograms.
//   k_place  blocks of 64 pairs (256 for large batches): each sums the block
//            histograms (n_e and the prefix of its own count block; read
//            from k_scan's output for large batches), recomputes the small
//            plan -- the split of every expert over its slots, padded
//            sizes, offsets, per-expert slot lists -- in LDS (block 0 also
//            writes the
//            per-expert / per-slot outputs and the header), then maps its
//            pairs rank -> slot -> row and writes the index outputs and
//            copies the rows, one wavefront per row with every load in
//            flight (the whole forward skips what stage 2 reads through
//            row_token directly: the rows for decode-sized batches, rows and
//            fp8 scales for the large-tile kernels).
// Global loads are issued before the values are needed: at one wavefront per
// SIMD every exposed memory latency (~0.3-0.5 us) adds up.
#include <algorithm>

#include "internal.h"

namespace tempo {
namespace {

// pairs per k_place block: 64 for decode-sized batches (more blocks in
// flight, each with a short critical path), 256 when k_scan runs (a quarter
// of the blocks recomputing the plan)
constexpr int kPlaceChunk = 64;
constexpr int kPlaceChunkLarge = 256;
constexpr int kScanBlocks = 32;  // above this many count blocks, k_scan computes the prefixes once
// single-workgroup stage 1: 16 wavefronts, at most kSmallRounds pairs per
// thread (batches up to 8192 pairs), per-wavefront masks and counts of up to
// 256 experts in LDS
constexpr int kSmallWaves = 16;
constexpr int kSmallRounds = 8;
constexpr int kSmallMaxE = 256;
constexpr int kSmallScalesMaxP = 4096;  // pairs up to which fp8 batches with permuted scales use it

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

// Tile-aware split (Sec. 2.2 after Eq. 2: partial splits snapped to tile
// boundaries): a boundary other than n_e moves to the nearest multiple of M
// (halves up), capped at n_e.
__device__ __forceinline__ uint64_t snap_boundary(uint64_t b, uint64_t n, int M) {
  if (b == n) return b;
  const uint64_t q = (b + (uint64_t)(M / 2)) / (uint64_t)M * (uint64_t)M;
  return q < n ? q : n;
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
__device__ __forceinline__ void plan_slots(const int32_t* n, int E, int S, int M, int snap, const int32_t* __restrict__ slot_expert,
                           const uint32_t* __restrict__ slot_weight, const uint32_t* __restrict__ remote_weight,
                           const int32_t* __restrict__ remote_replicas, int32_t* __restrict__ slot_counts,
                           int32_t* __restrict__ slot_offsets, int32_t* __restrict__ row_token,
                           uint32_t* __restrict__ hdr, SlotLds& L, uint32_t* s_err,
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
      uint64_t blo = ne * before / W, bhi = ne * (before + mine) / W;
      if (snap) {
        blo = snap_boundary(blo, ne, M);
        bhi = snap_boundary(bhi, ne, M);
      }
      lo = (int)blo;
      c = (int)(bhi - blo);
    }
    L.c[s] = c;
    L.lo[s] = lo;
    if (WRITE) slot_counts[s] = c;
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

// Plan for S <= 64 in one wavefront (lane s = slot s): the same split as
// plan_slots without block barriers -- per-expert weight sums and the
// slot-order position come from a readlane loop over the slots, offsets and
// totals from wavefront scans.  Fills the LDS slot tables (se, lo, c, off and
// the per-expert slot lists first[E] / next[S]; first must hold INT_MAX on
// entry) and, when write is set, the global per-slot outputs and the header
// (the caller marks the padding rows, with the whole block); the sticky
// error word is read from sticky_in (the header itself, or a copy the
// caller loaded early).
__device__ __forceinline__ void plan_slots_wave(const int32_t* n, int E, int S, int M, int snap, const int32_t* __restrict__ slot_expert,
                                const uint32_t* __restrict__ slot_weight, const uint32_t* __restrict__ remote_weight,
                                const int32_t* __restrict__ remote_replicas, SlotLds& L, int32_t* first,
                                int32_t* next, bool write, int32_t* __restrict__ slot_counts,
                                int32_t* __restrict__ slot_offsets, int32_t* __restrict__ row_token,
                                uint32_t* __restrict__ hdr, const uint32_t* sticky_in, uint32_t err_in, int timing,
                                uint64_t* __restrict__ t0, uint64_t* __restrict__ t1) {
  const int lane = threadIdx.x & 63;
  const bool live = lane < S;
  const int e = live ? slot_expert[lane] : -1;
  const uint32_t w = live ? slot_weight[lane] : 0u;
  const bool ok = live && e >= 0 && e < E;
  int rr = 0;
  uint32_t rw = 0;
  int ne = 0;
  if (ok) {
    rr = remote_replicas[e];
    rw = remote_weight[e];
    ne = n[e];
  }
  uint32_t err = err_in;
  if (__ballot(live && !ok)) err |= TEMPO_DERR_BAD_SLOT_EXPERT;
  uint64_t Wloc = 0, before = 0;
  int nloc = 0, nbefore = 0, nx = -1;
  for (int l = 0; l < S; l++) {
    const int el = __builtin_amdgcn_readlane(e, l);
    const uint32_t wl = (uint32_t)__builtin_amdgcn_readlane((int)w, l);
    if (ok && el == e) {
      Wloc += wl;
      nloc++;
      if (l < lane) {
        before += wl;
        nbefore++;
      }
      if (l > lane && nx < 0) nx = l;
    }
  }
  int c = 0, lo = 0;
  const bool has_remote = rw > 0u || rr > 0;
  const uint64_t Wtot = Wloc + (has_remote ? rw : 0u);
  if (ok) {
    uint64_t W = Wtot;
    uint64_t mine = w;
    const bool uniform = (W == 0) || (W >= (1ull << 32));
    if (uniform) {
      W = (uint64_t)nloc + (has_remote && rr > 0 ? (uint64_t)rr : 0ull);
      before = (uint64_t)nbefore;
      mine = 1;
    }
    uint64_t blo, bhi;
    if (ne < (1 << 20)) {
      // floor(a / W) in fp64 is exact here: a = n_e C < 2^52 is exact, the
      // quotient is below 2^20 so its spacing (<= 2^-33) is finer than the
      // distance 1/W of a non-integer a / W to the next integer
      const double dW = (double)W;
      blo = (uint64_t)floor((double)((uint64_t)ne * before) / dW);
      bhi = (uint64_t)floor((double)((uint64_t)ne * (before + mine)) / dW);
    } else {
      blo = (uint64_t)ne * before / W;
      bhi = (uint64_t)ne * (before + mine) / W;
    }
    if (snap) {
      blo = snap_boundary(blo, (uint64_t)ne, M);
      bhi = snap_boundary(bhi, (uint64_t)ne, M);
    }
    lo = (int)blo;
    c = (int)(bhi - blo);
  }
  if (__ballot(ok && Wtot >= (1ull << 32))) err |= TEMPO_DERR_WEIGHT_OVERFLOW;
  const int P = (c + M - 1) / M * M;
  int incl = P, tiles = P / M, g = c > 0, pairs = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(incl, d);
    if (lane >= d) incl += y;
    tiles += __shfl_xor(tiles, d);
    g += __shfl_xor(g, d);
    pairs += __shfl_xor(pairs, d);
  }
  const int off = incl - P;
  const int total = __shfl(incl, 63);
  if (live) {
    L.se[lane] = e;
    L.lo[lane] = lo;
    L.c[lane] = c;
    L.off[lane] = off;
    next[lane] = ok ? nx : -1;
    if (ok && nbefore == 0) first[e] = lane;
  }
  if (lane == 0) L.off[S] = total;
  if (!write) return;
  if (live) {
    slot_counts[lane] = c;
    slot_offsets[lane] = off;
    if (timing) {
      t0[lane] = ~0ull;
      t1[lane] = 0ull;
    }
  }
  if (lane == 0) {
    slot_offsets[S] = total;
    hdr[kHdrTiles] = (uint32_t)tiles;
    hdr[kHdrActive] = (uint32_t)g;
    hdr[kHdrPairs] = (uint32_t)pairs;
    hdr[kHdrLastErr] = err;
    hdr[kHdrSticky] = *sticky_in | err;
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
// launch 1: in-block ranks and block histograms
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kCountThreads) void k_count(const int32_t* __restrict__ ids, int Pv, int E, int ebits,
                                                          int32_t* __restrict__ blk_hist,
                                                          uint32_t* __restrict__ blk_err,
                                                          int32_t* __restrict__ local_rank) {
  constexpr int NW = kCountThreads / 64;
  extern __shared__ int32_t sm[];  // run[E], wc[NW][E]
  int32_t* run = sm;
  int32_t* wc = sm + E;
  const int tid = threadIdx.x;
  const int p = blockIdx.x * kCountThreads + tid;
  const int id = p < Pv ? ids[p] : -1;
  for (int i = tid; i < (NW + 1) * E; i += kCountThreads) sm[i] = 0;
  __syncthreads();
  int e = -1, bad = 0;
  if (id >= 0 && id < E) e = id;
  else if (id != -1) bad = 1;
  const int rk = rank_round<NW>(e, E, ebits, run, wc);
  if (e >= 0) local_rank[p] = rk;
  for (int x = tid; x < E; x += kCountThreads) blk_hist[(size_t)blockIdx.x * E + x] = run[x];
  const int any_bad = __syncthreads_or(bad);
  if (tid == 0) blk_err[blockIdx.x] = any_bad ? TEMPO_DERR_BAD_ID : 0u;
}

// ---------------------------------------------------------------------------
// launch 1b, large batches only: for every expert, the exclusive prefix of
// the per-block counts over the count blocks, blk_pre[b][e] = sum over b' < b
// of blk_hist[b'][e], and in row nblk the total n_e.  Without it every k_place
// block would sum all the block histograms itself, which for a prefill-sized
// batch re-reads them a thousand times.  A block of 256 threads takes 8
// experts; the 32 threads of an expert each sum a contiguous run of count
// blocks and scan the run totals with shuffles.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_scan(const int32_t* __restrict__ blk_hist, int nblk, int E,
                                              int32_t* __restrict__ blk_pre) {
  const int tid = threadIdx.x, q = tid & 31;
  const int e = blockIdx.x * 8 + (tid >> 5);
  const int per = (nblk + 31) / 32;
  const int b0 = min(q * per, nblk), b1 = min(b0 + per, nblk);
  // loads in batches of 8, all in flight (the values of the first batch are
  // kept for the second pass when a run is at most 8 blocks)
  int v[8];
  int sum = 0;
  for (int b = b0; b < b1; b += 8) {
#pragma unroll
    for (int u = 0; u < 8; u++) v[u] = (e < E && b + u < b1) ? blk_hist[(size_t)(b + u) * E + e] : 0;
#pragma unroll
    for (int u = 0; u < 8; u++) sum += v[u];
  }
  int incl = sum;
#pragma unroll
  for (int d = 1; d < 32; d <<= 1) {
    const int v = __shfl_up(incl, d, 32);
    if (q >= d) incl += v;
  }
  if (e < E) {
    int run = incl - sum;
    if (b1 - b0 <= 8) {
#pragma unroll
      for (int u = 0; u < 8; u++)
        if (b0 + u < b1) {
          blk_pre[(size_t)(b0 + u) * E + e] = run;
          run += v[u];
        }
    } else {
      for (int b = b0; b < b1; b++) {
        blk_pre[(size_t)b * E + e] = run;
        run += blk_hist[(size_t)b * E + e];
      }
    }
    if (q == 31) blk_pre[(size_t)nblk * E + e] = incl;
  }
}

// ---------------------------------------------------------------------------
// launch 2: plan (recomputed per block), rows of the pairs, index outputs,
// row copies
// ---------------------------------------------------------------------------

template <int ESIZE, int CHUNK>
__global__ __launch_bounds__(256) void k_place(
    const int32_t* __restrict__ ids, int P, int Pv, int K, int E, int S, int M, int snap, int H, int row_cap, int nblk,
    int copies, const int32_t* __restrict__ blk_hist, const int32_t* __restrict__ blk_pre,
    const uint32_t* __restrict__ blk_err,
    const int32_t* __restrict__ local_rank, const int32_t* __restrict__ slot_expert,
    const uint32_t* __restrict__ slot_weight, const uint32_t* __restrict__ remote_weight,
    const int32_t* __restrict__ remote_replicas, int32_t* __restrict__ expert_counts, uint32_t* __restrict__ cum_counts,
    int32_t* __restrict__ slot_counts, int32_t* __restrict__ slot_offsets, int32_t* __restrict__ pair_row,
    int32_t* __restrict__ row_token, const uint8_t* __restrict__ x, const float* __restrict__ x_scale,
    uint8_t* __restrict__ x_perm, float* __restrict__ x_perm_scale, uint32_t* __restrict__ hdr, int timing,
    uint64_t* __restrict__ t0, uint64_t* __restrict__ t1) {
  constexpr int NW = 4;
  extern __shared__ int32_t dyn[];  // n_all[E], n_before[E], first[E]
  int32_t* n_all = dyn;
  int32_t* n_before = dyn + E;
  int32_t* first = dyn + 2 * E;
  __shared__ SlotLds L;
  __shared__ int32_t s_next[kMaxS];
  __shared__ uint32_t s_w[kMaxS];
  __shared__ int s_tmp[64];
  __shared__ uint32_t s_err;
  __shared__ int32_t s_prow[CHUNK], s_ptok[CHUNK];
  __shared__ int s_wn[4];
  __shared__ int s_nplaced;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int base = blockIdx.x * CHUNK;
  const bool writer = blockIdx.x == 0;
  // own pairs' ids and in-block ranks (issued first)
  const int p = base + tid;
  int own_e = -1, own_rk = 0;
  if (tid < CHUNK && p < Pv) {
    own_e = ids[p];
    if (own_e >= 0 && own_e < E) own_rk = local_rank[p];
    else own_e = -1;
  }
  if (tid == 0) s_err = 0;
  // n_e and the prefix of this block's count block: from the scan (large
  // batches) or summed here from the block histograms
  const int cb = base / kCountThreads;
  for (int ex = tid; ex < E; ex += 256) {
    int all = 0, bef = 0, b = 0;
    if (blk_pre) {
      all = blk_pre[(size_t)nblk * E + ex];
      bef = blk_pre[(size_t)cb * E + ex];
      b = nblk;
    }
    for (; b + 16 <= nblk; b += 16) {
      int v[16];
#pragma unroll
      for (int u = 0; u < 16; u++) v[u] = blk_hist[(size_t)(b + u) * E + ex];
#pragma unroll
      for (int u = 0; u < 16; u++) {
        bef += (b + u < cb) ? v[u] : 0;
        all += v[u];
      }
    }
    for (; b < nblk; b++) {
      const int v = blk_hist[(size_t)b * E + ex];
      bef += (b < cb) ? v : 0;
      all += v;
    }
    n_all[ex] = all;
    n_before[ex] = bef;
    first[ex] = 0x7fffffff;
    if (writer) {
      expert_counts[ex] = all;
      if (cum_counts) cum_counts[ex] = cum_counts[ex] + (uint32_t)all;
    }
  }
  uint32_t eb = 0;
  if (writer)
    for (int b = tid; b < nblk; b += 256) eb |= blk_err[b];
  __syncthreads();
  if (eb) atomicOr(&s_err, eb);
  __syncthreads();
  // the plan: one wavefront when S <= 64, the block otherwise
  if (S <= 64) {
    if (tid < 64)
      plan_slots_wave(n_all, E, S, M, snap, slot_expert, slot_weight, remote_weight, remote_replicas, L, first, s_next,
                      writer, slot_counts, slot_offsets, row_token, hdr, hdr + kHdrSticky, s_err, timing, t0, t1);
  } else {
    if (writer)
      plan_slots<NW, true>(n_all, E, S, M, snap, slot_expert, slot_weight, remote_weight, remote_replicas, slot_counts,
                           slot_offsets, row_token, hdr, L, &s_err, s_w, s_tmp, timing, t0, t1);
    else
      plan_slots<NW, false>(n_all, E, S, M, snap, slot_expert, slot_weight, remote_weight, remote_replicas, slot_counts,
                            slot_offsets, row_token, hdr, L, &s_err, s_w, s_tmp, timing, t0, t1);
    for (int s2 = tid; s2 < S; s2 += 256) {
      const int ex = L.se[s2];
      int nx = -1;
      if (ex >= 0 && ex < E) {
        atomicMin(&first[ex], s2);
        for (int s3 = s2 + 1; s3 < S; s3++)
          if (L.se[s3] == ex) {
            nx = s3;
            break;
          }
      }
      s_next[s2] = nx;
    }
  }
  __syncthreads();
  // block 0 marks the padding rows of every slot, all threads together (one
  // lane per slot would take up to M - 1 dependent stores)
  if (writer && S <= 64)
    for (int s2 = 0; s2 < S; s2++)
      for (int r = L.off[s2] + L.c[s2] + tid; r < L.off[s2 + 1]; r += 256) row_token[r] = -1;
  // own pairs: rank -> slot -> row; the placed ones are compacted in pair
  // order (per wavefront by ballot, wavefronts in order)
  int row = -1;
  if (tid < CHUNK) {
    if (own_e >= 0) {
      const int r = n_before[own_e] + own_rk;
      for (int s2 = first[own_e]; s2 >= 0 && s2 < S; s2 = s_next[s2])
        if (r >= L.lo[s2] && r < L.lo[s2] + L.c[s2]) {
          row = L.off[s2] + (r - L.lo[s2]);
          break;
        }
      if (row >= row_cap) row = -1;  // defensive: never index past the buffers
    }
    if (p < P) {
      pair_row[p] = row;
      if (row >= 0) row_token[row] = p / K;
    }
  }
  const uint64_t m = __ballot(row >= 0);
  if (lane == 0) s_wn[w] = __popcll(m);
  __syncthreads();
  int wbase = 0;
  for (int i = 0; i < w; i++) wbase += s_wn[i];
  if (row >= 0) {
    const int pos = wbase + __popcll(m & ((1ull << lane) - 1ull));
    s_prow[pos] = row;
    s_ptok[pos] = p / K;
  }
  if (tid == 0) s_nplaced = s_wn[0] + s_wn[1] + s_wn[2] + s_wn[3];
  __syncthreads();
  const int R = s_nplaced;
  const int nch = H * ESIZE / 16;
  for (int j = w; j < R; j += 4) {
    if (ESIZE == 1 && (copies & 2)) {  // scales are stored block-major: [H/128][row_cap]
      const int ns = H / 128;
      for (int i = lane; i < ns; i += 64)
        x_perm_scale[(size_t)i * row_cap + s_prow[j]] = x_scale[(size_t)s_ptok[j] * ns + i];
    }
    if (!(copies & 1)) continue;
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
  }
}

// ---------------------------------------------------------------------------
// the whole of stage 1 in one workgroup (decode-sized bf16 batches whose rows
// the gate/up GEMM gathers itself).  Wavefront w ranks the contiguous run of
// pairs [w R 64, (w + 1) R 64) (R rounds of 64) without barriers: per round
// each lane ORs its bit into the wavefront's 64-bit mask of its expert (LDS),
// reads the mask back (its peers: the lanes with the same expert), and the
// wavefront's own running count per expert gives the offset of its earlier
// rounds; the first lane of a group advances the count and clears the mask.
// One scan per expert over the wavefronts' counts then turns the ranks into
// global stable ranks and gives n_e.  The plan's inputs are loaded into LDS
// together with the ids, so the plan runs on LDS alone.  Then rank -> slot ->
// row for every pair.  Same outputs as k_count + k_place without x_perm.
// ---------------------------------------------------------------------------

// Philox-4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC 2011): word 0
// of the block at counter (ctr, 0, 0, 0) and key (key, 0).  A round forms the
// 128-bit products of counter words 0 and 2 with the round multipliers,
// permutes the words and XORs in the key, which then advances by the Weyl
// constants.
__device__ __forceinline__ uint64_t philox4x64_10_w0(uint64_t ctr, uint64_t key) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = ctr, c1 = 0, c2 = 0, c3 = 0, k0 = key, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; r++) {
    const uint64_t hi0 = __umul64hi(c0, M0), lo0 = c0 * M0;
    const uint64_t hi1 = __umul64hi(c2, M1), lo1 = c2 * M1;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += W0;
    k1 += W1;
  }
  return c0;
}

__global__ __launch_bounds__(kSmallWaves * 64) void k_dispatch_small(
    const int32_t* __restrict__ ids, int P, int Pv, int K, int E, int S, int M, int snap, int sample, uint64_t seed,
    int row_cap, const int32_t* __restrict__ slot_expert, const uint32_t* __restrict__ slot_weight,
    const uint32_t* __restrict__ remote_weight, const int32_t* __restrict__ remote_replicas,
    int32_t* __restrict__ expert_counts, uint32_t* __restrict__ cum_counts, int32_t* __restrict__ slot_counts,
    int32_t* __restrict__ slot_offsets, int32_t* __restrict__ pair_row, int32_t* __restrict__ row_token,
    uint32_t* __restrict__ hdr, int timing, uint64_t* __restrict__ t0, uint64_t* __restrict__ t1) {
  constexpr int NW = kSmallWaves, BD = NW * 64;
  // pairs are ranked by a key: the expert (split), or the sampled slot
  const int KW = sample ? S : E;
  // dynamic LDS: peer masks [NW][KW] (u64), run[E], first[E], remote_replicas[E],
  // remote_weight[E], row weight W[E] (sampling), wavefront counts wc[NW][KW]
  extern __shared__ uint64_t dyn64[];
  uint64_t* masks = dyn64;
  int32_t* run = reinterpret_cast<int32_t*>(dyn64 + NW * KW);
  int32_t* first = run + E;
  int32_t* s_rr = run + 2 * E;
  uint32_t* s_rw = reinterpret_cast<uint32_t*>(run + 3 * E);
  uint32_t* s_W = reinterpret_cast<uint32_t*>(run + 4 * E);
  int32_t* wc = run + 5 * E;
  __shared__ SlotLds L;
  __shared__ int32_t s_next[kMaxS];
  __shared__ int32_t s_se[kMaxS];
  __shared__ uint32_t s_sw[kMaxS];
  __shared__ uint32_t s_w[kMaxS];
  __shared__ uint32_t s_effw[kMaxS];  // sampling: the slot's weight after the zero-sum fallback
  __shared__ int32_t s_cnt[kMaxS];    // sampling: pairs drawn per slot
  __shared__ int s_tmp[64];
  __shared__ uint32_t s_err, s_sticky;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int R = (Pv + BD - 1) / BD;  // rounds per wavefront (<= kSmallRounds)
  const int pw = w * R * 64 + lane;  // this lane's pair in round 0
  const float invK = 1.0f / (float)K;
  // every global load in flight first: the plan's inputs and the ids
  int se_in = -1, rr_in = 0;
  uint32_t sw_in = 0, rw_in = 0, sticky = 0;
  if (tid == 0) sticky = hdr[kHdrSticky];
  if (tid < S) {
    se_in = slot_expert[tid];
    sw_in = slot_weight[tid];
  }
  if (tid < E) {
    rr_in = remote_replicas[tid];
    rw_in = remote_weight[tid];
  }
  int e[kSmallRounds];
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) {
    const int p = pw + r * 64;
    e[r] = (r < R && p < Pv) ? ids[p] : -1;
  }
  for (int i = tid; i < NW * KW; i += BD) {
    masks[i] = 0;
    wc[i] = 0;
  }
  if (tid == 0) {
    s_err = 0;
    s_sticky = sticky;
  }
  if (tid < S) {
    s_se[tid] = se_in;
    s_sw[tid] = sw_in;
  }
  if (tid < E) {
    s_rr[tid] = rr_in;
    s_rw[tid] = rw_in;
    run[tid] = 0;
    first[tid] = 0x7fffffff;
  }
  int bad = 0;
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) {
    if (e[r] != -1 && (e[r] < 0 || e[r] >= E)) {
      bad = 1;
      e[r] = -1;
    }
  }
  __syncthreads();
  // the rank key of every pair: its expert, or the slot its draw picks
  int key[kSmallRounds];
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) key[r] = e[r];
  if (sample) {
    // per slot: the weight after the zero-sum fallback and the next slot of
    // its expert; per expert: the row weight W and the first local slot
    if (tid < S) {
      const int ex = s_se[tid];
      if (ex >= 0 && ex < E) {
        uint64_t Wloc = 0;
        int nloc = 0, nbefore = 0, nx = -1;
        for (int s2 = 0; s2 < S; s2++)
          if (s_se[s2] == ex) {
            Wloc += s_sw[s2];
            nloc++;
            if (s2 < tid) nbefore++;
            if (s2 > tid && nx < 0) nx = s2;
          }
        const int rr = s_rr[ex];
        const uint32_t rw = s_rw[ex];
        const bool has_remote = rw > 0u || rr > 0;
        uint64_t W = Wloc + (has_remote ? rw : 0u);
        uint32_t mine = s_sw[tid];
        if (W >= (1ull << 32)) atomicOr(&s_err, TEMPO_DERR_WEIGHT_OVERFLOW);
        if (W == 0 || W >= (1ull << 32)) {
          W = (uint64_t)nloc + (has_remote && rr > 0 ? (uint64_t)rr : 0ull);
          mine = 1;
        }
        s_effw[tid] = mine;
        s_next[tid] = nx;
        if (nbefore == 0) {
          first[ex] = tid;
          s_W[ex] = (uint32_t)W;
        }
      } else {
        atomicOr(&s_err, TEMPO_DERR_BAD_SLOT_EXPERT);
        s_next[tid] = -1;
      }
    }
    __syncthreads();
    // one draw per pair: Philox-4x64-10 word 0 at counter (p, 0, 0, 0), key
    // (seed, 0); u = floor(hi32 * W / 2^32); the first entry with u < C_j
    // (the local slots in order, then the remote share)
#pragma unroll
    for (int r = 0; r < kSmallRounds; r++) {
      int k = -1;
      if (e[r] >= 0) {
        atomicAdd(&run[e[r]], 1);
        const int s0 = first[e[r]];
        if (s0 < S) {
          const uint64_t u = ((philox4x64_10_w0((uint64_t)(pw + r * 64), seed) >> 32) * (uint64_t)s_W[e[r]]) >> 32;
          uint64_t C = 0;
          for (int s2 = s0; s2 >= 0 && s2 < S; s2 = s_next[s2]) {
            C += s_effw[s2];
            if (u < C) {
              k = s2;
              break;
            }
          }
        }
      }
      key[r] = k;
    }
  }
  // ranks within the wavefront's run
  int32_t* const mine = wc + w * KW;
  uint64_t* const mk = masks + w * KW;
  const uint64_t below = (1ull << lane) - 1ull;
  int rk[kSmallRounds];
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) {
    rk[r] = -1;
    const int kx = key[r];
    if (r < R && kx >= 0) {
      atomicOr(reinterpret_cast<unsigned long long*>(&mk[kx]), 1ull << lane);
      // (one LDS instruction for the whole wavefront: every lane's bit is in
      // before any lane reads the mask, and every read is done before the
      // first lane's clear)
      const uint64_t peers = mk[kx];
      const int rw = __popcll(peers & below);
      const int cnt = mine[kx];
      rk[r] = cnt + rw;
      if (rw == 0) {
        mine[kx] = cnt + __popcll(peers);
        mk[kx] = 0;
      }
    }
  }
  if (bad) atomicOr(&s_err, TEMPO_DERR_BAD_ID);
  __syncthreads();
  // per key: exclusive prefix over the wavefronts (in place) and the total
  // (n_e when ranking by expert, the slot's count when sampling)
  for (int kx = tid; kx < KW; kx += BD) {
    int acc = 0;
#pragma unroll
    for (int w2 = 0; w2 < NW; w2++) {
      const int v = wc[w2 * KW + kx];
      wc[w2 * KW + kx] = acc;
      acc += v;
    }
    if (sample) s_cnt[kx] = acc;
    else run[kx] = acc;
  }
  __syncthreads();
  for (int ex = tid; ex < E; ex += BD) {
    const int n = run[ex];
    expert_counts[ex] = n;
    if (cum_counts) cum_counts[ex] = cum_counts[ex] + (uint32_t)n;
  }
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++)
    if (key[r] >= 0) rk[r] += mine[key[r]];
  if (sample) {
    // padded sizes, offsets and the header from the drawn counts
    const int c = tid < S ? s_cnt[tid] : 0;
    const int Pz = (c + M - 1) / M * M;
    int total = 0;
    const int off = block_exclusive_scan<NW>(Pz, s_tmp, &total);
    if (tid < S) {
      L.off[tid] = off;
      L.c[tid] = c;
      slot_counts[tid] = c;
      slot_offsets[tid] = off;
      if (timing) {
        t0[tid] = ~0ull;
        t1[tid] = 0ull;
      }
    }
    if (tid == 0) {
      L.off[S] = total;
      slot_offsets[S] = total;
    }
    block_exclusive_scan<NW>(Pz / M, s_tmp, &total);
    const int ntiles = total;
    block_exclusive_scan<NW>(c > 0 ? 1 : 0, s_tmp, &total);
    const int G = total;
    block_exclusive_scan<NW>(c, s_tmp, &total);
    if (tid == 0) {
      hdr[kHdrTiles] = (uint32_t)ntiles;
      hdr[kHdrActive] = (uint32_t)G;
      hdr[kHdrPairs] = (uint32_t)total;
      hdr[kHdrLastErr] = s_err;
      hdr[kHdrSticky] = s_sticky | s_err;
    }
    __syncthreads();
    for (int s2 = w; s2 < S; s2 += NW)
      for (int r = L.off[s2] + L.c[s2] + lane; r < L.off[s2 + 1]; r += 64) row_token[r] = -1;
#pragma unroll
    for (int r = 0; r < kSmallRounds; r++) {
      const int p = pw + r * 64;
      if (r < R && p < P) {
        const int row = key[r] >= 0 ? L.off[key[r]] + rk[r] : -1;
        pair_row[p] = row;
        if (row >= 0) row_token[row] = (int)(((float)p + 0.5f) * invK);  // p / K exactly (as below)
      }
    }
    for (int p = R * BD + tid; p < P; p += BD) pair_row[p] = -1;
    return;
  }
  if (S <= 64) {
    if (tid < 64)
      plan_slots_wave(run, E, S, M, snap, s_se, s_sw, s_rw, s_rr, L, first, s_next, true, slot_counts, slot_offsets,
                      row_token, hdr, &s_sticky, s_err, timing, t0, t1);
    __syncthreads();
    // padding rows: one wavefront per slot
    for (int s2 = w; s2 < S; s2 += NW)
      for (int r = L.off[s2] + L.c[s2] + lane; r < L.off[s2 + 1]; r += 64) row_token[r] = -1;
  } else {
    plan_slots<NW, true>(run, E, S, M, snap, s_se, s_sw, s_rw, s_rr, slot_counts, slot_offsets, row_token, hdr, L,
                         &s_err, s_w, s_tmp, timing, t0, t1);
    for (int s2 = tid; s2 < S; s2 += BD) {
      const int ex = L.se[s2];
      int nx = -1;
      if (ex >= 0 && ex < E) {
        atomicMin(&first[ex], s2);
        for (int s3 = s2 + 1; s3 < S; s3++)
          if (L.se[s3] == ex) {
            nx = s3;
            break;
          }
      }
      s_next[s2] = nx;
    }
    __syncthreads();
  }
  // rank -> slot -> row for every pair (pairs of padding tokens: -1): the
  // expert's first slot for every round at once, the rest of its slot list
  // only where the rank lies beyond that slot
  int row[kSmallRounds];
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) {
    row[r] = -1;
    if (e[r] >= 0) {
      const int s2 = first[e[r]];
      if (s2 < S) {
        const int d = rk[r] - L.lo[s2];
        row[r] = d >= 0 && d < L.c[s2] ? L.off[s2] + d : -2;  // -2: look further
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kSmallRounds; r++) {
    if (row[r] == -2) {
      row[r] = -1;
      for (int s2 = s_next[first[e[r]]]; s2 >= 0 && s2 < S; s2 = s_next[s2])
        if (rk[r] >= L.lo[s2] && rk[r] < L.lo[s2] + L.c[s2]) {
          row[r] = L.off[s2] + (rk[r] - L.lo[s2]);
          break;
        }
    }
    if (row[r] >= row_cap) row[r] = -1;  // defensive: never index past the buffers
    const int p = pw + r * 64;
    if (r < R && p < P) {
      pair_row[p] = row[r];
      // the token p / K in fp32: for p < 2^13 and K <= 32 the product is
      // within 2^-10 of (p + 0.5) / K, whose distance to an integer is at
      // least 0.5 / K
      if (row[r] >= 0) row_token[row[r]] = (int)(((float)p + 0.5f) * invK);
    }
  }
  for (int p = R * BD + tid; p < P; p += BD) pair_row[p] = -1;
}

// Row copies after k_dispatch_small: the token rows into x_perm (when asked)
// and, for fp8, their activation scales into x_perm_scale (block-major; when
// it is not null), for the rows in use (slot_offsets[S]); one wavefront per
// row.
template <int ESIZE>
__global__ __launch_bounds__(256) void k_gather_rows(const int32_t* __restrict__ row_token,
                                                     const int32_t* __restrict__ slot_offsets, int S, int H, int row_cap,
                                                     int gather_rows, const uint8_t* __restrict__ x,
                                                     const float* __restrict__ x_scale, uint8_t* __restrict__ x_perm,
                                                     float* __restrict__ x_perm_scale) {
  const int lane = threadIdx.x & 63;
  const int used = min(slot_offsets[S], row_cap);
  const int nch = H * ESIZE / 16;
  for (int row = blockIdx.x * 4 + (threadIdx.x >> 6); row < used; row += gridDim.x * 4) {
    const int tok = row_token[row];
    if (tok < 0) continue;
    if (ESIZE == 1 && x_perm_scale) {
      const int ns = H / 128;
      for (int i = lane; i < ns; i += 64) x_perm_scale[(size_t)i * row_cap + row] = x_scale[(size_t)tok * ns + i];
    }
    if (!gather_rows) continue;
    const uint4* __restrict__ src = reinterpret_cast<const uint4*>(x) + (size_t)tok * nch;
    uint4* __restrict__ dst = reinterpret_cast<uint4*>(x_perm) + (size_t)row * nch;
    constexpr int U = 8;
    for (int c0 = lane; c0 < nch; c0 += 64 * U) {
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; u++) v[u] = src[min(c0 + u * 64, nch - 1)];
#pragma unroll
      for (int u = 0; u < U; u++)
        if (c0 + u * 64 < nch) dst[c0 + u * 64] = v[u];
    }
  }
}

}  // namespace

bool dispatch_sample_supported(const tempo_moe_shape& s) {
  return s.T * s.K <= kSmallRounds * kSmallWaves * 64 && s.E <= kSmallMaxE && s.S <= kMaxS;
}

hipError_t launch_dispatch(const tempo_moe_shape& s, const tempo_plan& plan, const int32_t* topk_ids, const void* x,
                           const float* x_scale, const tempo_dispatch_out& out, char* ws, const Layout& L,
                           bool timing, bool copy_rows, bool copy_scales, hipStream_t st) {
  const int P = s.T * s.K, Pv = s.T_valid * s.K;
  const int snap = (plan.flags & TEMPO_PLAN_SNAP_TILES) ? 1 : 0;
  const int sample = (plan.flags & TEMPO_PLAN_SAMPLE) ? 1 : 0;
  int ebits = 0;
  while ((1 << ebits) < s.E) ebits++;
  int32_t* blk_hist = reinterpret_cast<int32_t*>(ws + L.blk_hist);
  uint32_t* blk_err = reinterpret_cast<uint32_t*>(ws + L.blk_err);
  int32_t* local_rank = reinterpret_cast<int32_t*>(ws + L.local_rank);
  uint64_t* t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  uint64_t* t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  uint32_t* hdr = reinterpret_cast<uint32_t*>(ws + L.header);

  copy_scales = copy_scales && s.dtype != TEMPO_BF16;
  float* const xps = copy_scales ? out.x_perm_scale : nullptr;
  // one workgroup for decode-sized batches whose rows stage 2 reads from the
  // token rows, and for sampled replicas (then a row-copy launch for what is
  // asked for).  fp8 batches whose activation scales stage 2 reads permuted
  // take it up to kSmallScalesMaxP pairs, with a launch that copies the
  // scales: for more pairs the single workgroup's ranking costs more than
  // count + place (measured: 2048 pairs 15.6 against 20.3 us; 8192 pairs
  // 18.6 against 15.7 us)
  const bool small = P <= kSmallRounds * kSmallWaves * 64 && s.E <= kSmallMaxE;
  if (sample && !dispatch_sample_supported(s)) return hipErrorNotSupported;
  if (sample || (small && !copy_rows && (!copy_scales || P <= kSmallScalesMaxP))) {
    const int KW = sample ? s.S : s.E;
    const size_t lds = (size_t)kSmallWaves * KW * 8 + (size_t)(kSmallWaves * KW + 5 * s.E) * sizeof(int32_t);
    hipLaunchKernelGGL(k_dispatch_small, dim3(1), dim3(kSmallWaves * 64), lds, st, topk_ids, P, Pv, s.K, s.E, s.S,
                       s.m_tile, snap, sample, plan.seed, L.row_cap, plan.slot_expert,
                       plan.slot_weight, plan.remote_weight, plan.remote_replicas, out.expert_counts, out.cum_counts,
                       out.slot_counts, out.slot_offsets, out.pair_row, out.row_token, hdr, timing ? 1 : 0, t0, t1);
    if (copy_rows || copy_scales) {
      const int grid = std::min(ceil_div(L.row_cap, 4), persistent_grid(8));
      if (s.dtype == TEMPO_BF16)
        hipLaunchKernelGGL(k_gather_rows<2>, dim3(grid), dim3(256), 0, st, out.row_token, out.slot_offsets, s.S, s.H,
                           L.row_cap, copy_rows ? 1 : 0, static_cast<const uint8_t*>(x), x_scale,
                           static_cast<uint8_t*>(out.x_perm), xps);
      else
        hipLaunchKernelGGL(k_gather_rows<1>, dim3(grid), dim3(256), 0, st, out.row_token, out.slot_offsets, s.S, s.H,
                           L.row_cap, copy_rows ? 1 : 0, static_cast<const uint8_t*>(x), x_scale,
                           static_cast<uint8_t*>(out.x_perm), xps);
    }
    return hipGetLastError();
  }

  hipLaunchKernelGGL(k_count, dim3(L.nblk), dim3(kCountThreads), (kCountThreads / 64 + 1) * s.E * sizeof(int32_t), st,
                     topk_ids, Pv, s.E, ebits, blk_hist, blk_err, local_rank);
  // with more than kScanBlocks count blocks the prefixes are scanned once
  const int32_t* blk_pre = nullptr;
  if (L.nblk > kScanBlocks) {
    int32_t* pre = reinterpret_cast<int32_t*>(ws + L.blk_pre);
    hipLaunchKernelGGL(k_scan, dim3((s.E + 7) / 8), dim3(256), 0, st, blk_hist, L.nblk, s.E, pre);
    blk_pre = pre;
  }
  const bool large = blk_pre != nullptr;
  const int nb = ceil_div(P, large ? kPlaceChunkLarge : kPlaceChunk);
  // row and scale copies: inside k_place for small batches; for large ones a
  // row-parallel launch after it (a placing block holds a few dozen rows, too
  // few loads in flight)
  const int copies = large ? 0 : (copy_rows ? 1 : 0) | (copy_scales ? 2 : 0);
  const size_t lds = (size_t)3 * s.E * sizeof(int32_t);
  auto launch = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(nb), dim3(256), lds, st, topk_ids, P, Pv, s.K, s.E, s.S, s.m_tile, snap, s.H, L.row_cap,
                       L.nblk, copies, blk_hist, blk_pre, blk_err, local_rank, plan.slot_expert,
                       plan.slot_weight, plan.remote_weight, plan.remote_replicas, out.expert_counts, out.cum_counts,
                       out.slot_counts, out.slot_offsets, out.pair_row, out.row_token, static_cast<const uint8_t*>(x),
                       x_scale, static_cast<uint8_t*>(out.x_perm), out.x_perm_scale, hdr, timing ? 1 : 0, t0, t1);
  };
  if (s.dtype == TEMPO_BF16) {
    if (large) launch(k_place<2, kPlaceChunkLarge>);
    else launch(k_place<2, kPlaceChunk>);
  } else {
    if (large) launch(k_place<1, kPlaceChunkLarge>);
    else launch(k_place<1, kPlaceChunk>);
  }
  if (large && (copy_rows || copy_scales)) {
    const int grid = std::min(ceil_div(L.row_cap, 4), persistent_grid(8));
    if (s.dtype == TEMPO_BF16)
      hipLaunchKernelGGL(k_gather_rows<2>, dim3(grid), dim3(256), 0, st, out.row_token, out.slot_offsets, s.S, s.H,
                         L.row_cap, copy_rows ? 1 : 0, static_cast<const uint8_t*>(x), x_scale,
                         static_cast<uint8_t*>(out.x_perm), xps);
    else
      hipLaunchKernelGGL(k_gather_rows<1>, dim3(grid), dim3(256), 0, st, out.row_token, out.slot_offsets, s.S, s.H,
                         L.row_cap, copy_rows ? 1 : 0, static_cast<const uint8_t*>(x), x_scale,
                         static_cast<uint8_t*>(out.x_perm), xps);
  }
  return hipGetLastError();
}

}  // namespace tempo
