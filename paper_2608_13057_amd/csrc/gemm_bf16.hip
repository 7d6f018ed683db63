// Stage 2, bf16: grouped expert FFN over the M-tile-padded slot groups.
//   gate/up:  h = silu(A W_gate^T) * (A W_up^T)   (A = x_perm rows of a slot)
//   down:     y_perm = h W2^T
// (Sec. 2.1: "gate/up, activation, down"; Sec. 2.2: the cost of an activated
// replica is streaming its weights, every extra M-tile re-uses them.)
//
// One persistent kernel per GEMM, one workgroup per CU.  Work items are
// (M-tile, N-block) pairs; the tile count and the slot of each tile come from
// the stage-1 results in device memory (slot_offsets / slot_counts / header),
// so the launch has a fixed grid and needs no host round trip.  Workgroup b
// runs on XCD b mod 8 (the dispatcher's round-robin); each XCD owns a
// contiguous range of N-blocks, so an N-block of a slot's weights is fetched
// into one XCD's L2 and shared by every M-tile of that slot running there.
//
// Weights arrive in the packed layout of tempo_moe_pack_weights: the 128-row
// x K block of an item is contiguous, one 16 KB swizzled tile per step.
//
// Memory pipeline.  In the weight-streaming (flat) regime the kernel must keep
// ~100 KB per CU in flight to run near HBM bandwidth, so operand tiles go
// straight from global memory into an LDS ring with global_load_lds_dwordx4
// (no registers involved): stage k+NS-1 is in flight while stage k is
// multiplied.  A stage holds only the activation row groups that have real
// rows plus the weight tile, so the ring depth NS adapts per item (4 stages
// for a full 128-row tile, 8 for a decode-sized one).  Each wavefront waits only for its own loads of
// the stage it is about to use (vmcnt), then a plain workgroup barrier makes
// all wavefronts' data visible.  LDS rows are 128 bytes (64 bf16 of the
// contraction); the 16-byte chunk c of row r is stored at chunk c ^ (r & 7),
// so the MFMA fragment reads of 8 consecutive rows hit 8 distinct bank groups.
// Activation rows past the slot's real count are not loaded (their LDS rows
// hold stale values that only reach output rows which are never stored).
//
// Compute.  BM x 128 output tile (the gate/up instance holds 64 gate and the
// matching 64 up columns), 2 x 2 wavefronts of (BM/2) x 64, 32x32x16 bf16
// MFMA (lane layout verified on gfx950: A row / B column = lane % 32, 8
// consecutive k per lane; accumulator element i of lane l is row
// 8*(i/4) + 4*(l/32) + i%4, column l % 32).  SwiGLU and the bf16 rounding run
// on the accumulators.
//
// Every output row is produced by the same instruction sequence (same K
// order) wherever it lands, so results do not depend on the plan's split or
// on the M-tile.
#include "internal.h"

#include "gemm_common.h"

namespace tempo {
namespace {

using namespace gemm;

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int BK = 64;  // bf16 contraction elements per stage (128 bytes)

template <int BM, bool GATEUP>
__global__ __launch_bounds__(256, 1) void k_gemm_bf16(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                      size_t w_slot_stride, uint16_t* __restrict__ C,
                                                      const int32_t* __restrict__ slot_counts,
                                                      const int32_t* __restrict__ slot_offsets,
                                                      const int32_t* __restrict__ row_src, int S, int Kd,
                                                      int Nout, int max_tiles,
                                                      const uint32_t* __restrict__ hdr, uint64_t* __restrict__ t0,
                                                      uint64_t* __restrict__ t1, int timing) {
  constexpr int B_BYTES = BNW * ROWB;
  __shared__ __attribute__((aligned(1024))) char ring[RING_BYTES];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int MI = BM / 64;              // 32-row blocks per wavefront
  constexpr int NCOLS = GATEUP ? 64 : 128;  // output columns per tile
  constexpr int AG = BM / 32;               // A 8-row groups per wavefront
  constexpr int BG = BNW / 32;              // B 8-row groups per wavefront

  for (int s = tid; s <= S; s += 256) s_off[s] = slot_offsets[s];
  for (int s = tid; s < S; s += 256) s_cnt[s] = slot_counts[s];
  __syncthreads();

  int NT = (int)hdr[kHdrTiles];
  NT = NT < max_tiles ? NT : max_tiles;
  const int NB = Nout / NCOLS;
  const int xcd = blockIdx.x & 7, j0 = blockIdx.x >> 3, wpx = gridDim.x >> 3;
  const int nbx = (NB + 7) >> 3;
  const int nb_lo = xcd * nbx;
  const int my_nb = max(0, min(NB, nb_lo + nbx) - nb_lo);
  const int items = NT * my_nb;
  const int KT = Kd / BK;

  // this lane's place in a 1 KB (8-row) load group: row within the group and
  // the global chunk that lands in its swizzled LDS position
  const int lrow = lane >> 3, gchunk = (lane & 7) ^ (lane >> 3);

  for (int it = j0; it < items; it += wpx) {
    const int tile = it / my_nb;
    const int nb = nb_lo + it % my_nb;
    const int row0 = tile * BM;
    // per-item control values are wave-uniform: keep them in scalar registers
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, S, row0));
    const int nvalid = __builtin_amdgcn_readfirstlane(min(BM, s_off[slot] + s_cnt[slot] - row0));
    uint64_t tstart = 0;
    if (timing && tid == 0) tstart = __builtin_amdgcn_s_memrealtime();

    const uint16_t* __restrict__ Wsl = W + (size_t)slot * w_slot_stride;
    // per-lane source pointers at k = 0 for this wavefront's load groups
    const uint16_t* srcA[AG];
    const uint16_t* srcB[BG];
    int nA = 0;  // A groups this wavefront loads (those with a real row)
#pragma unroll
    for (int j = 0; j < AG; j++) {
      const int g = wave + 4 * j, r = g * 8 + lrow;
      // A row: the permuted row itself, or the source row it was routed from
      int ar = row0 + r;
      if (row_src) ar = (g * 8 < nvalid) ? max(row_src[row0 + min(r, nvalid - 1)], 0) : 0;
      srcA[j] = A + (size_t)ar * Kd + gchunk * 8;
      nA += (g * 8 < nvalid) ? 1 : 0;
    }
    // packed weights: the item's tiles are contiguous 16 KB blocks, one per
    // contraction step; group g of a tile is its g-th KB
#pragma unroll
    for (int j = 0; j < BG; j++) {
      const int g = wave + 4 * j;
      srcB[j] = Wsl + ((size_t)nb * KT * BNW * BK) + g * 8 * BK + lane * 8;
    }
    const int L = __builtin_amdgcn_readfirstlane(BG + nA);  // load instructions per stage for this wavefront
    // ring geometry of this item: a stage holds the activation groups that
    // have a real row, then the 16 KB weight tile; the fewer real rows, the
    // more stages fit and the more weight bytes are in flight
    const int a_groups = (nvalid + 7) >> 3;
    const int A_BYTES = a_groups * 8 * ROWB;
    const int STAGE = A_BYTES + B_BYTES;
    const int NS = min(NS_MAX, RING_BYTES / STAGE);
    // this wavefront's 32-row blocks with a real row
    const int mi_live = __builtin_amdgcn_readfirstlane((nvalid - wm * (BM / 2) + 31) >> 5);

    auto issue = [&](int kt) {
      char* st = ring + (kt % NS) * STAGE;
#pragma unroll
      for (int j = 0; j < AG; j++) {
        const int g = wave + 4 * j;
        if (g * 8 < nvalid)
          lds_dma16(srcA[j] + kt * BK, st + g * 8 * ROWB);
      }
#pragma unroll
      for (int j = 0; j < BG; j++) {
        const int g = wave + 4 * j;
        lds_dma16(srcB[j] + (size_t)kt * BNW * BK, st + A_BYTES + g * 8 * ROWB);
      }
    };

    f32x16 acc[MI][2];
#pragma unroll
    for (int mi = 0; mi < MI; mi++)
#pragma unroll
      for (int j = 0; j < 2; j++)
#pragma unroll
        for (int i = 0; i < 16; i++) acc[mi][j][i] = 0.f;

    barrier_nofence();  // every wavefront is done reading the ring (previous item)
#pragma unroll
    for (int s = 0; s < NS - 1; s++)
      if (s < KT) issue(s);
    for (int kt = 0; kt < KT; kt++) {
      wait_vmcnt(L * min(NS - 2, KT - 1 - kt));
      barrier_nofence();
      if (kt + NS - 1 < KT) issue(kt + NS - 1);
      const char* st = ring + (kt % NS) * STAGE;
      // every fragment of the stage is requested before the first MFMA
      constexpr int KS = BK / 16;
      bf16x8 a[KS][MI], b[KS][2];
#pragma unroll
      for (int ks = 0; ks < KS; ks++) {
        const int c = 2 * ks + (lane >> 5);
#pragma unroll
        for (int j = 0; j < 2; j++) {
          const int r = (GATEUP ? (j * 64 + wn * 32) : (wn * 64 + j * 32)) + (lane & 31);
          b[ks][j] = *reinterpret_cast<const bf16x8*>(st + A_BYTES + swz(r, c));
        }
#pragma unroll
        for (int mi = 0; mi < MI; mi++) {
          const int r = wm * (BM / 2) + mi * 32 + (lane & 31);
          if (mi < mi_live) a[ks][mi] = *reinterpret_cast<const bf16x8*>(st + swz(r, c));
        }
      }
#pragma unroll
      for (int ks = 0; ks < KS; ks++)
#pragma unroll
        for (int mi = 0; mi < MI; mi++)
          if (mi < mi_live)
#pragma unroll
            for (int j = 0; j < 2; j++)
              acc[mi][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][mi], b[ks][j], acc[mi][j], 0, 0, 0);
    }

    // epilogue
#pragma unroll
    for (int mi = 0; mi < MI; mi++) {
#pragma unroll
      for (int i = 0; i < 16; i++) {
        const int r = wm * (BM / 2) + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        if (r >= nvalid) continue;
        if (GATEUP) {
          const float g = acc[mi][0][i], u = acc[mi][1][i];
          const float h = g / (1.0f + __expf(-g)) * u;
          const int col = nb * 64 + wn * 32 + (lane & 31);
          C[(size_t)(row0 + r) * Nout + col] = f32_to_bf16_rne(h);
        } else {
#pragma unroll
          for (int j = 0; j < 2; j++) {
            const int col = nb * 128 + wn * 64 + j * 32 + (lane & 31);
            C[(size_t)(row0 + r) * Nout + col] = f32_to_bf16_rne(acc[mi][j][i]);
          }
        }
      }
    }
    if (timing && tid == 0) {
      const uint64_t tend = __builtin_amdgcn_s_memrealtime();
      atomicMin(reinterpret_cast<unsigned long long*>(&t0[slot]), (unsigned long long)tstart);
      atomicMax(reinterpret_cast<unsigned long long*>(&t1[slot]), (unsigned long long)tend);
    }
  }
}

template <int BM>
hipError_t launch_bm(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                     const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid,
                     hipStream_t st) {
  const uint32_t* hdr = reinterpret_cast<const uint32_t*>(ws + L.header);
  uint64_t* t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  uint64_t* t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  uint16_t* h = reinterpret_cast<uint16_t*>(ws + L.h);
  const int grid = persistent_grid(1);
  const int max_tiles = L.row_cap / BM;
  hipLaunchKernelGGL((k_gemm_bf16<BM, true>), dim3(grid), dim3(256), 0, st,
                     static_cast<const uint16_t*>(x_rows ? x_rows : d.x_perm), static_cast<const uint16_t*>(w.w13),
                     (size_t)2 * s.I * s.H, h, d.slot_counts, d.slot_offsets, x_rows ? d.row_token : nullptr, s.S, s.H,
                     s.I, max_tiles, hdr, t0, t1, timing ? 1 : 0);
  if (mid && hipEventRecord(mid, st) != hipSuccess) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_gemm_bf16<BM, false>), dim3(grid), dim3(256), 0, st, h,
                     static_cast<const uint16_t*>(w.w2), (size_t)s.H * s.I, static_cast<uint16_t*>(y_perm),
                     d.slot_counts, d.slot_offsets, nullptr, s.S, s.I, s.H, max_tiles, hdr, t0, t1, timing ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_experts_bf16(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                               const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid,
                               hipStream_t st) {
  if (s.m_tile == 128) return launch_bm<128>(s, d, w, x_rows, y_perm, ws, L, timing, mid, st);
  if (s.m_tile == 64) return launch_bm<64>(s, d, w, x_rows, y_perm, ws, L, timing, mid, st);
  return hipErrorInvalidValue;
}

}  // namespace tempo
