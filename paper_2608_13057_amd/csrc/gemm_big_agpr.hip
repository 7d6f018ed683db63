// Stage 2, bf16, for 256-row M-tiles: the linear regime of the cost model,
// where a slot's rows are many and the per-token compute (beta, Eq. 1)
// dominates the weight streaming (Sec. 2.2).  Here the work is a plain dense
// contraction, so it is organised for MFMA throughput rather than for HBM
// streaming:
//
// * Both operands are packed in MFMA operand order: the weights by
//   tempo_moe_pack_weights, the activation rows of each 256-row tile by
//   k_pack_rows below, and the gate/up result h by the gate/up epilogue, in
//   the layout the down GEMM reads.  One 16-element sub-step of 256 rows is
//   then eight 1 KB pieces of consecutive bytes, each the fragment of 32
//   rows that one MFMA operand register quadruple takes.
// * A work item is one (M-tile of 256 rows, 256 packed weight rows) pair;
//   items are handed out round-robin to a persistent grid (one workgroup per
//   CU) in an XCD-aware order.  There is no split of the contraction: each
//   item accumulates its sub-steps in order, so the result of a row depends
//   only on its own inputs.
// * Four wavefronts in a 2 x 2 arrangement each own a 128 x 128 block of the
//   item: 4 x 4 MFMA tiles of 32 x 32 (256 accumulator registers per lane,
//   kept in AGPRs).  The MFMAs take the weights as their first operand, so a
//   tile holds the transposed product: a lane owns one token row and runs of
//   four consecutive output columns.
// * The operands stream through an LDS ring of NSS slots of 16 KB, one slot
//   per sub-step (activations, then weights), filled by DMA.  A slot is
//   released one sub-step at a time: after each sub-step's barrier the DMA
//   of the sub-step NSS ahead goes into the slot freed by the previous one,
//   so the loads leave in an even stream well ahead of their use (a whole
//   step's burst at once would queue in the vector L1 and arrive late), and
//   the stream runs on across item boundaries: the next item's first
//   sub-steps load during this item's epilogue.  Fragments are
//   double-buffered in registers: the LDS reads of sub-step u + 1 are
//   interleaved with the MFMAs of sub-step u, and so are the DMA pieces,
//   at a different point for each wavefront.
// * Epilogue straight from the accumulators: SwiGLU (gate/up) into packed h
//   with 16-byte stores that fill 1 KB per instruction, or the bf16 rows of
//   y_perm (down), 16 bytes per lane and row.
#include "gemm_stream.h"

namespace tempo {
namespace {

using namespace gemm;

constexpr int BIG_M = 256;             // rows per item (the M-tile)
constexpr int BIG_N = 256;             // packed weight rows per item (two blocks of 128)
constexpr int SUB_BYTES = 8 * 1024;    // one 16-element sub-step of 256 rows: eight 1 KB fragment pieces
constexpr int SLOT = 2 * SUB_BYTES;    // ring slot: the activations, then the weights of one sub-step
constexpr int NSS = 9;                 // ring slots
constexpr int BIG_GM = 4;              // M-tiles per group of the item order

// Packed 256-row tile of K-element rows: sub-step u (elements 16u .. 16u+15)
// at u * SUB_BYTES; in it, piece b (rows 32b .. 32b+31) at b * 1024, where
// lane l holds row 32b + (l & 31), elements 16u + 8 (l >> 5) .. + 7.
__host__ __device__ constexpr size_t packed_tile_bytes(int K) { return (size_t)BIG_M * K * 2; }

// The activation rows of every 256-row tile in the packed order, from the
// token rows (gather: row r is token row_token[r] of A) or from permuted rows
// (row r of A); padding rows (row_token -1) are zero.  The workgroups of a
// fixed grid take the (tile, 64-element step) blocks of the live tiles in
// turn (the tile count is only known on the device; a grid sized for the
// most tiles the buffers allow would be mostly workgroups that exit at
// once, and launching those costs more than the copy).  In a block,
// wavefront w writes sub-step w: lane l loads the 16 bytes of row
// 32b + (l & 31), chunk 2w + (l >> 5), and the stores fill 1 KB each.
__global__ __launch_bounds__(256) void k_pack_rows(const char* __restrict__ A, int gather,
                                                   const int32_t* __restrict__ row_token,
                                                   const int32_t* __restrict__ slot_offsets, int S, int max_tiles,
                                                   int K, char* __restrict__ out) {
  const int KT = K / 64;
  const int blocks = max(0, min(slot_offsets[S] / BIG_M, max_tiles)) * KT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const size_t row_bytes = (size_t)K * 2;
#pragma unroll 1
  for (int blk = blockIdx.x; blk < blocks; blk += gridDim.x) {
    const int tile = blk / KT, k = blk - tile * KT;
    char* dst = out + (size_t)tile * packed_tile_bytes(K) + (size_t)(4 * k + w) * SUB_BYTES;
    const int col = k * 128 + (2 * w + (lane >> 5)) * 16;
    // the block's row indices, then all of its row loads, then the stores:
    // two memory latencies per block (padding rows load row 0 and store 0)
    int tok[8];
#pragma unroll
    for (int b = 0; b < 8; b++) tok[b] = row_token[tile * BIG_M + 32 * b + (lane & 31)];
    i32x4 v[8];
#pragma unroll
    for (int b = 0; b < 8; b++) {
      const int row = tile * BIG_M + 32 * b + (lane & 31);
      const int src = tok[b] < 0 ? 0 : gather ? tok[b] : row;
      v[b] = *reinterpret_cast<const i32x4*>(A + (size_t)src * row_bytes + col);
    }
#pragma unroll
    for (int b = 0; b < 8; b++) {
      const i32x4 z = {0, 0, 0, 0};
      *reinterpret_cast<i32x4*>(dst + b * 1024 + lane * 16) = tok[b] < 0 ? z : v[b];
    }
  }
}

// The GEMM of one wavefront of a workgroup; WV is the wavefront's index.
// Each of the four wavefronts runs its own instance (chosen once, at the top
// of the kernel), so that its position in the 2 x 2 arrangement and the
// point where it issues its DMA are constants.
template <bool GATEUP, int WV>
__device__ __forceinline__ void big_body(const GemmArgs& p, char* ring, const int32_t* s_off, const int32_t* s_cnt) {
  constexpr int NCOLS = GATEUP ? BIG_N / 2 : BIG_N;  // output columns per item
  constexpr int wm = WV & 1, wn = WV >> 1;           // this wavefront's 128-row and 128-weight-row halves
  const int lane = threadIdx.x & 63;

  const int NT = __builtin_amdgcn_readfirstlane(max(0, min(s_off[p.S] / BIG_M, p.max_tiles)));
  const int KT = p.Kd / 64;        // steps of 64 bf16
  const int NU = 4 * KT;           // sub-steps per item
  const int NBT = p.Nout / NCOLS;  // items per M-tile
  const int items = NT * NBT;

  // Item order.  Workgroups are dealt to the 8 XCDs in turn, so workgroup b
  // runs on XCD b % 8; each XCD takes a contiguous run of the item list per
  // round.  The list goes over groups of BIG_GM M-tiles with the tile index
  // fastest, so the 32 items an XCD runs at once cover 4 M-tiles x 8 weight
  // column blocks, which its L2 serves from 12 distinct streams.
  const int G = gridDim.x;
  const int lin0 = (G % 8 == 0) ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8 : blockIdx.x;
  const int my_items = lin0 < items ? (items - 1 - lin0) / G + 1 : 0;
  if (my_items == 0) return;
  auto item_of = [&](int n, int& tile, int& nbt) {
    const int it = lin0 + n * G;
    const int grp = it / (BIG_GM * NBT), w_in = it - grp * (BIG_GM * NBT);
    const int gm = min(BIG_GM, NT - grp * BIG_GM);  // tiles in this group
    nbt = w_in / gm;
    tile = grp * BIG_GM + (w_in - nbt * gm);
  };

  // DMA cursor: the next sub-step to load (item ordinal dn, sub-step du)
  // and where its pieces come from: a_src (activations) and w_src (this
  // wavefront's weight block), advanced per sub-step.  Past the last item
  // it loads the last item's sub-steps again, which nobody reads, so that
  // every sub-step issues the same number of loads and the waits below stay
  // exact.
  int dn = 0, du = 0;
  const char* a_src = nullptr;
  const char* w_src = nullptr;
  auto dma_item = [&]() {
    int tile, nbt;
    item_of(dn, tile, nbt);
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, p.S, tile * BIG_M));
    a_src = p.A + (size_t)tile * packed_tile_bytes(p.Kd);
    w_src = slot_tensor(p.W, p.w_slot_bytes, p.wtab, p.wfield, slot) + (size_t)(2 * nbt + (WV >> 1)) * KT * B_BYTES;
  };
  // This wavefront's share of a sub-step, as four 1 KB pieces: activation
  // pieces 2 WV and 2 WV + 1; weight pieces 2 WV and 2 WV + 1, i.e. the
  // 32-row blocks 2 (WV & 1) and 2 (WV & 1) + 1 of weight block WV >> 1,
  // whose sub-step ks sits at ks * 1 KB of the 4 KB piece of each 32-row
  // block in every 16 KB step.
  // (the piece offsets go into the scalar source address, so that a single
  // per-lane register, lane * 16, serves every piece)
  const uint32_t ring_lds = lds_addr(ring);
  const uint32_t lane16 = lane * 16;
  auto dma_piece = [&](uint32_t sl, int pc) {
    const char* src = pc < 2 ? a_src + (2 * WV + pc) * 1024 : w_src + (2 * (WV & 1) + (pc & 1)) * 4096;
    lds_dma16s(src, lane16, sl + (pc < 2 ? 0 : SUB_BYTES) + (2 * WV + (pc & 1)) * 1024);
  };
  auto dma_advance = [&]() {
    a_src += SUB_BYTES;
    w_src += (du & 3) == 3 ? B_BYTES - 3 * 1024 : 1024;
    if (++du == NU) {
      du = 0;
      if (dn + 1 < my_items) ++dn;
      dma_item();
    }
  };

  f32x16 acc[4][4];
  bf16x8 fa[2][4], fb[2][4];
  auto frag_a = [&](int slot, int buf, int i) {
    fa[buf][i] = *reinterpret_cast<const bf16x8*>(ring + slot * SLOT + (4 * wm + i) * 1024 + lane * 16);
  };
  auto frag_b = [&](int slot, int buf, int j) {
    fb[buf][j] = *reinterpret_cast<const bf16x8*>(ring + slot * SLOT + SUB_BYTES + (4 * wn + j) * 1024 + lane * 16);
  };

  // Sub-step g, in ring slot sc = g % NSS, in four groups i = 0..3: the four
  // MFMAs of row block i, two LDS reads of sub-step g + 1 (from slot sn)
  // after the first two, and after MFMA number WV one DMA piece of sub-step
  // g + NSS - 1 into slot (g - 1) % NSS (address sl), whose sub-step g - 1
  // every wavefront read before the previous barrier.  The four
  // wavefronts' pieces thus reach the texture addresser 32 cycles apart
  // (issued together they queue there and hold up the later wavefronts),
  // and the few non-MFMA instructions between two MFMAs stay in their
  // shadow (a wavefront issues about one instruction per four cycles).
  // Then, once sub-step g + 2 has landed and every wavefront holds sub-step
  // g + 1, the barrier.  Loads complete in order, and NSS - 3 sub-steps of
  // four loads each were issued after sub-step g + 2.  first: the item's
  // first sub-step, which starts its sums from zero.  The slots of the next
  // sub-step are worked out before the barrier.
  int sc = 0, sn = 1;
  uint32_t sl = ring_lds + (NSS - 1) * SLOT;
  auto substep = [&](int buf, bool first) {
    const f32x16 zero = {};
#pragma unroll
    for (int i = 0; i < 4; i++) {
#pragma unroll
      for (int j = 0; j < 4; j++) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[buf][j], fa[buf][i], first ? zero : acc[i][j], 0, 0, 0);
        if (j == 0) frag_a(sn, buf ^ 1, i);
        if (j == 1) frag_b(sn, buf ^ 1, i);
        __builtin_amdgcn_sched_barrier(0);
        if (j == WV) {
          dma_piece(sl, i);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    dma_advance();
    sl = ring_lds + sc * SLOT;
    sc = sn;
    sn = sn + 1 == NSS ? 0 : sn + 1;
    wait_lgkm0();
    __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(4 * (NSS - 3)));
    barrier_nofence();
    __builtin_amdgcn_sched_barrier(0);
  };

  // prologue: sub-steps 0 .. NSS - 2 into slots 0 .. NSS - 2 (the first
  // sub-step loads NSS - 1 into the last slot); sub-steps 0 and 1 landed
  // before the first reads
  dma_item();
#pragma unroll 1
  for (int g = 0; g < NSS - 1; g++) {
#pragma unroll
    for (int pc = 0; pc < 4; pc++) dma_piece(ring_lds + g * SLOT, pc);
    dma_advance();
  }
  __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(4 * (NSS - 3)));
  barrier_nofence();
#pragma unroll
  for (int i = 0; i < 4; i++) {
    frag_a(0, 0, i);
    frag_b(0, 0, i);
  }
  __builtin_amdgcn_sched_barrier(0);

#pragma unroll 1
  for (int n = 0; n < my_items; n++) {
    int tile, nbt;
    item_of(n, tile, nbt);
    const int row0 = tile * BIG_M;
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, p.S, row0));
    const int nvalid = __builtin_amdgcn_readfirstlane(min(BIG_M, s_off[slot] + s_cnt[slot] - row0));
    const uint64_t tstart = p.timing ? __builtin_amdgcn_s_memrealtime() : 0;  // (uniform: scalar registers)

    substep(0, true);
    substep(1, false);
#pragma unroll 1
    for (int u = 2; u < NU; u += 2) {
      substep(0, false);
      substep(1, false);
    }

    // Epilogue.  Lane l of tile (i, j) holds token row 128 wm + 32 i + (l & 31)
    // and, in element e, packed weight row 8 (e / 4) + 4 (l / 32) + e % 4 of
    // the 32-row piece j of block wn.  In a gate/up piece rows 0..15 are gate
    // columns and rows 16..31 the up columns with the same indices, so gate
    // and up of a column are elements e and e + 8 of one lane.
    // (The lane index is produced afresh here, so that the compiler keeps no
    // per-lane store address live across the item loop: a spill reload would
    // make it wait for every load in flight, the ring's DMA included.)
    int lid;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lid));
    const int l31 = lid & 31, h = lid >> 5;
    auto pack4 = [](float v0, float v1, float v2, float v3) {
      uint2 w;
      w.x = bf16x2_rne(v0, v1);
      w.y = bf16x2_rne(v2, v3);
      return w;
    };
    // Lanes l and l + 32 hold the two 8-byte halves (columns 8 q .. 8 q + 3
    // and 8 q + 4 .. 8 q + 7) of the same row; one lane swap per pair of
    // column chunks (q0, q1) gives lane l < 32 chunk q0 and lane l + 32
    // chunk q1 of row l, each as 16 consecutive bytes.
    auto swap16 = [](uint2 w0, uint2 w1) {
      const auto x = __builtin_amdgcn_permlane32_swap(w0.x, w1.x, false, false);
      const auto y = __builtin_amdgcn_permlane32_swap(w0.y, w1.y, false, false);
      return i32x4{(int)x[0], (int)y[0], (int)x[1], (int)y[1]};
    };
    if (GATEUP) {
      // h column c = 128 nbt + 64 wn + 16 j + 8 q + 4 h + m is element 4 h + m
      // of 8-column chunk q of sub-step j of the down GEMM's step 2 nbt + wn;
      // chunk q of row r is lane (r & 31) + 32 q of the piece of rows r / 32,
      // so after the swap lane l stores at l * 16: 1 KB in one instruction
      char* hb = static_cast<char*>(p.C) + (size_t)tile * packed_tile_bytes(p.Nout) + lid * 16;
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const f32x16& v = acc[i][j];
          uint2 w[2];
#pragma unroll
          for (int q = 0; q < 2; q++)
            w[q] = pack4(silu_mul(v[4 * q], v[4 * q + 8]), silu_mul(v[4 * q + 1], v[4 * q + 9]),
                         silu_mul(v[4 * q + 2], v[4 * q + 10]), silu_mul(v[4 * q + 3], v[4 * q + 11]));
          *reinterpret_cast<i32x4*>(hb + ((size_t)((2 * nbt + wn) * 4 + j) * 8 + 4 * wm + i) * 1024) =
              swap16(w[0], w[1]);
          // one tile at a time: reading every accumulator out at once would
          // spill
          __builtin_amdgcn_sched_barrier(0);
        }
    } else {
      const size_t ld = (size_t)p.Nout * 2;
      char* yb = static_cast<char*>(p.C) + (size_t)row0 * ld + (size_t)(nbt * NCOLS + 128 * wn + 8 * h) * 2;
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int r = 128 * wm + 32 * i + l31;
        char* yr = yb + r * ld;
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const f32x16& v = acc[i][j];
          uint2 w[4];
#pragma unroll
          for (int q = 0; q < 4; q++) w[q] = pack4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
          const i32x4 c0 = swap16(w[0], w[1]), c1 = swap16(w[2], w[3]);  // chunks 0 | 1 and 2 | 3
          if (r < nvalid) {  // padding rows of y_perm stay unwritten
            *reinterpret_cast<i32x4*>(yr + (32 * j) * 2) = c0;
            *reinterpret_cast<i32x4*>(yr + (32 * j + 16) * 2) = c1;
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    if (p.timing && WV == 0 && lid == 0) {
      const uint64_t tend = __builtin_amdgcn_s_memrealtime();
      atomicMin(reinterpret_cast<unsigned long long*>(&p.t0[slot]), (unsigned long long)tstart);
      atomicMax(reinterpret_cast<unsigned long long*>(&p.t1[slot]), (unsigned long long)tend);
    }
  }
  // no DMA into this workgroup's LDS may outlive it
  __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(0));
}

template <bool GATEUP>
__global__ __launch_bounds__(256, 1) void k_gemm_big(const GemmArgs p) {
  __shared__ __attribute__((aligned(1024))) char ring[NSS * SLOT];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];
  const int tid = threadIdx.x;
  for (int s = tid; s <= p.S; s += 256) s_off[s] = p.slot_offsets[s];
  for (int s = tid; s < p.S; s += 256) s_cnt[s] = p.slot_counts[s];
  __syncthreads();
  switch (__builtin_amdgcn_readfirstlane(tid >> 6)) {
    case 0: big_body<GATEUP, 0>(p, ring, s_off, s_cnt); break;
    case 1: big_body<GATEUP, 1>(p, ring, s_off, s_cnt); break;
    case 2: big_body<GATEUP, 2>(p, ring, s_off, s_cnt); break;
    default: big_body<GATEUP, 3>(p, ring, s_off, s_cnt); break;
  }
}

}  // namespace

bool experts_big_supported(const tempo_moe_shape& s) {
  return s.dtype == TEMPO_BF16 && s.m_tile == BIG_M && s.H % BIG_N == 0 && s.I % 128 == 0;
}

size_t experts_big_pack_bytes(const tempo_moe_shape& s, int row_cap) {
  return experts_big_supported(s) ? (size_t)row_cap * s.H * 2 : 0;
}

// Both GEMMs of stage 2 with 256 x 256 items.  The activation rows come from
// x_rows (token rows, gathered through row_token) or, if that is null, from
// the permuted rows in x_perm.
hipError_t launch_experts_big(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing,
                              const hipEvent_t* ev, hipStream_t st) {
  const int grid = persistent_grid(1);
  const int max_tiles = L.row_cap / BIG_M;
  auto mark = [&](int i) { return !ev || !ev[i] || hipEventRecord(ev[i], st) == hipSuccess; };

  const char* src = static_cast<const char*>(x_rows ? x_rows : d.x_perm);
  hipLaunchKernelGGL(k_pack_rows, dim3(persistent_grid(4)), dim3(256), 0, st, src, x_rows ? 1 : 0,
                     d.row_token, d.slot_offsets, s.S, max_tiles, s.H, ws + L.apack);

  GemmArgs a{};
  a.slot_counts = d.slot_counts;
  a.slot_offsets = d.slot_offsets;
  a.S = s.S;
  a.max_tiles = max_tiles;
  a.t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  a.t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  a.timing = timing ? 1 : 0;

  GemmArgs gu = a;
  gu.A = ws + L.apack;
  gu.W = static_cast<const char*>(w.w13);
  gu.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  gu.wfield = kFieldW13;
  gu.sfield = kFieldW13Scale;
  gu.w_slot_bytes = (size_t)2 * s.I * s.H * 2;
  gu.C = ws + L.h;  // packed h
  gu.Kd = s.H;
  gu.Nout = s.I;
  if (!mark(0)) return hipErrorLaunchFailure;  // after the pack: the GEMM kernel alone is timed
  hipLaunchKernelGGL(k_gemm_big<true>, dim3(grid), dim3(256), 0, st, gu);
  if (!mark(1) || !mark(2)) return hipErrorLaunchFailure;

  GemmArgs dn = a;
  dn.A = ws + L.h;
  dn.W = static_cast<const char*>(w.w2);
  dn.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  dn.wfield = kFieldW2;
  dn.sfield = kFieldW2Scale;
  dn.w_slot_bytes = (size_t)s.H * s.I * 2;
  dn.C = y_perm;
  dn.Kd = s.I;
  dn.Nout = s.H;
  hipLaunchKernelGGL(k_gemm_big<false>, dim3(grid), dim3(256), 0, st, dn);
  if (!mark(3)) return hipErrorLaunchFailure;
  return hipGetLastError();
}

}  // namespace tempo
