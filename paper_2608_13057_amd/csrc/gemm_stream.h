// Stage 2 grouped GEMM (bf16 and fp8 e4m3), the expert FFN of the activated
// slots over their M-tile-padded row groups (Sec. 2.1 gate/up, activation,
// down; Sec. 2.2: an activated replica costs the streaming of its weights,
// each further M-tile of rows re-uses them).
//
//   gate/up:  h = silu(A W_gate^T) * (A W_up^T)       A = the slot's rows of x
//   down:     y_perm = h W2^T
//
// Work decomposition (stream-K over fixed contraction chunks).  A work item
// is one (M-tile, output block of 128 weight rows) pair; its contraction of
// KT steps (128 bytes of every row per step) is cut into C fixed chunks of
// SPC steps (C at most GemmArgs::cmax: 2 for gate/up, 1 for down), SPC a
// multiple of CQ = 8 for every tile size (the last chunk is padded with
// empty steps to a multiple of the pipeline depth DR).  The chunks of all items,
// item by item, form one sequence that is split into contiguous ranges, one
// per workgroup (one workgroup per CU).  Range boundaries balance estimated
// time rather than chunk counts: a chunk of an M-tile with m live row blocks
// of 32 weighs W_BASE + m (the fixed cost of a step plus its MFMA work), taken
// from per-slot prefix sums in LDS.  When the output blocks divide by 8,
// workgroup b (dispatched to XCD b mod 8) only takes items of the b mod 8
// eighth of the output blocks, so one XCD's L2 holds each weight block that
// several M-tiles of a slot read.
//
// Arithmetic is fixed per row: chunk i of an item is accumulated by MFMA from
// zero in step order (c_i), and the result is ((c_0 + c_1) + c_2) + ... in
// fp32.  A workgroup that holds an item from chunk 0 keeps that running sum in
// registers; if its range ends inside the item it writes the running sum to a
// partial tile, and the workgroups holding the next chunks write each c_i to
// a partial tile of their own.  A fixup kernel then adds the chunks in order
// and applies the epilogue.  Results therefore do not depend on where the
// range boundaries fall, on the plan, or on the tile a row lands in.
//
// Memory pipeline.  A weight row block is used by exactly one wavefront
// (wavefront w multiplies the item's rows 32w..32w+31), so weights skip LDS:
// each wavefront loads its 4 KB of a step straight into registers with four
// 1 KB loads (the packed layout stores them in MFMA operand order), DR steps
// ahead, into a register ring indexed by step mod DR (the step loop is
// unrolled DR times so that the index is a compile-time constant).  The
// activation rows of a step are shared by the four wavefronts and go through
// an LDS ring of DR + 1 slots with global_load_lds_dwordx4 (DMA, no
// registers), issued just before the step's weight loads.  Loads complete in
// order and every step issues four weight loads, so "at most 4 (DR - 1)
// loads outstanding" means that this step's loads have landed; a barrier
// then makes every wavefront's activation rows visible.  The weight loads of
// a register set are issued on every step, also for the empty steps at the
// end, so that the compiler's own wait counts stay static.  When stage 1 left
// the rows in token order (the gate/up GEMM then gathers rows itself), the
// source rows of the M-tiles of the range (their row tables) are loaded into
// LDS before the stream starts.
//
// Compute.  BM x 128 tile per item; wavefront w multiplies all live row
// blocks of 32 by the item's weight rows 32w..32w+31, so the MFMA work is
// spread over the four SIMDs even for a decode tile of a few rows.  For
// gate/up the packed layout interleaves 16 gate rows and the same 16 up rows
// in every 32, so a wavefront holds matching gate and up columns (lanes l and
// l + 16) for SwiGLU.  bf16: 32x32x16 MFMA, 4 per step and row block; fp8:
// two 32x32x64 f8f6f4 MFMA per step into a step partial p that is added as
// acc += p * (sA[row] * sW).  Lane layout of the 32x32 MFMA family on gfx950:
// A row / B column = lane % 32, consecutive contraction elements per lane;
// accumulator element i of lane l is row 8*(i/4) + 4*(l/32) + i%4, column
// l % 32.  Finished output rows are staged in LDS and leave as whole rows,
// 16 bytes per lane.
#pragma once

#include <type_traits>

#include "gemm_common.h"

namespace tempo {
namespace gemm {

constexpr int NQ = 8;           // ring slots at most (the one being multiplied + the ones in flight)
// row tables (M-tiles) per workgroup range for the in-GEMM gather
__host__ __device__ constexpr int nrowt_of(int bm) { return bm >= 192 ? 8 : 16; }
constexpr int CMAX = 8;         // contraction chunks per work item (at most)
constexpr int PART_TILE = 128;  // columns of a partial tile (the 128 weight rows of an item)
// fixup record of a GEMM workgroup: source count (-1: nothing to complete),
// row0, output block, real rows, then the partial tiles (global tile index)
// holding chunks q1.. of the item in chunk order
constexpr int FIX_WORDS = 4 + CMAX;

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(int)))) int i32x8;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

struct GemmArgs {
  const char* A;            // activation rows (row_src == null: permuted rows; else token rows)
  const int32_t* row_src;   // null, or [row_cap] token of each permuted row (-1 = padding)
  const float* As;          // fp8: activation scales, block-major [Kd/128][as_ld]
  int as_ld;
  const char* W;            // packed weights (tempo_moe_pack_weights)
  size_t w_slot_bytes;
  const float* Wsp;         // fp8: packed weight scales [slot][block][step][4]
  size_t ws_slot_floats;
  const uint64_t* wtab;     // null, or the per-slot table (tempo_slot_weights [S])
  int wfield, sfield;       // the table fields of W and Wsp (SlotField)
  void* C;                  // output rows [row_cap][Nout]: bf16, or fp32 (fp8 gate/up)
  float* part;              // partial tiles [grid][CMAX][BM][128] fp32
  int32_t* fix;             // per workgroup: the split item whose chunk 0 it holds (FIX_WORDS int32)
  const int32_t* slot_counts;
  const int32_t* slot_offsets;
  int S, Kd, Nout, max_tiles;
  uint64_t* t0;
  uint64_t* t1;
  int timing;
  int cmax;                 // contraction chunks per work item, 1 .. CMAX (1: items are never split)
};

// Chunks per item of the two GEMMs (GemmArgs::cmax).  Fewer chunks mean
// fewer items split over workgroups, so fewer partial tiles to write and add
// up, against a coarser balance of the ranges.  Measured on the decode
// shares (64- and 128-row tiles) and the fp8 prefill share: gate/up is
// fastest with two chunks (its long contraction, H, leaves the ranges too
// coarse at one), down with one (its output has many blocks, so whole items
// balance well, and no fixup pass is needed).
constexpr int GATEUP_CHUNKS = 2, DOWN_CHUNKS = 1;

// Steps in flight per wavefront (DR): the weight slices of DR steps sit in
// registers (four 16-byte loads per lane and step), the activation rows of
// DR + 1 steps in the LDS ring.  Four steps (64 KB per workgroup) already
// exceed what the vector L1 keeps outstanding; a deeper ring only queues
// (measured: 8 steps were slightly slower than 4 on 64-row tiles, 2 much
// slower).
#ifndef TEMPO_DR64
#define TEMPO_DR64 4
#endif
#ifndef TEMPO_DR128
#define TEMPO_DR128 4
#endif
__host__ __device__ constexpr int gemm_dr(int bm) { return bm == 64 ? TEMPO_DR64 : bm <= 192 ? TEMPO_DR128 : 2; }
// Chunks are whole multiples of CQ steps for every tile size, so that the
// fixed summation order (the chunk boundaries) is the same whichever M-tile
// the rows land in; each DR divides CQ.
constexpr int CQ = 8;
static_assert(CQ % gemm_dr(64) == 0 && CQ % gemm_dr(128) == 0 && CQ % gemm_dr(192) == 0 && CQ % gemm_dr(256) == 0,
              "DR divides CQ");

// Work geometry; identical in the GEMM and in its fixup kernel.  Chunks are
// whole multiples of DR steps (the register ring is indexed by step mod DR at
// compile time); an item whose step count is not a multiple of DR ends in a
// few empty steps that load and multiply nothing.
struct Geo {
  int KT, SPC, C, SL;  // real steps per item; steps per chunk; chunks; steps of the last chunk (padded)
  int KTV;             // steps per item including the padding: (C - 1) * SPC + SL
  int groups, grp, j0, wpx, my_nb, nb_lo, items;
  int q0, q1;          // this workgroup's chunk range [q0, q1)
};

__host__ __device__ __forceinline__ int geo_groups(int NB, int grid) { return (NB % 8 == 0 && grid % 8 == 0) ? 8 : 1; }

// Ranges balance estimated time, not chunk counts: a chunk of an M-tile with
// m row blocks of 32 real rows costs W_BASE + m (a step's fixed work plus its
// MFMA and activation traffic per row block).  s_sw[s] holds the summed tile
// weights of slots before s (s_sw[S] = all tiles).
constexpr int W_BASE = 4;

template <int BM>
__device__ __forceinline__ int tile_weight(int rows) { return W_BASE + ((rows + 31) >> 5); }

// All threads of the block; ends with a barrier.  s_off / s_cnt must be ready.
// Wavefront 0 scans: lane l sums slots 4l..4l+3, then a shuffle scan.
template <int BM>
__device__ void build_slot_weights(const int32_t* s_off, const int32_t* s_cnt, int32_t* s_sw, int S) {
  static_assert(kMaxS <= 256, "four slots per lane");
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    int w[4], run = 0;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int s = 4 * l + i;
      int v = 0;
      if (s < S) {
        const int nt = (s_off[s + 1] - s_off[s]) / BM;
        v = nt > 0 ? (nt - 1) * tile_weight<BM>(BM) + tile_weight<BM>(s_cnt[s] - (nt - 1) * BM) : 0;
      }
      run += v;
      w[i] = run;
    }
    int incl = run;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int o = __shfl_up(incl, d);
      if (l >= d) incl += o;
    }
    const int excl = incl - run;
#pragma unroll
    for (int i = 0; i < 4; i++)
      if (4 * l + i < S) s_sw[4 * l + i + 1] = excl + w[i];
    if (l == 0) s_sw[0] = 0;
  }
  __syncthreads();
}

// First chunk of workgroup j of a group: the smallest chunk q whose weight
// prefix reaches j / wpx of the total.
template <int BM>
__device__ int range_lo(const Geo& g, int j, const int32_t* s_off, const int32_t* s_cnt, const int32_t* s_sw, int S) {
  const int U = g.items * g.C;
  if (j <= 0) return 0;
  if (j >= g.wpx) return U;
  const long long unit = (long long)g.my_nb * g.C;  // chunks per M-tile
  const long long T = unit * s_sw[S] * j / g.wpx;   // target weight
  // the first slot whose end lies beyond T
  int lo = 0, hi = S;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (unit * s_sw[mid + 1] > T) hi = mid;
    else lo = mid + 1;
  }
  if (lo == S) return U;
  const int nt = (s_off[lo + 1] - s_off[lo]) / BM;  // >= 1
  const long long wf = unit * tile_weight<BM>(BM);
  const long long rem = T - unit * s_sw[lo];
  const long long tf = min(rem / wf, (long long)(nt - 1));  // whole tiles of the slot before the target
  const int wt = tf < nt - 1 ? tile_weight<BM>(BM) : tile_weight<BM>(s_cnt[lo] - (nt - 1) * BM);
  const long long r = min((rem - tf * wf + wt - 1) / wt, unit);
  const long long q = (long long)(s_off[lo] / BM + tf) * unit + r;
  return (int)min(q, (long long)U);
}

template <int BM>
__device__ __forceinline__ Geo make_geo(int KT, int NB, int NT, int b, int grid, const int32_t* s_off,
                                        const int32_t* s_cnt, const int32_t* s_sw, int S, int cmax) {
  Geo g;
  constexpr int DR = gemm_dr(BM);
  g.KT = KT;
  const int cm = min(max(cmax, 1), CMAX);
  g.SPC = ((KT + cm - 1) / cm + CQ - 1) / CQ * CQ;
  g.C = (KT + g.SPC - 1) / g.SPC;
  g.SL = (KT - (g.C - 1) * g.SPC + DR - 1) / DR * DR;
  g.KTV = (g.C - 1) * g.SPC + g.SL;
  g.groups = geo_groups(NB, grid);
  g.grp = b % g.groups;
  g.j0 = b / g.groups;
  g.wpx = grid / g.groups;
  g.my_nb = NB / g.groups;
  g.nb_lo = g.grp * g.my_nb;
  g.items = NT * g.my_nb;
  g.q0 = range_lo<BM>(g, g.j0, s_off, s_cnt, s_sw, S);
  g.q1 = range_lo<BM>(g, g.j0 + 1, s_off, s_cnt, s_sw, S);
  return g;
}

// SwiGLU of one column: silu(g) * u, with silu(g) = g / (1 + e^-g) taken
// through the hardware reciprocal (v_rcp_f32, about 1 ulp).
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Partial tiles are stored lane-native: the 16 accumulator values of lane l
// of wavefront w for row block mi are 16 consecutive floats at
// ((mi * 4 + w) * 64 + l) * 16, i.e. four 16-byte stores per lane.  (Stores
// count in the same vmcnt as the ring's loads and may complete out of order
// with them, so the waits do not account for them: each store instruction
// issued makes the next waits conservative, and fewer is better.)
__device__ __forceinline__ int part_index(int mi, int w, int l, int i) { return ((mi * 4 + w) * 64 + l) * 16 + i; }

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>)
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

constexpr int GEMM_THREADS = 256;

// MX (fp8 only): the scales are powers of two and go to the MFMA as per-lane
// UE8M0 exponents (each lane supplies the activation row and the weight column
// it holds), so the products accumulate straight into the running sums.
template <bool FP8, int BM, bool GATEUP, bool MX = false>
__global__ __launch_bounds__(GEMM_THREADS, 1) void k_gemm(const GemmArgs p) {
  constexpr int MI = BM / 32;               // row blocks of 32
  constexpr int AG = BM / 32;               // activation 8-row groups per wavefront
  constexpr int DR = gemm_dr(BM);
  constexpr int EXTRA = FP8 ? BM * 4 + 128 : 0;  // fp8: BM activation scales, then 4 weight-scale words
  constexpr int NCOLS = GATEUP ? 64 : 128;  // output columns per item
  constexpr int BK = FP8 ? 128 : 64;        // contraction elements per step
  constexpr int NSL = DR + 1;               // activation ring slots
  constexpr int SLOT_MAX = BM * ROWB + EXTRA;
  constexpr int OUT_ES = GATEUP && FP8 ? 4 : 2;    // bytes per output element
  constexpr int ROW_OUT = NCOLS * OUT_ES;           // bytes of an item's output row: 128 or 256
  // output rows staged at a time (coalesced stores); 64 for 192-row tiles, whose
  // activation ring takes most of the LDS
  constexpr int STG_ROWS = BM % 128 == 0 ? 128 : 64;
  constexpr int STG_BYTES = STG_ROWS * ROW_OUT;
  constexpr int NROWT = nrowt_of(BM);

  __shared__ __attribute__((aligned(1024))) char ring[NSL * SLOT_MAX];
  __shared__ __attribute__((aligned(16))) char stg[STG_BYTES];
  __shared__ __attribute__((aligned(16))) int32_t s_rows[NROWT][BM];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];
  __shared__ int32_t s_sw[kMaxS + 1];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  for (int s = tid; s <= p.S; s += GEMM_THREADS) s_off[s] = p.slot_offsets[s];
  for (int s = tid; s < p.S; s += GEMM_THREADS) s_cnt[s] = p.slot_counts[s];
  __syncthreads();
  build_slot_weights<BM>(s_off, s_cnt, s_sw, p.S);

  // M-tiles in use, from the stage-1 offsets themselves (every P_s is a
  // multiple of BM), bounded by what the row buffers hold
  const int NT = __builtin_amdgcn_readfirstlane(max(0, min(s_off[p.S] / BM, p.max_tiles)));
  const Geo g = make_geo<BM>(p.Kd / BK, p.Nout / NCOLS, NT, blockIdx.x, gridDim.x, s_off, s_cnt, s_sw, p.S, p.cmax);
  if (g.q0 >= g.q1) {  // uniform: the whole workgroup leaves
    if (tid == 0) p.fix[(size_t)blockIdx.x * FIX_WORDS] = -1;
    return;
  }
  const int first_item = g.q0 / g.C;
  const int first_c = g.q0 - first_item * g.C;
  const int last_item = (g.q1 - 1) / g.C;
  const bool gather = p.row_src != nullptr;
  const uint32_t a_row_bytes = (uint32_t)p.Kd * (FP8 ? 1 : 2);
  const int lrow = lane >> 3, gchunk = (lane & 7) ^ (lane >> 3);
  const uint32_t ring_lds = lds_addr(ring);

  // row tables of the range's M-tiles (tiles past NROWT read row_src directly)
  const int tile_lo = first_item / g.my_nb;
  if (gather) {
    const int nt = min(last_item / g.my_nb - tile_lo + 1, NROWT);
    for (int t = wave; t < nt; t += 4)
      if (lane < BM / 4) lds_dma16(p.row_src + (size_t)(tile_lo + t) * BM + lane * 4, &s_rows[t][0]);
    __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(0));
  }
  barrier_nofence();

  // A ring slot holds the activation row groups of the range's largest M-tile
  // (and the step's scales for fp8).
  int amax = 0;
  for (int t = tile_lo + lane; t <= last_item / g.my_nb; t += 64) {
    const int sl = slot_of_row(s_off, p.S, t * BM);
    const int rows = min(BM, s_off[sl] + s_cnt[sl] - t * BM);
    amax = max(amax, rows);
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) amax = max(amax, __shfl_xor(amax, d));
  const int A_BYTES = __builtin_amdgcn_readfirstlane(((amax + 7) >> 3) * 1024);
  const int SLOT = A_BYTES + EXTRA;

  // steps of the range: SPC per chunk, SL for an item's last chunk
  const int F = (g.q1 - g.q0) * g.SPC - (g.q1 / g.C - g.q0 / g.C) * (g.SPC - g.SL);

  // ---- issue side: step iss of the range; its activation rows go to ring
  // slot iss % NSL, its weight slice to register set iss % DR ----
  int is_item = first_item, is_kt = first_c * g.SPC;
  int is_kt_end = min(g.KTV, (g.q1 - is_item * g.C) * g.SPC);
  int is_nvalid = 0;
  bool is_new = true;
  const char* a_base = p.A;
  const char* w_base = p.W;
  const char* as_base = nullptr;
  const char* ws_base = nullptr;
  uint32_t a_voff[AG];
  int iss = 0, is_slot = 0;
  i32x4 wr[DR][4];   // weight operands of the steps in flight

  auto setup_item = [&]() {
    const int tile = is_item / g.my_nb;
    const int nb = g.nb_lo + is_item - tile * g.my_nb;
    const int row0 = tile * BM;
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, p.S, row0));
    is_nvalid = __builtin_amdgcn_readfirstlane(min(BM, s_off[slot] + s_cnt[slot] - row0));
    w_base = slot_tensor(p.W, p.w_slot_bytes, p.wtab, p.wfield, slot) + (size_t)nb * g.KT * B_BYTES +
             wave * (B_BYTES / 4) + lane * 16;
    a_base = gather ? p.A : p.A + (size_t)row0 * a_row_bytes;
    const int tt = tile - tile_lo;
#pragma unroll
    for (int j = 0; j < AG; j++) {
      const int gi = wave + 4 * j;
      const int r = min(gi * 8 + lrow, is_nvalid - 1);
      uint32_t row = r;
      if (gather) {
        // (separate loads: one through a pointer that may be LDS or global
        // would be a generic load, whose wait drains the whole stream)
        int v;
        if (tt < NROWT) {
          v = s_rows[tt][r];
        } else {  // not reached when the host chose gathering: a plain load that waits for everything
          asm volatile("global_load_dword %0, %1, off\n\ts_waitcnt vmcnt(0)"
                       : "=v"(v)
                       : "v"(p.row_src + row0 + r)
                       : "memory");
        }
        row = max(v, 0);
      }
      a_voff[j] = row * a_row_bytes + gchunk * 16;
    }
    if (FP8) {
      as_base = reinterpret_cast<const char*>(p.As + row0);
      ws_base = slot_tensor(reinterpret_cast<const char*>(p.Wsp), p.ws_slot_floats * 4, p.wtab, p.sfield, slot) +
                (size_t)nb * g.KT * 16;
    }
    is_new = false;
  };

  // The four weight loads of a register set are issued on every call, also
  // past the end of the range and for the empty steps that pad an item (then
  // from one fixed 4 KB that stays in cache): the compiler counts the loads
  // issued after each set to place its waits, and a load skipped on some path
  // would make it wait for everything.
  const i32x4* const w_idle =
      reinterpret_cast<const i32x4*>(slot_tensor(p.W, p.w_slot_bytes, p.wtab, p.wfield, 0)) + lane;
  auto issue = [&](auto dd) {
    constexpr int d = decltype(dd)::value;
    const i32x4* wp = w_idle;
    if (iss < F) {
      if (is_new) setup_item();
      if (is_kt < g.KT) {
        const uint32_t sl = ring_lds + is_slot * SLOT;
        const char* ab = a_base + is_kt * ROWB;
#pragma unroll
        for (int j = 0; j < AG; j++) {
          const int gi = wave + 4 * j;
          if (gi * 8 < is_nvalid) lds_dma16s(ab, a_voff[j], sl + gi * 1024);
        }
        if (FP8) {
          if (wave == 3) {
            if (lane < BM / 4) lds_dma16s(as_base + (size_t)is_kt * p.as_ld * 4, lane * 16, sl + A_BYTES);
          } else if (wave == 2) {
            if (lane == 0) lds_dma16s(ws_base + is_kt * 16, 0, sl + A_BYTES + BM * 4);
          }
        }
        wp = reinterpret_cast<const i32x4*>(w_base + (size_t)is_kt * B_BYTES);
      }
      iss++;
      if (++is_slot == NSL) is_slot = 0;
      if (++is_kt == is_kt_end) {
        is_item++;
        is_kt = 0;
        is_kt_end = min(g.KTV, (g.q1 - is_item * g.C) * g.SPC);
        is_new = true;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; j++) wr[d][j] = __builtin_nontemporal_load(wp + j * 64);
  };

  // ---- consume side ----
  // A partial tile goes out lane-native (16-byte stores of 1 KB per
  // instruction); the lane index is laundered so that the compiler does not
  // keep every address live across the main loop.
  auto store_tile = [&](float* dst, const f32x16 (&v)[MI], int live) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int mi = 0; mi < MI; mi++)
      if (mi < live)
#pragma unroll
        for (int q = 0; q < 4; q++)
          *reinterpret_cast<float4*>(dst + part_index(mi, wave, ln, 4 * q)) =
              make_float4(v[mi][4 * q], v[mi][4 * q + 1], v[mi][4 * q + 2], v[mi][4 * q + 3]);
  };
  // Output rows staged in LDS (stg[r][NCOLS]) go out as whole rows, 16
  // bytes per lane, after a barrier (every wavefront staged its columns).
  auto flush_rows = [&](char* dst, size_t dst_stride, int nrows) {
    wait_lgkm0();
    barrier_nofence();
    constexpr int PER = ROW_OUT / 16;  // 16-byte pieces per row
    int t0 = tid;
    asm volatile("" : "+v"(t0));
#pragma unroll 2
    for (int idx = t0; idx < nrows * PER; idx += 256) {
      const int r = idx / PER, c = idx % PER;
      *reinterpret_cast<i32x4*>(dst + r * dst_stride + c * 16) = *reinterpret_cast<const i32x4*>(stg + r * ROW_OUT + c * 16);
    }
  };

  // Epilogue of a finished item: rows [r][NCOLS] into the staging area, then
  // out as whole rows (STG_ROWS rows at a time).
  auto finish = [&](const f32x16 (&v)[MI], int live, int nvalid, int row0, int nb) {
    const int rb = 4 * (lane >> 5);
#pragma unroll
    for (int h = 0; h < BM / STG_ROWS; h++) {
      if (h * STG_ROWS >= nvalid) break;
      if (h > 0) barrier_nofence();  // every wavefront is done reading the previous rows
#pragma unroll
      for (int mi = h * (STG_ROWS / 32); mi < (h + 1) * (STG_ROWS / 32); mi++) {
        if (mi >= live) break;
#pragma unroll
        for (int i = 0; i < 16; i++) {
          const int r = rb + (mi - h * (STG_ROWS / 32)) * 32 + 8 * (i >> 2) + (i & 3);
          if (GATEUP) {
            // lanes l and l ^ 16 hold the gate and the up value of one column
            const float up = __shfl_xor(v[mi][i], 16);
            if ((lane & 16) == 0) {
              const float hv = silu_mul(v[mi][i], up);
              const int o = r * NCOLS + wave * 16 + (lane & 15);
              if (FP8) reinterpret_cast<float*>(stg)[o] = hv;
              else reinterpret_cast<uint16_t*>(stg)[o] = f32_to_bf16_rne(hv);
            }
          } else {
            reinterpret_cast<uint16_t*>(stg)[r * NCOLS + wave * 32 + (lane & 31)] = f32_to_bf16_rne(v[mi][i]);
          }
        }
      }
      flush_rows(static_cast<char*>(p.C) + ((size_t)(row0 + h * STG_ROWS) * p.Nout + (size_t)nb * NCOLS) * OUT_ES,
                 (size_t)p.Nout * OUT_ES, min(nvalid - h * STG_ROWS, STG_ROWS));
    }
  };

  // the first DR steps (F is a multiple of DR)
  static_for<DR>([&](auto dd) { issue(dd); });

  // One step on ring slot st with weight set d: acc[mi] += A_mi W^T for the
  // live row blocks (mi < live; block 0 always is).
  auto compute = [&](auto dd, const char* st, f32x16(&acc)[MI], int live) {
    constexpr int d = decltype(dd)::value;
    const int bcol = lane & 31;
    if (!FP8) {
      // every fragment read of the step first, then the MFMAs (the scheduling
      // barrier keeps the reads from being spread between the MFMAs, which
      // would expose the LDS latency once per read)
      // (in groups of at most four row blocks, to bound the registers held)
      constexpr int GB = MI < 4 ? MI : 4;
#pragma unroll
      for (int m0 = 0; m0 < MI; m0 += GB) {
        if (m0 >= live) break;
        bf16x8 a[GB][4];
#pragma unroll
        for (int j = 0; j < GB; j++)
          if (m0 + j < live)
#pragma unroll
            for (int ks = 0; ks < 4; ks++)
              a[j][ks] = *reinterpret_cast<const bf16x8*>(st + swz((m0 + j) * 32 + bcol, 2 * ks + (lane >> 5)));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < GB; j++)
          if (m0 + j < live)
#pragma unroll
            for (int ks = 0; ks < 4; ks++)
              acc[m0 + j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  a[j][ks], reinterpret_cast<const bf16x8&>(wr[d][ks]), acc[m0 + j], 0, 0, 0);
      }
    } else {
      const float* sa_lds = reinterpret_cast<const float*>(st + A_BYTES);
      const float* sw_lds = sa_lds + BM;
      // gate/up: lanes with bit 4 clear hold gate columns, the others up columns
      const float sw = GATEUP ? sw_lds[(lane >> 4) & 1] : sw_lds[0];
      const i32x8 b0 = (i32x8){wr[d][0][0], wr[d][0][1], wr[d][0][2], wr[d][0][3],
                               wr[d][1][0], wr[d][1][1], wr[d][1][2], wr[d][1][3]};
      const i32x8 b1 = (i32x8){wr[d][2][0], wr[d][2][1], wr[d][2][2], wr[d][2][3],
                               wr[d][3][0], wr[d][3][1], wr[d][3][2], wr[d][3][3]};
      // MX: the exponent byte of a power-of-two fp32 scale is its UE8M0 code
      const int eb = MX ? (int)((__float_as_uint(sw) >> 23) & 0xFF) : 127;
#pragma unroll
      for (int mi = 0; mi < MI; mi++) {
        if (MX && mi < live) {
          const int r = mi * 32 + bcol;
          i32x8 a[2];
#pragma unroll
          for (int h = 0; h < 2; h++) {
            const int c = 4 * h + 2 * (lane >> 5);
            const i32x4 lo = *reinterpret_cast<const i32x4*>(st + swz(r, c));
            const i32x4 hi = *reinterpret_cast<const i32x4*>(st + swz(r, c + 1));
            a[h] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          }
          const int ea = (int)((__float_as_uint(sa_lds[r]) >> 23) & 0xFF);  // this lane's activation row
          acc[mi] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[0], b0, acc[mi], 0, 0, 0, ea, 0, eb);
          acc[mi] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[1], b1, acc[mi], 0, 0, 0, ea, 0, eb);
        } else if (!MX && mi < live) {
          const int r = mi * 32 + bcol;
          i32x8 a[2];
#pragma unroll
          for (int h = 0; h < 2; h++) {
            const int c = 4 * h + 2 * (lane >> 5);
            const i32x4 lo = *reinterpret_cast<const i32x4*>(st + swz(r, c));
            const i32x4 hi = *reinterpret_cast<const i32x4*>(st + swz(r, c + 1));
            a[h] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          }
          float4 sa4[4];
#pragma unroll
          for (int q = 0; q < 4; q++) sa4[q] = *reinterpret_cast<const float4*>(sa_lds + mi * 32 + 8 * q + 4 * (lane >> 5));
          f32x16 pp = {};
          pp = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[0], b0, pp, 0, 0, 0, 127, 0, 127);
          pp = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[1], b1, pp, 0, 0, 0, 127, 0, 127);
          const float sa[16] = {sa4[0].x, sa4[0].y, sa4[0].z, sa4[0].w, sa4[1].x, sa4[1].y, sa4[1].z, sa4[1].w,
                                sa4[2].x, sa4[2].y, sa4[2].z, sa4[2].w, sa4[3].x, sa4[3].y, sa4[3].z, sa4[3].w};
#pragma unroll
          for (int i = 0; i < 16; i++) acc[mi][i] += pp[i] * (sa[i] * sw);
        }
      }
    }
  };

  int k = 0, uc_slot = 0;
  uint64_t tstart = 0;
  // One piece of an item: the steps of one item inside this range.
#pragma unroll 1
  for (int ord = 0; k < F; ord++) {
    const int item = first_item + ord;
    const int tile = item / g.my_nb;
    const int nb = g.nb_lo + item - tile * g.my_nb;
    const int row0 = tile * BM;
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, p.S, row0));
    const int nvalid = __builtin_amdgcn_readfirstlane(min(BM, s_off[slot] + s_cnt[slot] - row0));
    const int live = (nvalid + 31) >> 5;
    const int c0 = ord == 0 ? first_c : 0;  // first chunk of the piece
    const int kt_end = min(g.KTV, (g.q1 - item * g.C) * g.SPC);
    const int n = kt_end - c0 * g.SPC;
    if (p.timing && tid == 0) tstart = __builtin_amdgcn_s_memrealtime();
    float* const part_mine = p.part + (size_t)blockIdx.x * CMAX * BM * PART_TILE;
    // running sum of the chunks of a piece that starts at chunk 0
    f32x16 R[MI];
#pragma unroll
    for (int mi = 0; mi < MI; mi++)
#pragma unroll
      for (int i = 0; i < 16; i++) R[mi][i] = 0.f;
#pragma unroll 1
    for (int c = c0, t = 0; t < n; c++) {
      const int steps = c == g.C - 1 ? g.SL : g.SPC;
      const int kt0 = c * g.SPC;
      f32x16 acc[MI];
#pragma unroll
      for (int mi = 0; mi < MI; mi++)
#pragma unroll
        for (int i = 0; i < 16; i++) acc[mi][i] = 0.f;
#pragma unroll 1
      for (int u = 0; u < steps; u += DR) {
        static_for<DR>([&](auto dd) {
          constexpr int d = decltype(dd)::value;
          // This step's loads are done once at most 4 (DR - 1) loads are
          // outstanding: every step issues its activation DMAs before its
          // four weight loads, each later step issues four weight loads,
          // and loads complete in order.  Then everyone's rows are in LDS.
          __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(4 * (DR - 1)));
          barrier_nofence();
          if (kt0 + u + d < g.KT) compute(dd, ring + uc_slot * SLOT, acc, live);
          if (++uc_slot == NSL) uc_slot = 0;
          // the next step for this register set, into the ring slot the
          // previous step left
          __builtin_amdgcn_sched_barrier(0);
          issue(dd);
          __builtin_amdgcn_sched_barrier(0);
        });
      }
      t += steps;
      k += steps;
      // end of a chunk: fold it into the running sum, or hand it to the fixup
      const bool piece_end = t == n;
      if (c0 > 0) {
        store_tile(part_mine + (size_t)(1 + c - c0) * BM * PART_TILE, acc, live);
      } else {
        if (c == 0) {
#pragma unroll
          for (int mi = 0; mi < MI; mi++) R[mi] = acc[mi];
        } else {
#pragma unroll
          for (int mi = 0; mi < MI; mi++)
            if (mi < live) R[mi] += acc[mi];
        }
        if (piece_end) {
          if (c == g.C - 1) {
            finish(R, live, nvalid, row0, nb);  // the whole item is here
          } else {
            store_tile(part_mine, R, live);  // running sum of chunks 0..c
          }
        }
      }
    }
    if (p.timing && tid == 0) {
      const uint64_t tend = __builtin_amdgcn_s_memrealtime();
      atomicMin(reinterpret_cast<unsigned long long*>(&p.t0[slot]), (unsigned long long)tstart);
      atomicMax(reinterpret_cast<unsigned long long*>(&p.t1[slot]), (unsigned long long)tend);
    }
  }


  // fixup record: if the last item of the range started here (chunk 0) and
  // continues past it, list where the later chunks' partial tiles are
  if (tid == 0) {
    int32_t* rec = p.fix + (size_t)blockIdx.x * FIX_WORDS;
    const int cf = last_item * g.C;
    if (cf >= g.q0 && g.q1 < cf + g.C) {
      const int tile = last_item / g.my_nb;
      const int row0 = tile * BM;
      const int slot = slot_of_row(s_off, p.S, row0);
      int n = 0, q = g.q1;
      for (int j = g.j0 + 1; j < g.wpx && q < cf + g.C; j++) {
        const int lo = range_lo<BM>(g, j, s_off, s_cnt, s_sw, p.S), hi = range_lo<BM>(g, j + 1, s_off, s_cnt, s_sw, p.S);
        for (; q < hi && q < cf + g.C; q++) rec[4 + n++] = (j * g.groups + g.grp) * CMAX + 1 + q - lo;
      }
      rec[1] = row0;
      rec[2] = g.nb_lo + last_item - tile * g.my_nb;
      rec[3] = min(BM, s_off[slot] + s_cnt[slot] - row0);
      rec[0] = n;
    } else {
      rec[0] = -1;
    }
  }
}

// Completes the items whose chunks were spread over several workgroups.  The
// GEMM workgroup b whose range holds chunk 0 of such an item left a record
// (row0, output block, real rows, the partial tiles of the later chunks in
// chunk order).  Workgroup b + gemm_grid * (4 mi + w) of this grid (grid =
// gemm_grid * BM / 8) takes what wavefront w held for row block mi: thread
// (l, q) adds float4 q of lane l of the running sum b stored and of every
// later chunk, in chunk order (all loads issued before the first add), then
// applies the epilogue of the GEMM to its 4 rows.  For gate/up the gate lane
// l (bit 4 clear) also reads the up lane l + 16; up lanes are idle.
template <bool FP8, int BM, bool GATEUP>
__global__ __launch_bounds__(256) void k_fixup(const GemmArgs p, int gemm_grid) {
  const int b = blockIdx.x % gemm_grid, mw = blockIdx.x / gemm_grid;
  const int mi = mw >> 2, w = mw & 3;
  const int32_t* rec = p.fix + (size_t)b * FIX_WORDS;
  const int nsrc = rec[0];
  if (nsrc < 0) return;
  const int row0 = rec[1], nb = rec[2], nvalid = rec[3];
  if (mi * 32 >= nvalid) return;
  const int l = threadIdx.x >> 2, q = threadIdx.x & 3;
  if (GATEUP && (l & 16)) return;
  const int rfirst = mi * 32 + 8 * q + 4 * (l >> 5);  // rows rfirst .. rfirst + 3
  if (rfirst >= nvalid) return;
  const size_t tile_elems = (size_t)BM * PART_TILE;
  const int og = part_index(mi, w, l, 4 * q), ou = part_index(mi, w, l + 16, 4 * q);
  const float* head = p.part + (size_t)b * CMAX * tile_elems;
  float4 xg[CMAX], xu[CMAX];
  xg[0] = *reinterpret_cast<const float4*>(head + og);
  if (GATEUP) xu[0] = *reinterpret_cast<const float4*>(head + ou);
#pragma unroll
  for (int i = 0; i < CMAX - 1; i++) {
    if (i < nsrc) {
      const float* t = p.part + (size_t)rec[4 + i] * tile_elems;
      xg[i + 1] = *reinterpret_cast<const float4*>(t + og);
      if (GATEUP) xu[i + 1] = *reinterpret_cast<const float4*>(t + ou);
    }
  }
  float4 g = xg[0], u = GATEUP ? xu[0] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int i = 1; i < CMAX; i++) {
    if (i <= nsrc) {
      g.x += xg[i].x, g.y += xg[i].y, g.z += xg[i].z, g.w += xg[i].w;
      if (GATEUP) u.x += xu[i].x, u.y += xu[i].y, u.z += xu[i].z, u.w += xu[i].w;
    }
  }
  const float gv[4] = {g.x, g.y, g.z, g.w}, uv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int e = 0; e < 4; e++) {
    const int r = rfirst + e;
    if (r >= nvalid) break;
    const size_t orow = (size_t)(row0 + r) * p.Nout;
    if (GATEUP) {
      const float h = silu_mul(gv[e], uv[e]);
      const int col = nb * 64 + w * 16 + (l & 15);
      if (FP8) static_cast<float*>(p.C)[orow + col] = h;
      else static_cast<uint16_t*>(p.C)[orow + col] = f32_to_bf16_rne(h);
    } else {
      static_cast<uint16_t*>(p.C)[orow + nb * 128 + w * 32 + (l & 31)] = f32_to_bf16_rne(gv[e]);
    }
  }
}

}  // namespace gemm
}  // namespace tempo
