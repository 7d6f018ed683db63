// Stage 2, bf16, for 256-row M-tiles: the linear regime of the cost model,
// where a slot's rows are many and the per-token compute (beta, Eq. 1)
// dominates the weight streaming (Sec. 2.2).  Here the work is a plain dense
// contraction, so it is organised for MFMA throughput rather than for HBM
// streaming:
//
// * A work item is one (M-tile of 256 rows, 256 packed weight rows) pair;
//   items are handed out round-robin to a persistent grid (one workgroup per
//   CU).  There is no split of the contraction: each item accumulates its
//   steps in order, so the result of a row depends only on its own inputs.
// * Four wavefronts in a 2 x 2 arrangement each own a 128 x 128 block of the
//   item: 4 x 4 MFMA tiles of 32 x 32 (256 accumulator registers per lane,
//   kept in AGPRs).  Per 16-element sub-step a wavefront reads 4 activation
//   and 4 weight fragments from LDS for 16 MFMAs -- half the LDS bytes per
//   MFMA of the streaming kernel's 1 x 4 arrangement.
// * A step (128 bytes of every row: 32 KB of activation rows, 32 KB of
//   weights) goes from global memory into LDS by DMA; two stages, the next
//   step's DMA issued before the current step's MFMAs.  The packed weight
//   layout stores each 32-row piece in MFMA operand order, so a weight
//   fragment read is 1 KB of consecutive LDS bytes.
// * Epilogue: SwiGLU (gate/up) or the bf16 rounding (down) on the fp32 sums,
//   staged in LDS and written out as whole rows.
#include "gemm_stream.h"

namespace tempo {
namespace {

using namespace gemm;

constexpr int BIG_M = 256;                       // rows per item (the M-tile)
constexpr int BIG_N = 256;                       // packed weight rows per item (two blocks of 128)
constexpr int A_STAGE = BIG_M * ROWB;            // 32 KB of activation rows per step
constexpr int STAGE = A_STAGE + 2 * B_BYTES;     // + two 16 KB weight blocks

template <bool GATEUP>
__global__ __launch_bounds__(256, 1) void k_gemm_big(const GemmArgs p) {
  constexpr int NCOLS = GATEUP ? BIG_N / 2 : BIG_N;  // output columns per item
  constexpr int ROW_OUT = NCOLS * 2;                  // bf16 output bytes per row of an item
  static_assert(BIG_M * ROW_OUT <= 2 * STAGE, "staged output rows fit in the ring");
  __shared__ __attribute__((aligned(1024))) char ring[2 * STAGE];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;  // this wavefront's 128-row and 128-weight-row halves

  const int nt_hdr = (int)p.hdr[kHdrTiles];
  for (int s = tid; s <= p.S; s += 256) s_off[s] = p.slot_offsets[s];
  for (int s = tid; s < p.S; s += 256) s_cnt[s] = p.slot_counts[s];
  __syncthreads();
  const int NT = __builtin_amdgcn_readfirstlane(min(nt_hdr, p.max_tiles));
  const int KT = p.Kd / 64;       // steps of 64 bf16
  const int NBT = p.Nout / NCOLS;  // items per M-tile
  const int items = NT * NBT;
  const uint32_t a_row_bytes = (uint32_t)p.Kd * 2;
  const uint32_t ring_lds = lds_addr(ring);
  const int lrow = lane >> 3, gchunk = (lane & 7) ^ (lane >> 3);

#pragma unroll 1
  for (int it = blockIdx.x; it < items; it += gridDim.x) {
    const int tile = it / NBT, nbt = it - tile * NBT;
    const int row0 = tile * BIG_M;
    const int slot = __builtin_amdgcn_readfirstlane(slot_of_row(s_off, p.S, row0));
    const int nvalid = __builtin_amdgcn_readfirstlane(min(BIG_M, s_off[slot] + s_cnt[slot] - row0));
    uint64_t tstart = 0;
    if (p.timing && tid == 0) tstart = __builtin_amdgcn_s_memrealtime();

    // DMA sources: activation 8-row group g = wave + 4j (rows past the real
    // ones re-read the last real row); weight piece q = wave + 4j of the two
    // blocks' 32 1 KB pieces of a step
    const char* a_base = p.A + (size_t)row0 * a_row_bytes;
    uint32_t a_voff[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
      const int r = min((wave + 4 * j) * 8 + lrow, nvalid - 1);
      a_voff[j] = (uint32_t)r * a_row_bytes + gchunk * 16;
    }
    const char* w_base = p.W + (size_t)slot * p.w_slot_bytes + (size_t)(2 * nbt) * KT * B_BYTES;
    auto issue = [&](int k, int stg) {
      const uint32_t sl = ring_lds + stg * STAGE;
      const char* ab = a_base + k * ROWB;
#pragma unroll
      for (int j = 0; j < 8; j++) lds_dma16s(ab, a_voff[j], sl + (wave + 4 * j) * 1024);
#pragma unroll
      for (int j = 0; j < 8; j++) {
        const int q = wave + 4 * j;
        const char* bb = w_base + (size_t)(q >> 4) * KT * B_BYTES + (size_t)k * B_BYTES;
        lds_dma16s(bb, (q & 15) * 1024 + lane * 16, sl + A_STAGE + q * 1024);
      }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++)
#pragma unroll
        for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;

    barrier_nofence();  // the previous item's output rows have left the ring
    issue(0, 0);
#pragma unroll 1
    for (int k = 0; k < KT; k++) {
      const int stg = k & 1;
      barrier_nofence();  // every wavefront is done with step k - 1, whose stage step k + 1 reuses
      if (k + 1 < KT) {
        issue(k + 1, stg ^ 1);
        __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(16));  // this wavefront's loads of step k are done
      } else {
        __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(0));
      }
      barrier_nofence();  // and everyone's
      const char* st = ring + stg * STAGE;
#pragma unroll
      for (int ks = 0; ks < 4; ks++) {
        bf16x8 a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; i++)
          a[i] = *reinterpret_cast<const bf16x8*>(st + swz(128 * wm + 32 * i + (lane & 31), 2 * ks + (lane >> 5)));
#pragma unroll
        for (int j = 0; j < 4; j++)
          b[j] = *reinterpret_cast<const bf16x8*>(st + A_STAGE + wn * B_BYTES + j * 4096 + ks * 1024 + lane * 16);
#pragma unroll
        for (int i = 0; i < 4; i++)
#pragma unroll
          for (int j = 0; j < 4; j++) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    }

    // epilogue: rows [r][NCOLS] of bf16 into the ring, then out as whole rows
    barrier_nofence();  // every wavefront is done reading the last step
    const int rb = 4 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++)
#pragma unroll
        for (int e = 0; e < 16; e++) {
          const int r = 128 * wm + 32 * i + rb + 8 * (e >> 2) + (e & 3);
          if (GATEUP) {
            // lanes l and l ^ 16 hold the gate and the up value of one column
            const float up = __shfl_xor(acc[i][j][e], 16);
            if ((lane & 16) == 0) {
              const int col = 64 * wn + 16 * j + (lane & 15);
              reinterpret_cast<uint16_t*>(ring)[r * NCOLS + col] = f32_to_bf16_rne(silu_mul(acc[i][j][e], up));
            }
          } else {
            const int col = 128 * wn + 32 * j + (lane & 31);
            reinterpret_cast<uint16_t*>(ring)[r * NCOLS + col] = f32_to_bf16_rne(acc[i][j][e]);
          }
        }
    wait_lgkm0();
    barrier_nofence();
    {
      constexpr int PER = ROW_OUT / 16;  // 16-byte pieces per row
      char* dst = static_cast<char*>(p.C) + ((size_t)row0 * p.Nout + (size_t)nbt * NCOLS) * 2;
      const size_t stride = (size_t)p.Nout * 2;
      int t0 = tid;
      asm volatile("" : "+v"(t0));
#pragma unroll 2
      for (int idx = t0; idx < nvalid * PER; idx += 256) {
        const int r = idx / PER, c = idx % PER;
        *reinterpret_cast<i32x4*>(dst + r * stride + c * 16) = *reinterpret_cast<const i32x4*>(ring + r * ROW_OUT + c * 16);
      }
    }
    if (p.timing && tid == 0) {
      const uint64_t tend = __builtin_amdgcn_s_memrealtime();
      atomicMin(reinterpret_cast<unsigned long long*>(&p.t0[slot]), (unsigned long long)tstart);
      atomicMax(reinterpret_cast<unsigned long long*>(&p.t1[slot]), (unsigned long long)tend);
    }
  }
}

}  // namespace

bool experts_big_supported(const tempo_moe_shape& s) {
  return s.dtype == TEMPO_BF16 && s.m_tile == BIG_M && s.H % BIG_N == 0 && s.I % 128 == 0;
}

// Both GEMMs of stage 2 with 256 x 256 items (x_perm must hold the permuted
// rows: this kernel does not gather).
hipError_t launch_experts_big(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              void* y_perm, char* ws, const Layout& L, bool timing, const hipEvent_t* ev,
                              hipStream_t st) {
  const int grid = persistent_grid(1);
  GemmArgs a{};
  a.slot_counts = d.slot_counts;
  a.slot_offsets = d.slot_offsets;
  a.S = s.S;
  a.max_tiles = L.row_cap / BIG_M;
  a.hdr = reinterpret_cast<const uint32_t*>(ws + L.header);
  a.t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  a.t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  a.timing = timing ? 1 : 0;
  auto mark = [&](int i) { return !ev || !ev[i] || hipEventRecord(ev[i], st) == hipSuccess; };

  GemmArgs gu = a;
  gu.A = static_cast<const char*>(d.x_perm);
  gu.W = static_cast<const char*>(w.w13);
  gu.w_slot_bytes = (size_t)2 * s.I * s.H * 2;
  gu.C = ws + L.h;
  gu.Kd = s.H;
  gu.Nout = s.I;
  hipLaunchKernelGGL(k_gemm_big<true>, dim3(grid), dim3(256), 0, st, gu);
  if (!mark(0) || !mark(1)) return hipErrorLaunchFailure;

  GemmArgs dn = a;
  dn.A = ws + L.h;
  dn.W = static_cast<const char*>(w.w2);
  dn.w_slot_bytes = (size_t)s.H * s.I * 2;
  dn.C = y_perm;
  dn.Kd = s.I;
  dn.Nout = s.H;
  hipLaunchKernelGGL(k_gemm_big<false>, dim3(grid), dim3(256), 0, st, dn);
  if (!mark(2)) return hipErrorLaunchFailure;
  return hipGetLastError();
}

}  // namespace tempo
