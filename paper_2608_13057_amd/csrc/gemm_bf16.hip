// Stage 2, bf16: grouped expert FFN over the M-tile-padded slot groups.
//   gate/up:  h = silu(A W_gate^T) * (A W_up^T)   (A = x_perm rows of a slot)
//   down:     y_perm = h W2^T
// (Sec. 2.1: "gate/up, activation, down"; Sec. 2.2: the cost of an activated
// replica is streaming its weights, every extra M-tile re-uses them.)
//
// One persistent kernel per GEMM.  Work items are (M-tile, N-block) pairs; the
// tile count and the slot of each tile come from the stage-1 results in device
// memory (slot_offsets / slot_counts / header), so the launch needs no host
// round trip and has a fixed grid.  Workgroup b runs on XCD b mod 8 (the
// hardware's round-robin); each XCD owns a contiguous range of N-blocks, so
// the weight block of an N-block is fetched into one XCD's L2 and shared by
// every M-tile of the slot that runs there, and the activation tile is shared
// by the XCD's N-blocks.
//
// Tile: BM rows x 128 weight rows x 64 of the contraction per step, 256
// threads as 2 x 2 wavefronts, each wavefront (BM/2) x 64 outputs with
// v_mfma_f32_32x32x16_bf16 (lane layout verified on gfx950: A row / B column =
// lane % 32, 8 consecutive k per lane; accumulator element i of lane l is
// row 8*(i/4) + 4*(l/32) + i%4, column l % 32).  Operand tiles are staged
// global -> registers -> LDS with two LDS buffers; LDS rows are padded by 16
// bytes so the 16-byte fragment reads of 8 consecutive rows hit distinct banks.
// Rows past a slot's real count are never loaded (zero-filled in LDS) nor
// stored.  The gate/up instance puts gate columns n..n+63 and up columns
// n..n+63 in one tile so that each lane holds matching g and u values and
// SwiGLU runs in registers.
//
// Every output row is produced by the same instruction sequence (same K
// order) wherever it lands, so results do not depend on the plan's split.
#include "internal.h"

namespace tempo {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int BK = 64;
constexpr int BNW = 128;      // weight rows per tile
constexpr int LDS_ROW = BK + 8;  // bf16 elements per padded LDS row

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <int BM, bool GATEUP>
__global__ __launch_bounds__(256, 2) void k_gemm_bf16(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                      size_t w_slot_stride, uint16_t* __restrict__ C,
                                                      const int32_t* __restrict__ slot_counts,
                                                      const int32_t* __restrict__ slot_offsets, int S, int Kd,
                                                      int Nout, int up_off, int max_tiles,
                                                      const uint32_t* __restrict__ hdr, uint64_t* __restrict__ t0,
                                                      uint64_t* __restrict__ t1, int timing) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BNW * LDS_ROW];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int MI = BM / 64;  // 32-row blocks per wavefront
  constexpr int NCOLS = GATEUP ? 64 : 128;  // output columns per tile

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

  for (int it = j0; it < items; it += wpx) {
    const int tile = it / my_nb;
    const int nb = nb_lo + it % my_nb;
    // slot of this tile: largest s with s_off[s] <= tile*BM
    const int row0 = tile * BM;
    int lo = 0, hi = S;  // invariant: s_off[lo] <= row0 < s_off[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_off[mid] <= row0) lo = mid;
      else hi = mid;
    }
    const int slot = lo;
    const int nvalid = min(BM, s_off[slot] + s_cnt[slot] - row0);
    uint64_t tstart = 0;
    if (timing && tid == 0) tstart = __builtin_amdgcn_s_memrealtime();

    const uint16_t* __restrict__ Wsl = W + (size_t)slot * w_slot_stride;
    // global source rows of the B tile
    auto wrow = [&](int r) -> int {
      if (GATEUP) return r < 64 ? nb * 64 + r : up_off + nb * 64 + (r - 64);
      return nb * 128 + r;
    };

    constexpr int ACH = BM * BK / 8 / 256;   // 16-byte chunks per thread (A)
    constexpr int BCH = BNW * BK / 8 / 256;  // (B)
    uint4 ra[ACH], rb[BCH];
    auto gload = [&](int k0) {
#pragma unroll
      for (int i = 0; i < ACH; i++) {
        const int c = tid + 256 * i, r = c >> 3, kc = c & 7;
        if (r < nvalid) ra[i] = *reinterpret_cast<const uint4*>(A + (size_t)(row0 + r) * Kd + k0 + kc * 8);
        else ra[i] = make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < BCH; i++) {
        const int c = tid + 256 * i, r = c >> 3, kc = c & 7;
        rb[i] = *reinterpret_cast<const uint4*>(Wsl + (size_t)wrow(r) * Kd + k0 + kc * 8);
      }
    };
    auto lstore = [&](int buf) {
#pragma unroll
      for (int i = 0; i < ACH; i++) {
        const int c = tid + 256 * i, r = c >> 3, kc = c & 7;
        *reinterpret_cast<uint4*>(&sA[buf][r * LDS_ROW + kc * 8]) = ra[i];
      }
#pragma unroll
      for (int i = 0; i < BCH; i++) {
        const int c = tid + 256 * i, r = c >> 3, kc = c & 7;
        *reinterpret_cast<uint4*>(&sB[buf][r * LDS_ROW + kc * 8]) = rb[i];
      }
    };

    f32x16 acc[MI][2];
#pragma unroll
    for (int mi = 0; mi < MI; mi++)
#pragma unroll
      for (int j = 0; j < 2; j++)
#pragma unroll
        for (int i = 0; i < 16; i++) acc[mi][j][i] = 0.f;

    const int KT = Kd / BK;
    gload(0);
    __syncthreads();  // previous item's readers are done with buffer 0
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; kt++) {
      const int buf = kt & 1;
      if (kt + 1 < KT) gload((kt + 1) * BK);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ks++) {
        bf16x8 a[MI], b[2];
        const int kk = ks * 16 + (lane >> 5) * 8;
#pragma unroll
        for (int mi = 0; mi < MI; mi++)
          a[mi] = *reinterpret_cast<const bf16x8*>(
              &sA[buf][(wm * (BM / 2) + mi * 32 + (lane & 31)) * LDS_ROW + kk]);
#pragma unroll
        for (int j = 0; j < 2; j++) {
          const int brow = GATEUP ? (j * 64 + wn * 32) : (wn * 64 + j * 32);
          b[j] = *reinterpret_cast<const bf16x8*>(&sB[buf][(brow + (lane & 31)) * LDS_ROW + kk]);
        }
#pragma unroll
        for (int mi = 0; mi < MI; mi++)
#pragma unroll
          for (int j = 0; j < 2; j++)
            acc[mi][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[j], acc[mi][j], 0, 0, 0);
      }
      if (kt + 1 < KT) lstore(buf ^ 1);
      __syncthreads();
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
                     void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid, hipStream_t st) {
  const uint32_t* hdr = reinterpret_cast<const uint32_t*>(ws + L.header);
  uint64_t* t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  uint64_t* t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  uint16_t* h = reinterpret_cast<uint16_t*>(ws + L.h);
  const int grid = persistent_grid();
  const int max_tiles = L.row_cap / BM;
  hipLaunchKernelGGL((k_gemm_bf16<BM, true>), dim3(grid), dim3(256), 0, st,
                     static_cast<const uint16_t*>(d.x_perm), static_cast<const uint16_t*>(w.w13),
                     (size_t)2 * s.I * s.H, h, d.slot_counts, d.slot_offsets, s.S, s.H, s.I, s.I, max_tiles, hdr, t0,
                     t1, timing ? 1 : 0);
  if (mid && hipEventRecord(mid, st) != hipSuccess) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_gemm_bf16<BM, false>), dim3(grid), dim3(256), 0, st, h,
                     static_cast<const uint16_t*>(w.w2), (size_t)s.H * s.I, static_cast<uint16_t*>(y_perm),
                     d.slot_counts, d.slot_offsets, s.S, s.I, s.H, 0, max_tiles, hdr, t0, t1, timing ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_experts_bf16(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                               void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid, hipStream_t st) {
  if (s.m_tile == 128) return launch_bm<128>(s, d, w, y_perm, ws, L, timing, mid, st);
  if (s.m_tile == 64) return launch_bm<64>(s, d, w, y_perm, ws, L, timing, mid, st);
  return hipErrorInvalidValue;
}

}  // namespace tempo
