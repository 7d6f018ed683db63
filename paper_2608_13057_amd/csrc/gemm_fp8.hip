// Stage 2, fp8: grouped expert FFN with OCP e4m3 activations and weights and
// fp32 block scales (activations 1 x 128 along the contraction, weights
// 128 x 128), the DeepSeek-V3 / Qwen3-FP8 convention the paper's fp8 grouped
// GEMM runs (Sec. 2.2).
//   gate/up:  h = silu(g) * u with g, u = sum_kb (A_kb W_kb^T) * sA[row,kb] * sW[blk,kb]
//   requant:  h -> e4m3 with per-row 1 x 128 scales amax / 448 (saturating)
//   down:     y_perm = sum_kb (h_kb W2_kb^T) * sh[row,kb] * sW2[blk,kb]  -> bf16
//
// Same persistent, XCD-aware work split and direct-to-LDS ring as the bf16
// kernel (gemm_bf16.hip); one pipeline stage is one 128-element scale block
// of the contraction (128 bytes per row), multiplied with two
// v_mfma_scale_f32_32x32x64_f8f6f4 (e4m3 x e4m3, unit hardware scales) into a
// per-stage partial that is then scaled by sA[row] * sW and added to the fp32
// accumulator.  The activation scales of a stage are one contiguous column of
// the scale-block-major scale array, so they arrive in the stage with one DMA;
// the weight scales of an item are staged in LDS when the item starts.
#include "gemm_common.h"

namespace tempo {
namespace {

using namespace gemm;

typedef __attribute__((__vector_size__(8 * sizeof(int)))) int i32x8;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int BK = 128;  // e4m3 contraction elements per stage (128 bytes) = one scale block
constexpr int MAX_KT = 64;

template <int BM, bool GATEUP>
__global__ __launch_bounds__(256, 1) void k_gemm_fp8(const uint8_t* __restrict__ A, const float* __restrict__ As,
                                                     int as_ld, const uint8_t* __restrict__ W,
                                                     size_t w_slot_stride, const float* __restrict__ Ws,
                                                     int ws_rows, float* __restrict__ Cf, uint16_t* __restrict__ Cb,
                                                     const int32_t* __restrict__ slot_counts,
                                                     const int32_t* __restrict__ slot_offsets,
                                                     const int32_t* __restrict__ row_src, int S, int Kd,
                                                     int Nout, int max_tiles, const uint32_t* __restrict__ hdr,
                                                     uint64_t* __restrict__ t0, uint64_t* __restrict__ t1,
                                                     int timing) {
  constexpr int SA_BYTES = 1024;  // the stage's BM activation scales (<= 512 B), 1 KB aligned
  __shared__ __attribute__((aligned(1024))) char ring[RING_BYTES];
  __shared__ int32_t s_off[kMaxS + 1];
  __shared__ int32_t s_cnt[kMaxS];
  __shared__ float s_ws[2][MAX_KT];  // weight scales of the item's two row blocks, per stage

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int MI = BM / 64;
  constexpr int NCOLS = GATEUP ? 64 : 128;
  constexpr int AG = BM / 32;
  constexpr int BG = BNW / 32;

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
  const int lrow = lane >> 3, gchunk = (lane & 7) ^ (lane >> 3);

  for (int it = j0; it < items; it += wpx) {
    const int tile = it / my_nb;
    const int nb = nb_lo + it % my_nb;
    const int row0 = tile * BM;
    const int slot = slot_of_row(s_off, S, row0);
    const int nvalid = min(BM, s_off[slot] + s_cnt[slot] - row0);
    uint64_t tstart = 0;
    if (timing && tid == 0) tstart = __builtin_amdgcn_s_memrealtime();

    const uint8_t* __restrict__ Wsl = W + (size_t)slot * w_slot_stride;
    const uint8_t* srcA[AG];
    const uint8_t* srcB[BG];
    int nA = 0;
#pragma unroll
    for (int j = 0; j < AG; j++) {
      const int g = wave + 4 * j, r = g * 8 + lrow;
      // A row: the permuted row itself, or the source row it was routed from
      int ar = row0 + r;
      if (row_src) ar = (g * 8 < nvalid) ? max(row_src[row0 + min(r, nvalid - 1)], 0) : 0;
      srcA[j] = A + (size_t)ar * Kd + gchunk * 16;
      nA += (g * 8 < nvalid) ? 1 : 0;
    }
#pragma unroll
    for (int j = 0; j < BG; j++) {
      const int g = wave + 4 * j;
      srcB[j] = Wsl + ((size_t)nb * KT * BNW * BK) + g * 8 * BK + lane * 16;
    }
    // the stage's activation scales: BM contiguous floats of column kt, moved
    // by BM/4 lanes of the last wavefront
    const bool sa_loader = (wave == 3) && (lane < BM / 4);
    const float* srcS = As + row0 + lane * 4;
    const int L = BG + nA + (wave == 3 ? 1 : 0);

    const int a_groups = (nvalid + 7) >> 3;
    const int A_BYTES = a_groups * 8 * ROWB;
    const int STAGE = A_BYTES + B_BYTES + SA_BYTES;
    const int NS = min(NS_MAX, RING_BYTES / STAGE);
    const int mi_live = (nvalid - wm * (BM / 2) + 31) >> 5;

    auto issue = [&](int kt) {
      char* st = ring + (kt % NS) * STAGE;
#pragma unroll
      for (int j = 0; j < AG; j++) {
        const int g = wave + 4 * j;
        if (g * 8 < nvalid) lds_dma16(srcA[j] + kt * BK, st + g * 8 * ROWB);
      }
#pragma unroll
      for (int j = 0; j < BG; j++) {
        const int g = wave + 4 * j;
        lds_dma16(srcB[j] + (size_t)kt * BNW * BK, st + A_BYTES + g * 8 * ROWB);
      }
      if (wave == 3) {
        if (sa_loader) lds_dma16(srcS + (size_t)kt * as_ld, st + A_BYTES + B_BYTES);
      }
    };

    f32x16 acc[MI][2];
#pragma unroll
    for (int mi = 0; mi < MI; mi++)
#pragma unroll
      for (int j = 0; j < 2; j++)
#pragma unroll
        for (int i = 0; i < 16; i++) acc[mi][j][i] = 0.f;

    barrier_nofence();  // every wavefront is done with the ring and s_ws (previous item)
    // weight scales of the item's row blocks: gate/up -> gate block and up block; down -> one block
    {
      const int blk0 = GATEUP ? (nb * 64) / 128 : nb;
      const int blk1 = GATEUP ? (Nout + nb * 64) / 128 : nb;
      const float* ws_slot = Ws + (size_t)slot * ws_rows * KT;
      for (int i = tid; i < 2 * KT; i += 256)
        s_ws[i / KT][i % KT] = ws_slot[(size_t)(i < KT ? blk0 : blk1) * KT + i % KT];
      wait_lgkm0();  // the scale stores are in LDS before the first stage's barrier
    }
#pragma unroll
    for (int s = 0; s < NS - 1; s++)
      if (s < KT) issue(s);
    for (int kt = 0; kt < KT; kt++) {
      wait_vmcnt(L * min(NS - 2, KT - 1 - kt));
      barrier_nofence();
      if (kt + NS - 1 < KT) issue(kt + NS - 1);
      const char* st = ring + (kt % NS) * STAGE;
      const float* sa_lds = reinterpret_cast<const float*>(st + A_BYTES + B_BYTES);
      i32x8 b[2][2];
#pragma unroll
      for (int j = 0; j < 2; j++) {
        const int r = (GATEUP ? (j * 64 + wn * 32) : (wn * 64 + j * 32)) + (lane & 31);
#pragma unroll
        for (int h = 0; h < 2; h++) {
          const int c = 4 * h + 2 * (lane >> 5);
          const i32x4 lo = *reinterpret_cast<const i32x4*>(st + A_BYTES + swz(r, c));
          const i32x4 hi = *reinterpret_cast<const i32x4*>(st + A_BYTES + swz(r, c + 1));
          b[j][h] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
      }
      const float sw0 = s_ws[0][kt], sw1 = s_ws[GATEUP ? 1 : 0][kt];
#pragma unroll
      for (int mi = 0; mi < MI; mi++) {
        if (mi >= mi_live) continue;
        const int r = wm * (BM / 2) + mi * 32 + (lane & 31);
        i32x8 a[2];
#pragma unroll
        for (int h = 0; h < 2; h++) {
          const int c = 4 * h + 2 * (lane >> 5);
          const i32x4 lo = *reinterpret_cast<const i32x4*>(st + swz(r, c));
          const i32x4 hi = *reinterpret_cast<const i32x4*>(st + swz(r, c + 1));
          a[h] = (i32x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
        // activation scales of this lane's 16 accumulator rows (4 runs of 4)
        float sa[16];
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const float4 v =
              *reinterpret_cast<const float4*>(sa_lds + wm * (BM / 2) + mi * 32 + 8 * q + 4 * (lane >> 5));
          sa[4 * q] = v.x;
          sa[4 * q + 1] = v.y;
          sa[4 * q + 2] = v.z;
          sa[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int j = 0; j < 2; j++) {
          f32x16 p = {};
          p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[0], b[j][0], p, 0, 0, 0, 127, 0, 127);
          p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[1], b[j][1], p, 0, 0, 0, 127, 0, 127);
          const float sw = j == 0 ? sw0 : sw1;
#pragma unroll
          for (int i = 0; i < 16; i++) acc[mi][j][i] += p[i] * (sa[i] * sw);
        }
      }
    }

    // epilogue: gate/up -> SwiGLU in fp32 (quantised by k_quant_h); down -> bf16
#pragma unroll
    for (int mi = 0; mi < MI; mi++) {
#pragma unroll
      for (int i = 0; i < 16; i++) {
        const int r = wm * (BM / 2) + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        if (r >= nvalid) continue;
        if (GATEUP) {
          const float g = acc[mi][0][i], u = acc[mi][1][i];
          const int col = nb * 64 + wn * 32 + (lane & 31);
          Cf[(size_t)(row0 + r) * Nout + col] = g / (1.0f + __expf(-g)) * u;
        } else {
#pragma unroll
          for (int j = 0; j < 2; j++) {
            const int col = nb * 128 + wn * 64 + j * 32 + (lane & 31);
            Cb[(size_t)(row0 + r) * Nout + col] = f32_to_bf16_rne(acc[mi][j][i]);
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

// h (fp32, real rows) -> e4m3 with one fp32 scale per row and 128-column block:
// scale = amax / 448 (1 if the block is all zero), q = e4m3(h / scale) with
// round-to-nearest-even, magnitudes saturated at 448.  One wavefront per row,
// two columns per lane per block.  Scales are stored block-major.
__global__ __launch_bounds__(256) void k_quant_h(const float* __restrict__ h32, int I, int row_cap,
                                                 const int32_t* __restrict__ row_token,
                                                 const int32_t* __restrict__ slot_offsets, int S,
                                                 uint8_t* __restrict__ h8, float* __restrict__ h_scale) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= row_cap || row >= slot_offsets[S] || row_token[row] < 0) return;
  const float2* src = reinterpret_cast<const float2*>(h32 + (size_t)row * I);
  uint16_t* dst = reinterpret_cast<uint16_t*>(h8 + (size_t)row * I);
  for (int b = 0; b < I / 128; b++) {
    const float2 v = src[b * 64 + lane];
    float m = fmaxf(fabsf(v.x), fabsf(v.y));
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d));
    const float sc = m > 0.f ? m / 448.0f : 1.0f;
    const float q0 = fminf(fmaxf(v.x / sc, -448.f), 448.f), q1 = fminf(fmaxf(v.y / sc, -448.f), 448.f);
    dst[b * 64 + lane] = (uint16_t)(__builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false) & 0xFFFF);
    if (lane == 0) h_scale[(size_t)b * row_cap + row] = sc;
  }
}

template <int BM>
hipError_t launch_bm(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                     const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid,
                     hipStream_t st) {
  const uint32_t* hdr = reinterpret_cast<const uint32_t*>(ws + L.header);
  uint64_t* t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  uint64_t* t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  float* h32 = reinterpret_cast<float*>(ws + L.h32);
  uint8_t* h8 = reinterpret_cast<uint8_t*>(ws + L.h);
  float* hs = reinterpret_cast<float*>(ws + L.h_scale);
  const int grid = persistent_grid(1);
  const int max_tiles = L.row_cap / BM;
  hipLaunchKernelGGL((k_gemm_fp8<BM, true>), dim3(grid), dim3(256), 0, st,
                     static_cast<const uint8_t*>(x_rows ? x_rows : d.x_perm), d.x_perm_scale, L.row_cap,
                     static_cast<const uint8_t*>(w.w13), (size_t)2 * s.I * s.H, w.w13_scale, 2 * s.I / 128, h32,
                     nullptr, d.slot_counts, d.slot_offsets, x_rows ? d.row_token : nullptr, s.S, s.H, s.I, max_tiles,
                     hdr, t0, t1, timing ? 1 : 0);
  hipLaunchKernelGGL(k_quant_h, dim3(ceil_div(L.row_cap, 4)), dim3(256), 0, st, h32, s.I, L.row_cap, d.row_token,
                     d.slot_offsets, s.S, h8, hs);
  if (mid && hipEventRecord(mid, st) != hipSuccess) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_gemm_fp8<BM, false>), dim3(grid), dim3(256), 0, st, h8, hs, L.row_cap,
                     static_cast<const uint8_t*>(w.w2), (size_t)s.H * s.I, w.w2_scale, s.H / 128, nullptr,
                     static_cast<uint16_t*>(y_perm), d.slot_counts, d.slot_offsets, nullptr, s.S, s.I, s.H, max_tiles,
                     hdr, t0, t1, timing ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

bool experts_supported(const tempo_moe_shape& s) {
  if (s.dtype == TEMPO_FP8_E4M3) return s.H / 128 <= MAX_KT && s.I / 128 <= MAX_KT;
  return true;
}

hipError_t launch_experts_fp8(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, hipEvent_t mid,
                              hipStream_t st) {
  if (s.m_tile == 128) return launch_bm<128>(s, d, w, x_rows, y_perm, ws, L, timing, mid, st);
  if (s.m_tile == 64) return launch_bm<64>(s, d, w, x_rows, y_perm, ws, L, timing, mid, st);
  return hipErrorInvalidValue;
}

}  // namespace tempo
