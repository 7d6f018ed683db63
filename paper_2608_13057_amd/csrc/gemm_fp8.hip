// Stage 2, fp8: the stream-K grouped GEMM of gemm_stream.h with OCP e4m3
// activations and weights and fp32 block scales (activations 1 x 128 along
// the contraction, weights 128 x 128), the DeepSeek-V3 / Qwen3-FP8 convention
// the paper's fp8 grouped GEMM runs (Sec. 2.2).
//   gate/up:  h = silu(g) * u with g, u = sum_kb (A_kb W_kb^T) * sA[row,kb] * sW[blk,kb]
//   requant:  h -> e4m3 with per-row 1 x 128 scales amax / 448 (saturating;
//             rounded up to a power of two for the UE8M0 variant, whose GEMMs
//             apply the scales in the MFMA's block scaling)
//   down:     y_perm = sum_kb (h_kb W2_kb^T) * sh[row,kb] * sW2[blk,kb]  -> bf16
// One pipeline step is one 128-element scale block of the contraction.
#include <algorithm>

#include "gemm_stream.h"

namespace tempo {
namespace {

using namespace gemm;

// h (fp32, real rows) -> e4m3 with one fp32 scale per row and 128-column block:
// scale = amax / 448 (1 if the block is all zero), q = e4m3(h / scale) with
// round-to-nearest-even, magnitudes saturated at 448.  One wavefront per row,
// two columns per lane per block; the loads of up to 16 blocks are issued
// together before their reductions, so a row waits for one memory latency
// per 16 blocks rather than one per block.  Scales are stored block-major.
// MX: the scale is rounded up to a power of two (UE8M0), the smallest one at
// least amax / 448.
template <bool MX>
__global__ __launch_bounds__(256) void k_quant_h(const float* __restrict__ h32, int I, int row_cap,
                                                 const int32_t* __restrict__ row_token,
                                                 const int32_t* __restrict__ slot_offsets, int S,
                                                 uint8_t* __restrict__ h8, float* __restrict__ h_scale) {
  // a fixed grid walks the rows in use (one wavefront per row): a grid sized
  // for row_cap would be mostly workgroups that exit at once
  const int lane = threadIdx.x & 63;
  const int used = min(row_cap, slot_offsets[S]);
#pragma unroll 1
  for (int row = blockIdx.x * 4 + (threadIdx.x >> 6); row < used; row += gridDim.x * 4) {
    if (row_token[row] < 0) continue;
    const float2* src = reinterpret_cast<const float2*>(h32 + (size_t)row * I);
    uint16_t* dst = reinterpret_cast<uint16_t*>(h8 + (size_t)row * I);
    constexpr int NBL = 16;  // blocks loaded together
    const int NB = I / 128;
#pragma unroll 1
    for (int b0 = 0; b0 < NB; b0 += NBL) {
      float2 vb[NBL];
#pragma unroll
      for (int k = 0; k < NBL; k++) vb[k] = b0 + k < NB ? src[(b0 + k) * 64 + lane] : make_float2(0.f, 0.f);
#pragma unroll
      for (int k = 0; k < NBL; k++) {
        const int b = b0 + k;
        if (b >= NB) break;
        const float2 v = vb[k];
        float m = fmaxf(fabsf(v.x), fabsf(v.y));
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d));
        float sc = m > 0.f ? m / 448.0f : 1.0f;
        if (MX && m > 0.f) {
          uint32_t bits = __float_as_uint(sc);
          if (bits & 0x7FFFFFu) bits = (bits & 0xFF800000u) + 0x800000u;  // next power of two up
          sc = __uint_as_float(bits);
        }
        const float q0 = fminf(fmaxf(v.x / sc, -448.f), 448.f), q1 = fminf(fmaxf(v.y / sc, -448.f), 448.f);
        dst[b * 64 + lane] = (uint16_t)(__builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false) & 0xFFFF);
        if (lane == 0) h_scale[(size_t)b * row_cap + row] = sc;
      }
    }
  }
}

template <int BM, bool MX>
hipError_t launch_bm(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                     const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, const hipEvent_t* ev,
                     hipStream_t st) {
  const int grid = persistent_grid(1);
  GemmArgs a{};
  a.as_ld = L.row_cap;
  a.part = reinterpret_cast<float*>(ws + L.part);
  a.fix = reinterpret_cast<int32_t*>(ws + L.fix);
  a.slot_counts = d.slot_counts;
  a.slot_offsets = d.slot_offsets;
  a.S = s.S;
  a.max_tiles = L.row_cap / BM;
  a.t0 = reinterpret_cast<uint64_t*>(ws + L.slot_t0);
  a.t1 = reinterpret_cast<uint64_t*>(ws + L.slot_t1);
  a.timing = timing ? 1 : 0;
  float* h32 = reinterpret_cast<float*>(ws + L.h32);
  uint8_t* h8 = reinterpret_cast<uint8_t*>(ws + L.h);
  float* hs = reinterpret_cast<float*>(ws + L.h_scale);

  // gate/up + SwiGLU -> h32 [row_cap, I] fp32
  GemmArgs gu = a;
  gu.A = static_cast<const char*>(x_rows ? x_rows : d.x_perm);
  gu.row_src = x_rows ? d.row_token : nullptr;
  gu.As = d.x_perm_scale;
  gu.W = static_cast<const char*>(w.w13);
  gu.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  gu.wfield = kFieldW13;
  gu.sfield = kFieldW13Scale;
  gu.w_slot_bytes = (size_t)2 * s.I * s.H;
  gu.Wsp = w.w13_scale;
  gu.ws_slot_floats = (size_t)(s.I / 64) * (s.H / 128) * 4;
  gu.C = h32;
  gu.Kd = s.H;
  gu.Nout = s.I;
  gu.cmax = GATEUP_CHUNKS;
  auto mark = [&](int i) { return !ev || !ev[i] || hipEventRecord(ev[i], st) == hipSuccess; };
  if (!mark(0)) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_gemm<true, BM, true, MX>), dim3(grid), dim3(GEMM_THREADS), 0, st, gu);
  if (!mark(1)) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_fixup<true, BM, true>), dim3(grid * (BM / 8)), dim3(256), 0, st, gu, grid);
  hipLaunchKernelGGL(k_quant_h<MX>, dim3(std::min(ceil_div(L.row_cap, 4), persistent_grid(8))), dim3(256), 0, st, h32, s.I, L.row_cap, d.row_token,
                     d.slot_offsets, s.S, h8, hs);
  if (!mark(2)) return hipErrorLaunchFailure;

  // down -> y_perm [row_cap, H] bf16
  GemmArgs dn = a;
  dn.A = reinterpret_cast<const char*>(h8);
  dn.As = hs;
  dn.W = static_cast<const char*>(w.w2);
  dn.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  dn.wfield = kFieldW2;
  dn.sfield = kFieldW2Scale;
  dn.w_slot_bytes = (size_t)s.H * s.I;
  dn.Wsp = w.w2_scale;
  dn.ws_slot_floats = (size_t)(s.H / 128) * (s.I / 128) * 4;
  dn.C = y_perm;
  dn.Kd = s.I;
  dn.Nout = s.H;
  dn.cmax = DOWN_CHUNKS;
  hipLaunchKernelGGL((k_gemm<true, BM, false, MX>), dim3(grid), dim3(GEMM_THREADS), 0, st, dn);
  if (!mark(3)) return hipErrorLaunchFailure;
  // (with one chunk per item no down item is split: nothing to complete)
  if (dn.cmax > 1)
    hipLaunchKernelGGL((k_fixup<true, BM, false>), dim3(grid * (BM / 8)), dim3(256), 0, st, dn, grid);
  return hipGetLastError();
}

}  // namespace

bool experts_supported(const tempo_moe_shape&) { return true; }

bool experts_reads_token_scales(const tempo_moe_shape& s) { return experts_big_f8_supported(s); }

hipError_t launch_experts_fp8(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              const void* x_rows, const float* x_rows_scale, void* y_perm, char* ws, const Layout& L,
                              bool timing, const hipEvent_t* ev, hipStream_t st) {
  if (s.dtype == TEMPO_FP8_E4M3_UE8M0) {
    if (experts_big_f8_supported(s))
      return launch_experts_big_f8(s, d, w, x_rows, x_rows_scale, y_perm, ws, L, timing, ev, st);
    if (s.m_tile == 128) return launch_bm<128, true>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
    if (s.m_tile == 64) return launch_bm<64, true>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
    if (s.m_tile == 256) return launch_bm<256, true>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
    if (s.m_tile == 192) return launch_bm<192, true>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
    return hipErrorInvalidValue;
  }
  if (s.m_tile == 128) return launch_bm<128, false>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  if (s.m_tile == 64) return launch_bm<64, false>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  if (s.m_tile == 256) return launch_bm<256, false>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  if (s.m_tile == 192) return launch_bm<192, false>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  return hipErrorInvalidValue;
}

}  // namespace tempo
