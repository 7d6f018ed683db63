// Stage 2, bf16: the stream-K grouped GEMM of gemm_stream.h with bf16
// operands and fp32 accumulation; h is rounded to bf16 (round to nearest
// even) after SwiGLU, y_perm to bf16 after the down projection.
#include "gemm_stream.h"

namespace tempo {
namespace {

using namespace gemm;

template <int BM>
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
  char* h = ws + L.h;

  // gate/up + SwiGLU -> h [row_cap, I] bf16
  GemmArgs gu = a;
  gu.A = static_cast<const char*>(x_rows ? x_rows : d.x_perm);
  gu.row_src = x_rows ? d.row_token : nullptr;
  gu.W = static_cast<const char*>(w.w13);
  gu.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  gu.wfield = kFieldW13;
  gu.sfield = kFieldW13Scale;
  gu.w_slot_bytes = (size_t)2 * s.I * s.H * 2;
  gu.C = h;
  gu.Kd = s.H;
  gu.Nout = s.I;
  gu.cmax = GATEUP_CHUNKS;
  auto mark = [&](int i) { return !ev || !ev[i] || hipEventRecord(ev[i], st) == hipSuccess; };
  if (!mark(0)) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_gemm<false, BM, true>), dim3(grid), dim3(GEMM_THREADS), 0, st, gu);
  if (!mark(1)) return hipErrorLaunchFailure;
  hipLaunchKernelGGL((k_fixup<false, BM, true>), dim3(grid * (BM / 8)), dim3(256), 0, st, gu, grid);
  if (!mark(2)) return hipErrorLaunchFailure;

  // down -> y_perm [row_cap, H] bf16
  GemmArgs dn = a;
  dn.A = h;
  dn.W = static_cast<const char*>(w.w2);
  dn.wtab = reinterpret_cast<const uint64_t*>(w.slot_table);
  dn.wfield = kFieldW2;
  dn.sfield = kFieldW2Scale;
  dn.w_slot_bytes = (size_t)s.H * s.I * 2;
  dn.C = y_perm;
  dn.Kd = s.I;
  dn.Nout = s.H;
  dn.cmax = DOWN_CHUNKS;
  hipLaunchKernelGGL((k_gemm<false, BM, false>), dim3(grid), dim3(GEMM_THREADS), 0, st, dn);
  if (!mark(3)) return hipErrorLaunchFailure;
  // (with one chunk per item no down item is split: nothing to complete)
  if (dn.cmax > 1)
    hipLaunchKernelGGL((k_fixup<false, BM, false>), dim3(grid * (BM / 8)), dim3(256), 0, st, dn, grid);
  return hipGetLastError();
}

}  // namespace

bool experts_gather_rows(const tempo_moe_shape& s, const Layout& L) {
  // the large-tile kernels pack the token rows themselves
  if (experts_big_supported(s) || experts_big_f8_supported(s)) return true;
  // upper bound of the M-tiles one workgroup range of the gate/up GEMM spans
  const int grid = persistent_grid(1);
  const int NB = s.I / 64;
  const long long groups = geo_groups(NB, grid), wpx = grid / groups;
  // ranges balance weighted chunks; a range holds at most 1/wpx of the total
  // weight, which is largest when every tile is full, and its tiles weigh at
  // least W_BASE + 1 each
  const long long max_tiles = L.row_cap / s.m_tile;
  const long long wfull = W_BASE + s.m_tile / 32, wmin = W_BASE + 1;
  const long long tiles = (max_tiles * wfull + wpx * wmin - 1) / (wpx * wmin) + 2;
  return tiles <= nrowt_of(s.m_tile);
}

hipError_t launch_experts_bf16(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                               const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing, const hipEvent_t* ev,
                               hipStream_t st) {
  if (s.m_tile == 128) return launch_bm<128>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  if (s.m_tile == 64) return launch_bm<64>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  if (s.m_tile == 256) {
    if (experts_big_supported(s)) return launch_experts_big(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
    return launch_bm<256>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  }
  if (s.m_tile == 192) return launch_bm<192>(s, d, w, x_rows, y_perm, ws, L, timing, ev, st);
  return hipErrorInvalidValue;
}

}  // namespace tempo
