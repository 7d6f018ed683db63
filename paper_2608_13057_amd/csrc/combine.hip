// Stage 3: routing-weighted combine (Sec. 2.1: the per-token weighted sum of
// the expert outputs that follows the grouped GEMMs; on an EP group this is
// the partial sum the combine all-to-all adds up).
//   y[t] = sum_{k ascending, pair_row[t,k] >= 0} topk_w[t,k] * y_perm[pair_row[t,k]]
// fp32 accumulation, one bf16 rounding at the end; rows t >= T_valid and rows
// without a local pair are zero.  One wavefront per token row, 16-byte loads
// and stores (8 bf16 per lane), up to 8 loads per lane in flight; HBM-bound.
#include "internal.h"

namespace tempo {
namespace {

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ __launch_bounds__(256) void k_combine(int T, int T_valid, int K, int H, const int32_t* __restrict__ pair_row,
                                                 const float* __restrict__ topk_w,
                                                 const uint16_t* __restrict__ y_perm, uint16_t* __restrict__ y,
                                                 int S, const int32_t* __restrict__ slot_counts,
                                                 const uint64_t* __restrict__ t0, const uint64_t* __restrict__ t1,
                                                 uint64_t* __restrict__ slot_time_ns) {
  __shared__ int32_t s_row[4][kMaxK];
  __shared__ float s_w[4][kMaxK];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wv;
  if (slot_time_ns && blockIdx.x == 0)
    for (int s = threadIdx.x; s < S; s += 256)
      slot_time_ns[s] = slot_counts[s] > 0 ? (t1[s] - t0[s]) * 10ull : 0ull;  // 100 MHz counter
  if (t >= T) return;
  // the token's local pairs in ascending k, compacted per wavefront (every
  // lane reads all of them below, also lanes that own no column)
  int row = -1;
  float wt = 0.f;
  if (lane < K && t < T_valid) {
    row = pair_row[(size_t)t * K + lane];
    wt = topk_w[(size_t)t * K + lane];
  }
  const uint64_t m = __ballot(row >= 0);
  const int nv = __popcll(m);
  if (row >= 0) {
    const int pos = __popcll(m & ((1ull << lane) - 1ull));
    s_row[wv][pos] = row;
    s_w[wv][pos] = wt;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  uint4* __restrict__ yo = reinterpret_cast<uint4*>(y + (size_t)t * H);
  const int nch = H / 8;
  constexpr int U = 8;  // 16-byte chunks per lane in flight
  for (int c0 = lane; c0 < nch; c0 += 64 * U) {
    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; u++)
#pragma unroll
      for (int q = 0; q < 8; q++) acc[u][q] = 0.f;
    for (int j = 0; j < nv; j++) {
      const int r = s_row[wv][j];
      const float wk = s_w[wv][j];
      const uint4* __restrict__ src = reinterpret_cast<const uint4*>(y_perm + (size_t)r * H);
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; u++)
        if (c0 + u * 64 < nch) v[u] = src[c0 + u * 64];
#pragma unroll
      for (int u = 0; u < U; u++) {
        const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int q = 0; q < 4; q++) {
          acc[u][2 * q] += wk * __uint_as_float(w4[q] << 16);
          acc[u][2 * q + 1] += wk * __uint_as_float(w4[q] & 0xFFFF0000u);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; u++) {
      if (c0 + u * 64 >= nch) continue;
      uint4 o;
      o.x = (uint32_t)f32_to_bf16_rne(acc[u][0]) | ((uint32_t)f32_to_bf16_rne(acc[u][1]) << 16);
      o.y = (uint32_t)f32_to_bf16_rne(acc[u][2]) | ((uint32_t)f32_to_bf16_rne(acc[u][3]) << 16);
      o.z = (uint32_t)f32_to_bf16_rne(acc[u][4]) | ((uint32_t)f32_to_bf16_rne(acc[u][5]) << 16);
      o.w = (uint32_t)f32_to_bf16_rne(acc[u][6]) | ((uint32_t)f32_to_bf16_rne(acc[u][7]) << 16);
      yo[c0 + u * 64] = o;
    }
  }
}

}  // namespace

hipError_t launch_combine(const tempo_moe_shape& s, const int32_t* pair_row, const float* topk_w, const void* y_perm,
                          void* y, const int32_t* slot_counts, const uint64_t* t0, const uint64_t* t1,
                          uint64_t* slot_time_ns, hipStream_t st) {
  hipLaunchKernelGGL(k_combine, dim3(ceil_div(s.T, 4)), dim3(256), 0, st, s.T, s.T_valid, s.K, s.H, pair_row, topk_w,
                     static_cast<const uint16_t*>(y_perm), static_cast<uint16_t*>(y), s.S, slot_counts, t0, t1,
                     slot_time_ns);
  return hipGetLastError();
}

}  // namespace tempo
