// Stage 3: routing-weighted combine (Sec. 2.1: the per-token weighted sum of
// the expert outputs that follows the grouped GEMMs; on an EP group this is
// the partial sum the combine all-to-all adds up).
//   y[t] = sum_{k ascending, pair_row[t,k] >= 0} topk_w[t,k] * y_perm[pair_row[t,k]]
// fp32 accumulation, one bf16 rounding at the end; rows t >= T_valid and rows
// without a local pair are zero.  One wavefront per token row, 16-byte loads
// and stores (8 bf16 per lane), HBM-bound.
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
  // the token's K rows and weights, staged per wavefront (every lane of the
  // wavefront reads all K of them below, also lanes that own no column)
  if (lane < K) {
    const bool ok = t < T_valid;
    s_row[wv][lane] = ok ? pair_row[(size_t)t * K + lane] : -1;
    s_w[wv][lane] = ok ? topk_w[(size_t)t * K + lane] : 0.f;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  uint4* __restrict__ yo = reinterpret_cast<uint4*>(y + (size_t)t * H);
  for (int c = lane; c < H / 8; c += 64) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < K; k++) {
      const int r = s_row[wv][k];
      const float wk = s_w[wv][k];
      if (r < 0) continue;
      const uint4 v = *reinterpret_cast<const uint4*>(y_perm + (size_t)r * H + c * 8);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; q++) {
        acc[2 * q] += wk * __uint_as_float(u[q] << 16);
        acc[2 * q + 1] += wk * __uint_as_float(u[q] & 0xFFFF0000u);
      }
    }
    uint4 o;
    o.x = (uint32_t)f32_to_bf16_rne(acc[0]) | ((uint32_t)f32_to_bf16_rne(acc[1]) << 16);
    o.y = (uint32_t)f32_to_bf16_rne(acc[2]) | ((uint32_t)f32_to_bf16_rne(acc[3]) << 16);
    o.z = (uint32_t)f32_to_bf16_rne(acc[4]) | ((uint32_t)f32_to_bf16_rne(acc[5]) << 16);
    o.w = (uint32_t)f32_to_bf16_rne(acc[6]) | ((uint32_t)f32_to_bf16_rne(acc[7]) << 16);
    yo[c] = o;
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
