// Stage 3: routing-weighted combine (Sec. 2.1: the per-token weighted sum of
// the expert outputs that follows the grouped GEMMs; on an EP group this is
// the partial sum the combine all-to-all adds up).
//   y[t] = sum_{k ascending, pair_row[t,k] >= 0} topk_w[t,k] * y_perm[pair_row[t,k]]
// fp32 accumulation, one bf16 rounding at the end; rows t >= T_valid and rows
// without a local pair are zero.  16-byte loads and stores (8 bf16 per lane);
// HBM-bound.
#include "internal.h"

namespace tempo {
namespace {

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// One wavefront per (token, 512-column segment): each lane owns 8 columns,
// reads the token's K rows and weights (one load each, issued together) and
// then the K 16-byte pieces of y_perm at once, so the kernel waits on two
// memory latencies whatever K is.
constexpr int kCombKU = 8;  // pairs whose loads are in flight together

__global__ __launch_bounds__(256) void k_combine(int T, int T_valid, int K, int H, const int32_t* __restrict__ pair_row,
                                                 const float* __restrict__ topk_w,
                                                 const uint16_t* __restrict__ y_perm, uint16_t* __restrict__ y,
                                                 int S, const int32_t* __restrict__ slot_counts,
                                                 const uint64_t* __restrict__ t0, const uint64_t* __restrict__ t1,
                                                 uint64_t* __restrict__ slot_time_ns) {
  const int lane = threadIdx.x & 63;
  const int nseg = (H + 511) / 512;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (slot_time_ns && blockIdx.x == 0)
    for (int s = threadIdx.x; s < S; s += 256)
      slot_time_ns[s] = slot_counts[s] > 0 ? (t1[s] - t0[s]) * 10ull : 0ull;  // 100 MHz counter
  const int t = wid / nseg, seg = wid - t * nseg;
  if (t >= T) return;
  const int c = seg * 64 + lane;  // this lane's 16-byte chunk (8 columns)
  const bool own = c < H / 8;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (t < T_valid) {
    for (int k0 = 0; k0 < K; k0 += kCombKU) {
      int r[kCombKU];
      float wk[kCombKU];
#pragma unroll
      for (int u = 0; u < kCombKU; u++) {
        const bool ok = k0 + u < K;
        r[u] = ok ? pair_row[(size_t)t * K + k0 + u] : -1;
        wk[u] = ok ? topk_w[(size_t)t * K + k0 + u] : 0.f;
      }
      uint4 v[kCombKU];
#pragma unroll
      for (int u = 0; u < kCombKU; u++)
        if (r[u] >= 0 && own) v[u] = *reinterpret_cast<const uint4*>(y_perm + (size_t)r[u] * H + c * 8);
      // ascending k: the fp32 sum is formed in the order of the definition
#pragma unroll
      for (int u = 0; u < kCombKU; u++) {
        if (r[u] < 0 || !own) continue;
        const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int q = 0; q < 4; q++) {
          acc[2 * q] += wk[u] * __uint_as_float(w4[q] << 16);
          acc[2 * q + 1] += wk[u] * __uint_as_float(w4[q] & 0xFFFF0000u);
        }
      }
    }
  }
  if (!own) return;
  uint4 o;
  o.x = (uint32_t)f32_to_bf16_rne(acc[0]) | ((uint32_t)f32_to_bf16_rne(acc[1]) << 16);
  o.y = (uint32_t)f32_to_bf16_rne(acc[2]) | ((uint32_t)f32_to_bf16_rne(acc[3]) << 16);
  o.z = (uint32_t)f32_to_bf16_rne(acc[4]) | ((uint32_t)f32_to_bf16_rne(acc[5]) << 16);
  o.w = (uint32_t)f32_to_bf16_rne(acc[6]) | ((uint32_t)f32_to_bf16_rne(acc[7]) << 16);
  *reinterpret_cast<uint4*>(y + (size_t)t * H + c * 8) = o;
}

}  // namespace

hipError_t launch_combine(const tempo_moe_shape& s, const int32_t* pair_row, const float* topk_w, const void* y_perm,
                          void* y, const int32_t* slot_counts, const uint64_t* t0, const uint64_t* t1,
                          uint64_t* slot_time_ns, hipStream_t st) {
  const int waves = s.T * ((s.H + 511) / 512);
  hipLaunchKernelGGL(k_combine, dim3(ceil_div(waves, 4)), dim3(256), 0, st, s.T, s.T_valid, s.K, s.H, pair_row, topk_w,
                     static_cast<const uint16_t*>(y_perm), static_cast<uint16_t*>(y), s.S, slot_counts, t0, t1,
                     slot_time_ns);
  return hipGetLastError();
}

}  // namespace tempo
