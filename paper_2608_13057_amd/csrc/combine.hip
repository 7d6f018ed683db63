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

// Two fp32 values as bf16 (round to nearest even) in one word, lo in the
// low half: gfx950's packed conversion.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// One wavefront per (token, 512-column segment): each lane owns 8 columns.
// The token is uniform over the wavefront, so its K row indices and weights
// are scalar loads and the skip of a pair without a local row is a uniform
// branch; the K 16-byte pieces of y_perm are then loaded together, so the
// kernel waits on two memory latencies whatever K is.  Lanes past the end of
// a short row load a valid piece and store nothing.
constexpr int kCombKU = 8;  // pairs whose loads are in flight together

__global__ __launch_bounds__(256) void k_combine(int T, int T_valid, int K, int H, const int32_t* __restrict__ pair_row,
                                                 const float* __restrict__ topk_w,
                                                 const uint16_t* __restrict__ y_perm, uint16_t* __restrict__ y,
                                                 int S, const int32_t* __restrict__ slot_counts,
                                                 const uint64_t* __restrict__ t0, const uint64_t* __restrict__ t1,
                                                 uint64_t* __restrict__ slot_time_ns) {
  const int lane = threadIdx.x & 63;
  const int nseg = (H + 511) / 512;
  const int wid = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  if (slot_time_ns && blockIdx.x == 0)
    for (int s = threadIdx.x; s < S; s += 256)
      slot_time_ns[s] = slot_counts[s] > 0 ? (t1[s] - t0[s]) * 10ull : 0ull;  // 100 MHz counter
  const int t = wid / nseg, seg = wid - t * nseg;
  if (t >= T) return;
  const int c = seg * 64 + lane;  // this lane's 16-byte chunk (8 columns)
  const bool own = c < H / 8;
  const int cl = own ? c : 0;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (t < T_valid) {
    for (int k0 = 0; k0 < K; k0 += kCombKU) {
      int r[kCombKU];
      float wk[kCombKU];
      const int32_t* pr = pair_row + (size_t)t * K + k0;
      const float* pw = topk_w + (size_t)t * K + k0;
      if (k0 + kCombKU <= K) {  // (a whole group: one scalar load of each array)
#pragma unroll
        for (int u = 0; u < kCombKU; u++) {
          r[u] = __builtin_amdgcn_readfirstlane(pr[u]);
          wk[u] = pw[u];
        }
      } else {
#pragma unroll
        for (int u = 0; u < kCombKU; u++) {
          const bool ok = k0 + u < K;
          r[u] = ok ? __builtin_amdgcn_readfirstlane(pr[u]) : -1;
          wk[u] = ok ? pw[u] : 0.f;
        }
      }
      uint4 v[kCombKU];
#pragma unroll
      for (int u = 0; u < kCombKU; u++)
        v[u] = r[u] >= 0 ? *reinterpret_cast<const uint4*>(y_perm + (size_t)r[u] * H + cl * 8) : make_uint4(0, 0, 0, 0);
      // ascending k: the fp32 sum is formed in the order of the definition
#pragma unroll
      for (int u = 0; u < kCombKU; u++) {
        if (r[u] < 0) continue;
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
  o.x = bf16x2_rne(acc[0], acc[1]);
  o.y = bf16x2_rne(acc[2], acc[3]);
  o.z = bf16x2_rne(acc[4], acc[5]);
  o.w = bf16x2_rne(acc[6], acc[7]);
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
