// One-time weight re-layout for the stage-2 kernels.
//
// A stage-2 work item multiplies a tile of activation rows by one output block
// of 128 weight rows, 128 bytes of the contraction at a time (a step).  Each
// of the four wavefronts of a workgroup multiplies 32 of the block's rows and
// loads them itself, straight into registers, as MFMA operands.  The packed
// layout therefore stores, per slot, output block by output block, the steps
// of the block one after another; a step is four 4 KB pieces (one per
// wavefront, rows 32w..32w+31), and a piece is four 1 KB loads in the order
// the MFMA operand registers want them: load j, lane l holds the 16-byte
// chunk c(j, l) of row 32w + (l & 31), with
//   bf16 (32x32x16 MFMA):    c = 2j + (l >> 5)
//   fp8  (32x32x64 MFMA):    c = 4(j >> 1) + 2(l >> 5) + (j & 1)
// so every load instruction of the stream reads 1 KB of consecutive bytes.
// For the gate/up matrix an output block pairs gate rows n..n+63 with up rows
// I+n..I+n+63, interleaved in groups of 16 (gate n..n+15, up I+n..I+n+15,
// gate n+16.., ...), so a 32-row slice multiplied by one wavefront holds
// matching gate and up columns for SwiGLU.
//
// fp8 weight scales are packed per (output block, contraction step) as four
// words, so that a step's scales travel with the step in one 16-byte load:
// gate/up {scale of the gate rows' 128-block, scale of the up rows' block,
// 0, 0}; down {scale of the block, 0, 0, 0}.
#include "internal.h"

namespace tempo {
namespace {

// one thread per 16-byte chunk of the packed slot
__global__ __launch_bounds__(256) void k_pack(const uint4* __restrict__ src, uint4* __restrict__ dst, int S,
                                              int rows, int row_chunks, int gateup, int half_rows, int fp8) {
  const size_t per_slot = (size_t)rows * row_chunks;
  const size_t total = per_slot * S;
  const int KT = row_chunks / 8;
  for (size_t o = (size_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (size_t)gridDim.x * 256) {
    const size_t s = o / per_slot;
    size_t q = o % per_slot;
    const int l = (int)(q & 63);
    q >>= 6;
    const int j = (int)(q & 3);
    q >>= 2;
    const int w = (int)(q & 3);
    q >>= 2;
    const int kt = (int)(q % KT);
    const int nb = (int)(q / KT);
    const int r = 32 * w + (l & 31);  // row of the output block
    const int c = fp8 ? 4 * (j >> 1) + 2 * (l >> 5) + (j & 1) : 2 * j + (l >> 5);
    int row;
    // gate/up: 16-row groups alternate gate and up: group 2w holds gate rows
    // 64nb+16w.., group 2w+1 the matching up rows
    if (gateup) row = ((r >> 4) & 1 ? half_rows : 0) + nb * 64 + (r >> 5) * 16 + (r & 15);
    else row = nb * 128 + r;
    dst[o] = src[s * per_slot + (size_t)row * row_chunks + kt * 8 + c];
  }
}

// one thread per packed 4-word entry [slot][block][step]
__global__ __launch_bounds__(256) void k_pack_scales(const float* __restrict__ nat, float4* __restrict__ dst, int S,
                                                     int nblk, int KT, int nat_rows, int gateup, int half_blocks) {
  const size_t total = (size_t)S * nblk * KT;
  for (size_t o = (size_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (size_t)gridDim.x * 256) {
    const int kt = (int)(o % KT);
    const size_t q = o / KT;
    const int nb = (int)(q % nblk);
    const size_t s = q / nblk;
    const float* ns = nat + s * nat_rows * KT;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (gateup) {
      v.x = ns[(size_t)(nb / 2) * KT + kt];
      v.y = ns[(size_t)(half_blocks + nb / 2) * KT + kt];
    } else {
      v.x = ns[(size_t)nb * KT + kt];
    }
    dst[o] = v;
  }
}

}  // namespace

hipError_t launch_pack(const tempo_moe_shape& s, const tempo_expert_weights& nat, const tempo_expert_weights& pk,
                       hipStream_t st) {
  const int es = s.dtype == TEMPO_BF16 ? 2 : 1;
  // gate/up: rows 2I, row bytes H*es; down: rows H, row bytes I*es
  const int rc13 = s.H * es / 16, rc2 = s.I * es / 16;
  const size_t n13 = (size_t)s.S * 2 * s.I * rc13, n2 = (size_t)s.S * s.H * rc2;
  const int g13 = (int)((n13 + 255) / 256 < 65536 ? (n13 + 255) / 256 : 65536);
  const int g2 = (int)((n2 + 255) / 256 < 65536 ? (n2 + 255) / 256 : 65536);
  hipLaunchKernelGGL(k_pack, dim3(g13), dim3(256), 0, st, static_cast<const uint4*>(nat.w13),
                     static_cast<uint4*>(const_cast<void*>(pk.w13)), s.S, 2 * s.I, rc13, 1, s.I, es == 1);
  hipLaunchKernelGGL(k_pack, dim3(g2), dim3(256), 0, st, static_cast<const uint4*>(nat.w2),
                     static_cast<uint4*>(const_cast<void*>(pk.w2)), s.S, s.H, rc2, 0, 0, es == 1);
  if (s.dtype != TEMPO_BF16) {
    // gate/up: I/64 output blocks x H/128 steps; down: H/128 blocks x I/128 steps
    const size_t m13 = (size_t)s.S * (s.I / 64) * (s.H / 128), m2 = (size_t)s.S * (s.H / 128) * (s.I / 128);
    hipLaunchKernelGGL(k_pack_scales, dim3((int)((m13 + 255) / 256 < 65536 ? (m13 + 255) / 256 : 65536)), dim3(256), 0,
                       st, nat.w13_scale, reinterpret_cast<float4*>(const_cast<float*>(pk.w13_scale)), s.S, s.I / 64,
                       s.H / 128, 2 * s.I / 128, 1, s.I / 128);
    hipLaunchKernelGGL(k_pack_scales, dim3((int)((m2 + 255) / 256 < 65536 ? (m2 + 255) / 256 : 65536)), dim3(256), 0,
                       st, nat.w2_scale, reinterpret_cast<float4*>(const_cast<float*>(pk.w2_scale)), s.S, s.H / 128,
                       s.I / 128, s.H / 128, 0, 0);
  }
  return hipGetLastError();
}

}  // namespace tempo
