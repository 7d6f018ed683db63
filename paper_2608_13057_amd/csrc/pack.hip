// One-time weight re-layout for the stage-2 kernels.
//
// A stage-2 work item multiplies a tile of activation rows by one output block
// of 128 weight rows, 128 bytes of the contraction at a time.  The packed
// layout stores, per slot, output block by output block, the contraction steps
// of that block one after another, each step as a 16 KB tile of 128 rows x 8
// chunks of 16 bytes, chunk c of row r at position c ^ (r & 7).  A DMA group
// of 8 rows is then one contiguous 1 KB that lands in LDS already swizzled,
// and a work item streams its 128 rows x K weights as one contiguous block.
// For the gate/up matrix an output block pairs gate rows n..n+63 with up rows
// I+n..I+n+63 so SwiGLU sees matching columns.
#include "internal.h"

namespace tempo {
namespace {

// one thread per 16-byte chunk of the packed slot
__global__ __launch_bounds__(256) void k_pack(const uint4* __restrict__ src, uint4* __restrict__ dst, int S,
                                              int rows, int row_chunks, int gateup, int half_rows) {
  const size_t per_slot = (size_t)rows * row_chunks;
  const size_t total = per_slot * S;
  const int KT = row_chunks / 8;
  for (size_t o = (size_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (size_t)gridDim.x * 256) {
    const size_t s = o / per_slot;
    size_t q = o % per_slot;
    const int p = (int)(q & 7);
    q >>= 3;
    const int r = (int)(q & 127);
    q >>= 7;
    const int kt = (int)(q % KT);
    const int nb = (int)(q / KT);
    int row;
    if (gateup) row = r < 64 ? nb * 64 + r : half_rows + nb * 64 + (r - 64);
    else row = nb * 128 + r;
    const int c = p ^ (r & 7);
    dst[o] = src[s * per_slot + (size_t)row * row_chunks + kt * 8 + c];
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
                     static_cast<uint4*>(const_cast<void*>(pk.w13)), s.S, 2 * s.I, rc13, 1, s.I);
  hipLaunchKernelGGL(k_pack, dim3(g2), dim3(256), 0, st, static_cast<const uint4*>(nat.w2),
                     static_cast<uint4*>(const_cast<void*>(pk.w2)), s.S, s.H, rc2, 0, 0);
  return hipGetLastError();
}

}  // namespace tempo
