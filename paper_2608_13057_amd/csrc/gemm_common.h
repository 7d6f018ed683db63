// Pipeline helpers shared by the stage-2 grouped GEMMs (bf16 and fp8).
#pragma once

#include "internal.h"

namespace tempo {
namespace gemm {

constexpr int ROWB = 128;               // bytes per LDS tile row (one contraction step)
constexpr int BNW = 128;                // weight rows per tile
constexpr int B_BYTES = BNW * ROWB;     // 16 KB weight tile per step
constexpr int RING_BYTES = 144 * 1024;  // LDS ring shared by the pipeline stages
constexpr int NS_MAX = 8;

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] bits 3:0, vmcnt[5:4] bits 15:14, expcnt 6:4 and lgkmcnt 11:8 at
// their maximum so they do not wait).  n must be exact or an underestimate
// of the loads that may stay outstanding.
#define TEMPO_VMCNT_IMM(n) (((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))
__device__ __forceinline__ void wait_vmcnt(int n) {
  switch (n) {
#define TEMPO_W(i) \
  case i:          \
    __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(i)); \
    break;
    TEMPO_W(0) TEMPO_W(1) TEMPO_W(2) TEMPO_W(3) TEMPO_W(4) TEMPO_W(5) TEMPO_W(6) TEMPO_W(7)
    TEMPO_W(8) TEMPO_W(9) TEMPO_W(10) TEMPO_W(11) TEMPO_W(12) TEMPO_W(13) TEMPO_W(14) TEMPO_W(15)
    TEMPO_W(16) TEMPO_W(17) TEMPO_W(18) TEMPO_W(19) TEMPO_W(20) TEMPO_W(21) TEMPO_W(22) TEMPO_W(23)
    TEMPO_W(24) TEMPO_W(25) TEMPO_W(26) TEMPO_W(27) TEMPO_W(28) TEMPO_W(29) TEMPO_W(30) TEMPO_W(31)
    TEMPO_W(32) TEMPO_W(33) TEMPO_W(34) TEMPO_W(35) TEMPO_W(36) TEMPO_W(37) TEMPO_W(38) TEMPO_W(39)
    TEMPO_W(40) TEMPO_W(41) TEMPO_W(42) TEMPO_W(43) TEMPO_W(44) TEMPO_W(45) TEMPO_W(46) TEMPO_W(47)
    TEMPO_W(48) TEMPO_W(49) TEMPO_W(50) TEMPO_W(51) TEMPO_W(52) TEMPO_W(53) TEMPO_W(54) TEMPO_W(55)
    TEMPO_W(56) TEMPO_W(57) TEMPO_W(58) TEMPO_W(59) TEMPO_W(60) TEMPO_W(61) TEMPO_W(62) TEMPO_W(63)
#undef TEMPO_W
    default:
      __builtin_amdgcn_s_waitcnt(TEMPO_VMCNT_IMM(0));
  }
}

// Wait until this wavefront's LDS (and scalar memory) operations are done.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Workgroup barrier without a memory fence (the fence would make the
// compiler wait for every outstanding load, draining the pipeline); the
// empty asm statements keep LDS accesses on their side of the barrier.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16 bytes per active lane from global memory straight into LDS at
// lds_base + 16 * lane (global_load_lds_dwordx4; the LDS base goes in M0).
// Issued from inline assembly so that the compiler does not track it: it
// would otherwise wait for every such load before each LDS read, since it
// cannot tell which ring stage a read touches.  The caller waits with
// wait_vmcnt before using the data.  Nothing else in these kernels uses M0.
__device__ __forceinline__ void lds_dma16(const void* gptr, const void* lds_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off" ::"v"(gptr),
      "s"(lds)
      : "memory", "m0");
}

// The same DMA with a uniform 64-bit base in scalar registers and a 32-bit
// per-lane byte offset (global address = sbase + voff): the base of a stream
// advances with two scalar adds per step instead of a 64-bit add per lane.
__device__ __forceinline__ void lds_dma16s(const void* sbase, uint32_t voff, uint32_t lds_addr) {
  const uint64_t b = (uint64_t)(uintptr_t)sbase;
  const uint64_t bu = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds_addr);
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1" ::"v"(voff),
      "s"(bu), "s"(l)
      : "memory", "m0");
}

// LDS byte address of a shared-memory pointer (the low 32 bits of its
// generic address).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// Byte offset of 16-byte chunk c of row r in a swizzled tile (chunk c of a
// row is stored at position c ^ (r & 7), so 8 consecutive rows read at the
// same chunk hit 8 distinct bank groups).
__device__ __forceinline__ int swz(int r, int c) { return r * ROWB + ((c ^ (r & 7)) << 4); }

// Slot of global M-tile row0 (largest s with off[s] <= row0; off has S+1
// entries, row0 < off[S]).
__device__ __forceinline__ int slot_of_row(const int32_t* off, int S, int row0) {
  int lo = 0, hi = S;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (off[mid] <= row0) lo = mid;
    else hi = mid;
  }
  return lo;
}

}  // namespace gemm
}  // namespace tempo
