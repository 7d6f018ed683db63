// Pipeline helpers shared by the stage-2 grouped GEMMs (bf16 and fp8).
#pragma once

#include "internal.h"

namespace tempo {
namespace gemm {

constexpr int ROWB = 128;               // bytes of a row per contraction step
constexpr int BNW = 128;                // weight rows per work item
constexpr int B_BYTES = BNW * ROWB;     // 16 KB of weights per step of a work item

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two fp32 values as bf16, rounded to nearest even, in one word (lo in the
// low half): gfx950's packed conversion, one instruction for the pair; the
// same bits as f32_to_bf16_rne for every finite value.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] bits 3:0, vmcnt[5:4] bits 15:14, expcnt 6:4 and lgkmcnt 11:8 at
// their maximum so they do not wait); n is a compile-time constant <= 63.
#define TEMPO_VMCNT_IMM(n) (((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))

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
// s_waitcnt vmcnt before using the data.  Nothing else in these kernels uses M0.
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

// The same DMA for the lanes set in `lanes` only.  EXEC is switched inside
// the asm statement and restored there, so the load needs no branch around
// it (a branch would split the caller's basic block, and the scheduling
// fences that order its MFMAs hold only within one block).
__device__ __forceinline__ void lds_dma16s_lanes(uint64_t sbase, uint32_t voff, uint32_t lds_addr, uint64_t lanes) {
  uint64_t saved;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, %4\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %3\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(lds_addr), "s"(sbase), "s"(lanes)
      : "memory", "m0");
}

// LDS byte address of a shared-memory pointer (the low 32 bits of its
// generic address).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// Byte offset of 16-byte chunk c of row r in a swizzled tile (chunk c of a
// row is stored at position c ^ (r & 7), so 8 consecutive rows read at the
// same chunk hit 8 distinct bank groups).
__device__ __forceinline__ int swz(int r, int c) { return r * ROWB + ((c ^ (r & 7)) << 4); }

// Packed weight tensor field of a per-slot table entry (tempo_slot_weights).
enum SlotField : int { kFieldW13 = 0, kFieldW13Scale = 1, kFieldW2 = 2, kFieldW2Scale = 3 };

// Base of slot s's packed tensor: entry s of the per-slot table when the
// caller gave one (tempo_slot_weights, four pointers per entry), else s
// slots into the contiguous [S] tensor.  s is uniform.  The entry is read
// with a scalar load in inline assembly: the compiler would otherwise use a
// vector load (it cannot tell the table from the memory the kernel writes)
// and wait for every vector load in flight before using it, the operand
// DMA ring included.
__device__ __forceinline__ const char* slot_tensor(const char* base, size_t per_slot, const uint64_t* table, int field,
                                                   int s) {
  if (!table) return base + (size_t)s * per_slot;
  const uint64_t* e = table + (size_t)s * 4 + field;
  uint64_t v;
  asm volatile("s_load_dwordx2 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(e) : "memory");
  return reinterpret_cast<const char*>(v);
}

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
