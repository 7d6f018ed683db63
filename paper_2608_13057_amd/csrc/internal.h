// Internal declarations shared by the HIP translation units of libtempo_moe.
// Not part of the public ABI (include/tempo_moe.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/tempo_moe.h"

namespace tempo {

// Pairs handled by one block of the counting kernel (one pair per thread; the
// granularity of the per-block histograms).
constexpr int kCountThreads = 256;

constexpr int kMaxE = 1024;
constexpr int kMaxS = 256;
constexpr int kMaxK = 32;

// Workspace header words (uint32 slots at the start of the workspace).
enum HeaderWord : int {
  kHdrSticky = 0,  // OR of the device error bits since the last read
  kHdrLastErr = 1, // error bits of the last dispatch
  kHdrTiles = 2,   // sum over slots of P_s / m_tile
  kHdrActive = 3,  // G: slots with c_s > 0
  kHdrPairs = 4,   // N: pairs placed locally
};

// Byte offsets of the workspace regions for one shape.
struct Layout {
  size_t header;      // 256 B of uint32 words
  size_t blk_hist;    // [nblk][E] int32 per-block counts
  size_t blk_pre;     // [nblk + 1][E] int32 exclusive prefixes over the count blocks, then the totals (large batches)
  size_t blk_err;     // [nblk] uint32
  size_t local_rank;  // [T*K] int32 stable rank of a pair within its block and expert
  size_t slot_t0;     // [S] uint64 first stage-2 tile start (real-time counter)
  size_t slot_t1;     // [S] uint64 last stage-2 tile end
  size_t h;           // [row_cap, I] bf16 or e4m3 (256-row bf16 tiles: packed in MFMA operand order)
  size_t h_scale;     // [I/128, row_cap] fp32 (fp8 only; scale-block-major)
  size_t h32;         // [row_cap, I] fp32 gate/up output before re-quantisation (fp8 only)
  size_t y_perm;      // [row_cap, H] bf16
  size_t apack;       // 256-row large-tile kernels only: the activation rows packed in MFMA operand order
  size_t part;        // [grid][8][m_tile][128] fp32 stage-2 partial tiles
  size_t fix;         // [grid][12] int32 stage-2 fixup records
  size_t total;
  int nblk;
  int row_cap;
};

Layout make_layout(const tempo_moe_shape& s);

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---- launchers (stream-ordered, no synchronisation) ----
// copy_rows = false leaves x_perm unwritten, copy_scales = false (or bf16)
// x_perm_scale (stage 2 then reads them through row_token).
// Whether sampled replicas (TEMPO_PLAN_SAMPLE) are available for this shape.
bool dispatch_sample_supported(const tempo_moe_shape& s);

hipError_t launch_dispatch(const tempo_moe_shape& s, const tempo_plan& plan, const int32_t* topk_ids,
                           const void* x, const float* x_scale, const tempo_dispatch_out& out, char* ws,
                           const Layout& L, bool timing, bool copy_rows, bool copy_scales, hipStream_t st);

// ev: null, or 4 events (each nullable) recorded right before the gate/up
// GEMM kernel (after the activation pack of the large-tile kernels), after
// it, after the gate/up step and after the down GEMM kernel.
// x_rows: null -> the gate/up GEMM reads d.x_perm; otherwise it reads the
// activation rows x_rows[row_token[row]] (x_rows = the unpermuted x).  fp8:
// the stream-K GEMM reads the scales from d.x_perm_scale; the large-tile
// kernel from x_rows_scale[row_token[row]] ([tokens][H/128] fp32) when
// x_rows is given, else from d.x_perm_scale.  Whether stage 2 reads the
// token rows, and their fp8 scales, itself: experts_gather_rows /
// experts_reads_token_scales.
hipError_t launch_experts_bf16(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                               const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing,
                               const hipEvent_t* ev, hipStream_t st);

hipError_t launch_experts_fp8(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              const void* x_rows, const float* x_rows_scale, void* y_perm, char* ws, const Layout& L,
                              bool timing, const hipEvent_t* ev, hipStream_t st);

// bf16 with 256-row M-tiles (and H a multiple of 256): both GEMMs as 256 x 256
// items on MFMA-blocked wavefronts (the large-tile kernel), with the
// activation rows first packed into the workspace (experts_big_pack_bytes of
// it) from x_rows (token rows, through row_token) or, if null, from x_perm.
bool experts_big_supported(const tempo_moe_shape& s);
size_t experts_big_pack_bytes(const tempo_moe_shape& s, int row_cap);
hipError_t launch_experts_big(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                              const void* x_rows, void* y_perm, char* ws, const Layout& L, bool timing,
                              const hipEvent_t* ev, hipStream_t st);

// UE8M0 fp8 with 256-row M-tiles (H a multiple of 256): both GEMMs as
// 256 x 256 items on the hardware-scaled fp8 MFMA, with the activation rows
// and their scale exponents first packed into the workspace
// (experts_big_f8_pack_bytes of it) and h re-quantised in the gate/up
// epilogue.
bool experts_big_f8_supported(const tempo_moe_shape& s);
size_t experts_big_f8_pack_bytes(const tempo_moe_shape& s, int row_cap);
hipError_t launch_experts_big_f8(const tempo_moe_shape& s, const tempo_dispatch_out& d, const tempo_expert_weights& w,
                                 const void* x_rows, const float* x_rows_scale, void* y_perm, char* ws,
                                 const Layout& L, bool timing, const hipEvent_t* ev, hipStream_t st);

hipError_t launch_combine(const tempo_moe_shape& s, const int32_t* pair_row, const float* topk_w, const void* y_perm,
                          void* y, const int32_t* slot_counts, const uint64_t* t0, const uint64_t* t1,
                          uint64_t* slot_time_ns, hipStream_t st);

hipError_t launch_pack(const tempo_moe_shape& s, const tempo_expert_weights& natural,
                       const tempo_expert_weights& packed, hipStream_t st);

// Whether stage 2 gathers the activation rows itself (through row_token)
// rather than reading rows that stage 1 permuted into x_perm: true for the
// large-tile kernel, whose pack step gathers them, and for the streaming
// GEMM when every workgroup's range spans few enough M-tiles (the row tables
// of its M-tiles sit in LDS).
bool experts_gather_rows(const tempo_moe_shape& s, const Layout& L);
bool experts_reads_token_scales(const tempo_moe_shape& s);

// Whether stage-2 kernels exist for this shape's element type and M-tile.
bool experts_supported(const tempo_moe_shape& s);

// Workgroups of a persistent kernel with per_cu resident workgroups per CU
// (a multiple of 8, the XCD count).
int persistent_grid(int per_cu);

}  // namespace tempo
