/*
 * tempo_moe.h -- C ABI of an MI355X (gfx950) library that runs one GPU's
 * share of an expert-parallel MoE block under a per-batch dispatch plan.
 *
 * Source of the method: TEMPO, "Makespan-Aware Expert-Parallel Load Balancing
 * Across Memory- and Compute-Bound Regimes" (arXiv 2608.13057).  The calls
 * follow the paper's problem statement (Sec. 3.1, Eq. 3): per-expert token
 * counts n_e come from the router, replica sets R(e) from the placement layer,
 * and a dispatch assigns each expert's tokens to its replicas in shares
 * x_{e,g}; a replica with x > 0 is "activated".  On one GPU that is:
 *
 *   stage 1  tempo_moe_dispatch  count + plan application + permute into
 *                                M-tile-padded groups (Sec. 4.4, Sec. 2.2/Eq. 2)
 *   stage 2  tempo_moe_experts   per local slot: gate/up GEMM, SwiGLU, down
 *                                GEMM (Sec. 2.1, Sec. 2.2)
 *   stage 3  tempo_moe_combine   routing-weighted sum over the top-k pairs
 *                                (Sec. 2.1)
 *   all      tempo_moe_forward   stages 1-3 in order on one stream
 *
 * Conventions for every call
 *   - Pointers marked "device" are HIP device pointers owned by the caller;
 *     the library never allocates, frees or keeps them.  Pointers marked
 *     "host" are read during the call only.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and the call returns without synchronising.  Inputs must stay valid
 *     and unmodified until the stream has passed the enqueued work.  No call
 *     allocates device memory or synchronises (except tempo_moe_device_error),
 *     so the enqueued work can be captured into a HIP graph.
 *   - Return value: TEMPO_OK (0) or a TEMPO_E* code.  Argument errors are
 *     detected on the host before anything is enqueued; nothing is written
 *     then.  Errors in the *data* (routing ids, plan rows) are detected on the
 *     device: the offending pair or slot is dropped and a bit is OR-ed into a
 *     sticky word in the workspace (see tempo_moe_device_error).
 *   - Matrices are row-major.  bf16 values are stored as their 16-bit
 *     patterns; fp8 values are OCP E4M3 ("e4m3fn") bytes with fp32 block
 *     scales: activations use 1 x 128 blocks along the hidden/intermediate
 *     dimension, weights use 128 x 128 blocks.
 */
#ifndef TEMPO_MOE_H
#define TEMPO_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
#define TEMPO_OK 0
#define TEMPO_EINVAL 1       /* a null pointer, a bad dimension or m_tile, a mis-sized buffer */
#define TEMPO_EWORKSPACE 2   /* workspace_bytes smaller than tempo_moe_query's answer */
#define TEMPO_EDEVICE 3      /* the HIP runtime refused a launch or a copy */
#define TEMPO_EUNSUPPORTED 4 /* valid but outside what the kernels cover (see tempo_moe_query) */

/* bits of the sticky device error word */
#define TEMPO_DERR_BAD_ID 1u           /* a routing id not -1 and outside [0, E): pair dropped */
#define TEMPO_DERR_BAD_SLOT_EXPERT 2u  /* slot_expert[s] outside [0, E): slot receives nothing */
#define TEMPO_DERR_WEIGHT_OVERFLOW 4u  /* an expert's plan weights sum to >= 2^32: split uniformly */

/* element types */
/* tempo_plan.flags */
#define TEMPO_PLAN_SNAP_TILES 1u /* tile-aware split: boundaries on multiples of m_tile (see tempo_plan) */
#define TEMPO_PLAN_SAMPLE 2u     /* one sampled replica per pair instead of the split (see tempo_plan) */

#define TEMPO_BF16 0
#define TEMPO_FP8_E4M3 1
/* fp8 e4m3 whose scales (x_scale, w13_scale, w2_scale) are powers of two
 * (UE8M0): stage 2 applies them in the MFMA's hardware block scaling instead
 * of scaling every step's partial sums, and re-quantises h with the smallest
 * power of two >= amax / 448.  Scales that are not powers of two give wrong
 * results (their mantissas are dropped). */
#define TEMPO_FP8_E4M3_UE8M0 2

/*
 * Problem shape.
 *   T        token rows in the batch buffer (>= 1)
 *   T_valid  rows [0, T_valid) are real; rows beyond are graph padding, their
 *            pairs are neither counted nor placed and their y rows are zero
 *            (Sec. 4.4: counts are masked against graph-padding rows)
 *   K        experts per token (top-k), 1 <= K <= 32
 *   E        logical experts, 1 <= E <= 1024
 *   S        local expert slots (replicas held by this GPU), 1 <= S <= 256
 *   H, I     hidden and expert-intermediate sizes, multiples of 128
 *   m_tile   M-tile: every activated slot's rows are padded to a multiple of
 *            it (Sec. 2.2, Eq. 2); 64, 128, 192 or 256
 *   dtype    TEMPO_BF16, TEMPO_FP8_E4M3 or TEMPO_FP8_E4M3_UE8M0 (activations and weights)
 */
typedef struct tempo_moe_shape {
  int32_t T, T_valid, K, E, S, H, I, m_tile, dtype;
} tempo_moe_shape;

/*
 * Per-batch plan (all device pointers).  Sec. 3.1: x_{e,g} >= 0 with
 * sum_g x_{e,g} = n_e over the replicas R(e).  On this GPU the replicas of
 * expert e are its local slots (slot_expert[s] == e, in ascending s) plus,
 * when remote_weight[e] > 0 or remote_replicas[e] > 0, one entry standing for
 * all replicas on other GPUs, ordered last.  With weights w_j and W = sum w_j,
 * entry j receives the expert's pairs of rank [floor(n_e C_{j-1} / W),
 * floor(n_e C_j / W)) where C_j = w_0 + ... + w_j and ranks order the expert's
 * valid pairs by p = t*K + k.  Rows are renormalised at use, so any scaling
 * of a row is the same plan; a row with W = 0 is split uniformly over the
 * replicas holding the expert (weight 1 per local slot, remote_replicas[e]
 * for the remote entry), as the paper's kernel does for a torn table row
 * (Sec. 4.4).
 *   slot_expert     [S] int32   logical expert held by slot s
 *   slot_weight     [S] uint32  share weight of slot s
 *   remote_weight   [E] uint32  share weight kept by replicas on other GPUs
 *   remote_replicas [E] int32   number of replicas on other GPUs (>= 0)
 *   flags           host value: 0, or TEMPO_PLAN_SNAP_TILES for the
 *                   tile-aware split (Sec. 2.2 after Eq. 2: partial splits
 *                   snapped to tile boundaries): every boundary
 *                   floor(n_e C_j / W) other than n_e moves to the nearest
 *                   multiple of m_tile (halves up), capped at n_e, so all of
 *                   an expert's local rows but the last entry's fill whole
 *                   M-tiles.  TEMPO_PLAN_SAMPLE: the deployed semantics
 *                   (Sec. 4.4): every valid pair p = t*K + k of expert e
 *                   draws r = word 0 of Philox-4x64-10 (Salmon et al.,
 *                   SC 2011) at counter (p, 0, 0, 0) with key (seed, 0),
 *                   u = floor(hi32(r) * W / 2^32), and goes to the first
 *                   entry j with u < C_j (same entries, weights and zero-sum
 *                   fallback as the split); the rows of a slot hold its
 *                   pairs in ascending p.  Supported for T*K <= 8192 and
 *                   E <= 256 (else TEMPO_EUNSUPPORTED).  Both bits, or any
 *                   other bit: TEMPO_EINVAL.
 *   seed            host value: the generator key for TEMPO_PLAN_SAMPLE
 */
typedef struct tempo_plan {
  const int32_t* slot_expert;
  const uint32_t* slot_weight;
  const uint32_t* remote_weight;
  const int32_t* remote_replicas;
  uint32_t flags;
  uint64_t seed;
} tempo_plan;

/*
 * Stage-1 outputs (all device pointers, caller-allocated).  row_cap comes
 * from tempo_moe_query.  Slot s owns rows [slot_offsets[s], slot_offsets[s+1])
 * = P_s = m_tile * ceil(c_s / m_tile) rows, of which the first c_s are real
 * and the rest are padding.
 *   expert_counts [E] int32   n_e over valid pairs, for all E experts
 *   slot_counts   [S] int32   c_s
 *   slot_offsets  [S+1] int32 exclusive prefix sum of P_s
 *   row_token     [row_cap] int32  token of each row; -1 on padding rows.
 *                 Entries at or beyond slot_offsets[S] are not written.
 *   pair_row      [T*K] int32 row of pair p = t*K + k, -1 if the pair is not
 *                 placed on this GPU (remote share, dropped id, padding row)
 *   cum_counts    [E] uint32  nullable; if given, cum_counts[e] += n_e
 *                 (mod 2^32): the paper's persistent cumulative counter whose
 *                 window counts are recovered by wrap-safe differencing
 *   x_perm        [row_cap, H] bf16 or fp8: x_perm[row] = x[row_token[row]]
 *                 on real rows; padding rows are not written
 *   x_perm_scale  [H/128, row_cap] fp32, fp8 only (NULL for bf16): the scale
 *                 of row r and 128-column block b at b * row_cap + r
 *                 (block-major, so stage 2 reads the scales of one
 *                 contraction block contiguously); padding rows not written
 */
typedef struct tempo_dispatch_out {
  int32_t* expert_counts;
  int32_t* slot_counts;
  int32_t* slot_offsets;
  int32_t* row_token;
  int32_t* pair_row;
  uint32_t* cum_counts;
  void* x_perm;
  float* x_perm_scale;
} tempo_dispatch_out;

/*
 * One slot's packed weight tensors (device pointers), as
 * tempo_moe_pack_weights writes them for a shape with S = 1; an entry of the
 * per-slot table of tempo_expert_weights.
 */
typedef struct tempo_slot_weights {
  const void* w13;
  const float* w13_scale;
  const void* w2;
  const float* w2_scale;
} tempo_slot_weights;

/*
 * Expert weights of the S local slots (device pointers).  A replica slot
 * holds its own copy of its expert's weights.  In the natural layout:
 *   w13       [S, 2I, H]  rows 0..I-1 gate projection, rows I..2I-1 up projection
 *   w13_scale [S, 2I/128, H/128] fp32, fp8 only
 *   w2        [S, H, I]   down projection
 *   w2_scale  [S, H/128, I/128] fp32, fp8 only
 * tempo_moe_experts / tempo_moe_forward take the packed layout written by
 * tempo_moe_pack_weights: w13 and w2 of the same sizes, and (fp8) packed
 * scales of 4 fp32 words per (output block, 128-element contraction step):
 *   w13_scale packed [S, I/64, H/128, 4]: {gate-row block scale, up-row block
 *             scale, 0, 0} of the output block pairing gate rows 64n..64n+63
 *             with up rows I+64n..I+64n+63
 *   w2_scale  packed [S, H/128, I/128, 4]: {block scale, 0, 0, 0}
 * All device buffers must be 16-byte aligned.
 */
typedef struct tempo_expert_weights {
  const void* w13;
  const float* w13_scale;
  const void* w2;
  const float* w2_scale;
  /* Stage 2 only, nullable: a device array [S] whose entry s holds slot s's
   * packed tensors wherever they live (the replica sets of Sec. 3.1 come from
   * a placement that puts each slot's weights where it likes).  When given,
   * the four pointers above are ignored (and may be NULL); each entry's
   * tensors are those of a 1-slot pack.  Stage 2 reads each entry once per
   * work item.  tempo_moe_pack_weights ignores this field. */
  const tempo_slot_weights* slot_table;
} tempo_expert_weights;

/*
 * Sizes for a shape.  *workspace_bytes: the workspace every other call needs
 * (one per stream in flight); *row_cap = T*K + S*(m_tile-1) rounded up to a
 * multiple of 128, the rows of the permuted buffers.  The workspace must be
 * zero-filled once before its first use (it holds the sticky error word);
 * after that it is reused without clearing.  *packed_bytes_per_slot: the
 * bytes of one slot's packed weights, w13 + w2 (2I*H + H*I elements) plus,
 * for fp8, the packed scales (I/64 * H/128 + H/128 * I/128 entries of 16
 * bytes) -- what a slot table entry points at.  Returns TEMPO_EINVAL /
 * TEMPO_EUNSUPPORTED for shapes the library rejects.  Any output pointer may
 * be NULL.
 */
int tempo_moe_query(const tempo_moe_shape* shape, size_t* workspace_bytes, int32_t* row_cap,
                    size_t* packed_bytes_per_slot);

/*
 * One-time re-layout of expert weights for the stage-2 kernels (not part of
 * the per-batch path; run it when weights are loaded).  natural holds w13 /
 * w2 in the natural layout above; packed->w13 / packed->w2 are caller
 * buffers of the same byte sizes that receive the packed layout, in which
 * every (output block of 128 weight rows, contraction step of 128 bytes)
 * tile of a slot is one contiguous 16 KB block and the tiles of an output
 * block follow each other along the contraction, so stage 2 streams each
 * activated slot's weights front to back.  Inside a tile, rows 32w..32w+31
 * form the 4 KB piece w, stored as four 1 KB loads in MFMA operand order:
 * load j, lane l (0..63) holds the 16-byte chunk c of row 32w + l%32, with
 * c = 2j + l/32 (bf16) or c = 4(j/2) + 2(l/32) + j%2 (fp8).  For w13 output block n holds gate
 * rows 64n..64n+63 and the same up rows, interleaved in groups of 16 rows
 * (gate 64n..64n+15, up I+64n..I+64n+15, gate 64n+16.., ...).  fp8: packed->w13_scale / w2_scale are
 * caller buffers of the packed scale sizes above that receive the packed
 * scales (bf16: scale pointers are ignored).  Returns TEMPO_EINVAL for null
 * or aliasing buffers.
 */
int tempo_moe_pack_weights(const tempo_moe_shape* shape, const tempo_expert_weights* natural,
                           const tempo_expert_weights* packed, void* stream);

/*
 * Stage 1 (Sec. 4.4 fused count collection + dispatch, Sec. 2.2 / Eq. 2
 * M-tile padding).  topk_ids [T, K] int32 device, -1 = no expert.
 * x [T, H] device (bf16 or fp8), x_scale [T, H/128] fp32 device (fp8 only,
 * else NULL).  Deterministic: positions come from a stable counting sort,
 * never from atomics.
 */
int tempo_moe_dispatch(const tempo_moe_shape* shape, const tempo_plan* plan, const int32_t* topk_ids,
                       const void* x, const float* x_scale, const tempo_dispatch_out* out, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Stage 2 (Sec. 2.1 "gate/up, activation, down"; Sec. 2.2 weight streaming).
 * For every slot with c_s > 0: h = silu(x_perm W_gate^T) * (x_perm W_up^T)
 * with silu(z) = z / (1 + e^-z), then y_perm = h W2^T.  Slots with c_s = 0
 * read no weights.  Reads slot_counts, slot_offsets, row_token and x_perm
 * (and x_perm_scale) of a stage-1 result from device memory, so no host
 * round trip is needed; expert_counts and pair_row may be NULL.  The number
 * of M-tiles comes from slot_offsets[S] / m_tile (capped at row_cap /
 * m_tile), so the workspace need not be the one stage 1 used: any
 * workspace of tempo_moe_query's size serves.
 * y_perm [row_cap, H] bf16 device: real rows written,
 * padding rows not.  Accumulation is fp32; h is rounded to bf16 (bf16 path)
 * or quantised to e4m3 with 1 x 128 fp32 scales amax/448, round to nearest
 * even, saturating at 448 (fp8 path; the fp8 contraction applies the
 * activation and weight block scales once per 128-element block); y_perm is
 * rounded to bf16.  The arithmetic of a row does not depend on which slot
 * or tile it lands in.
 */
int tempo_moe_experts(const tempo_moe_shape* shape, const tempo_dispatch_out* disp,
                      const tempo_expert_weights* weights, void* y_perm, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * Stage 3 (Sec. 2.1 combine).  y[t] = sum over k ascending of
 * topk_w[t,k] * y_perm[pair_row[t,k]] over pairs with pair_row >= 0, in fp32,
 * rounded to bf16; rows with no local pair and rows t >= T_valid are zero.
 * topk_w [T, K] fp32 device; y [T, H] bf16 device.  On an EP group, y is
 * this GPU's partial sum that the combine all-to-all would add up.
 */
int tempo_moe_combine(const tempo_moe_shape* shape, const int32_t* pair_row, const float* topk_w,
                      const void* y_perm, void* y, void* stream);

/*
 * Stages 1-3 on one stream.  disp receives the stage-1 outputs (caller
 * buffers as for tempo_moe_dispatch), except that x_perm is left unwritten
 * where stage 2 gathers the token rows itself (decode-sized batches, and
 * the 256-row large-tile kernels of bf16 and UE8M0 fp8, whose GEMMs read
 * the rows packed in MFMA operand order in the workspace), and so is
 * x_perm_scale for the large-tile fp8 kernel, which packs the token rows'
 * own scales; y_perm lives in the workspace.
 * slot_time_ns [S] uint64 device, nullable: per slot, the span from the
 * first stage-2 tile that started on it to the last that ended, measured
 * with the GPU's 100 MHz real-time counter (0 for slots with c_s = 0).
 * Spans of concurrently running slots overlap; it is exact for one slot.
 * stage_events: nullable host array of TEMPO_STAGE_EVENTS (8) hipEvent_t
 * (created by the caller; each entry nullable) recorded on `stream` before
 * stage 1, after stage 1, right before the gate/up GEMM kernel (after the
 * activation pack of the 256-row large-tile kernels), after it, after the
 * whole gate/up step (split-item fixup and, for fp8, the re-quantisation of
 * h), after the down GEMM kernel, after the whole down step and after
 * stage 3, for per-stage and per-kernel timing.
 */
#define TEMPO_STAGE_EVENTS 8
int tempo_moe_forward(const tempo_moe_shape* shape, const tempo_plan* plan, const int32_t* topk_ids,
                      const float* topk_w, const void* x, const float* x_scale, const tempo_expert_weights* weights,
                      const tempo_dispatch_out* disp, void* y, uint64_t* slot_time_ns, void* const* stage_events,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * tempo_moe_forward with the library's own static scratch array as the
 * workspace, so the call takes no workspace argument and allocates nothing.
 * Arguments, outputs and errors are those of tempo_moe_forward, except:
 *   - the shape's workspace (tempo_moe_query) must fit in
 *     TEMPO_STATIC_SCRATCH_BYTES, else TEMPO_EWORKSPACE is returned before
 *     anything is enqueued (decode-sized shapes fit: e.g. 18 slots of
 *     H 4096 / I 1536 with 512 tokens, top-8, m_tile 64);
 *   - every GPU holds one copy of the array from the first call on it until
 *     the process ends, and every call on that GPU uses it: calls that
 *     overlap on one GPU (concurrent streams, or a second call enqueued
 *     before the first has run on another stream) race on it, so serialise
 *     them on one stream;
 *   - the array keeps the last call's contents; nothing in it needs to start
 *     at zero, and the sticky device error word it holds cannot be read
 *     (data errors are still handled: offending pairs are dropped).
 * TEMPO_EDEVICE if the array's device address cannot be looked up.
 */
#define TEMPO_STATIC_SCRATCH_BYTES (128u << 20)
int tempo_moe_forward_static(const tempo_moe_shape* shape, const tempo_plan* plan, const int32_t* topk_ids,
                             const float* topk_w, const void* x, const float* x_scale,
                             const tempo_expert_weights* weights, const tempo_dispatch_out* disp, void* y,
                             uint64_t* slot_time_ns, void* const* stage_events, void* stream);

/*
 * Synchronises `stream`, returns the sticky device error word (OR of the
 * TEMPO_DERR_* bits seen by every dispatch since the last read) in *bits and
 * clears it.  Returns TEMPO_EDEVICE if the synchronisation fails.
 */
int tempo_moe_device_error(void* workspace, void* stream, uint32_t* bits);

/*
 * Per-expert pair counts of a window from two snapshots of the cumulative
 * counters (tempo_dispatch_out.cum_counts; Sec. 4.4: a persistent cumulative
 * counter needs no zeroing kernel, the reader recovers window counts by
 * differencing): window[e] = (after[e] - before[e]) mod 2^32, exact while a
 * window adds fewer than 2^32 pairs to an expert.  Host arrays of E entries;
 * touches no GPU.  TEMPO_EINVAL for a null pointer or E < 1.
 */
int tempo_moe_counter_window(int32_t E, const uint32_t* before, const uint32_t* after, uint32_t* window);

/* A static string describing a TEMPO_* return code. */
const char* tempo_moe_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* TEMPO_MOE_H */
