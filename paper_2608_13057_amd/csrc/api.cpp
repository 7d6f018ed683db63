// Host side of the C ABI declared in include/tempo_moe.h: argument
// validation (before anything is enqueued), workspace layout, and the
// stream-ordered launches of the stage kernels.  No call allocates device
// memory or synchronises, except tempo_moe_device_error.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstring>

#include "internal.h"

namespace tempo {

static size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

Layout make_layout(const tempo_moe_shape& s) {
  Layout L{};
  const size_t P = (size_t)s.T * s.K;
  L.nblk = (int)((P + kCountThreads - 1) / kCountThreads);
  // rounded up to 128 rows so that every block-major scale column starts on a
  // 512-byte boundary (stage 2 moves them with 16-byte DMA loads)
  L.row_cap = (int)((P + (size_t)s.S * (s.m_tile - 1) + 127) / 128 * 128);
  const size_t eh = s.dtype == TEMPO_BF16 ? 2 : 1;
  size_t o = 0;
  L.header = o;
  o = align_up(o + 256);
  L.blk_hist = o;
  o = align_up(o + (size_t)L.nblk * s.E * 4);
  L.blk_pre = o;
  o = align_up(o + (size_t)(L.nblk + 1) * s.E * 4);
  L.blk_err = o;
  o = align_up(o + (size_t)L.nblk * 4);
  L.local_rank = o;
  o = align_up(o + P * 4);

  L.slot_t0 = o;
  o = align_up(o + (size_t)s.S * 8);
  L.slot_t1 = o;
  o = align_up(o + (size_t)s.S * 8);
  L.h = o;
  o = align_up(o + (size_t)L.row_cap * s.I * eh);
  L.h_scale = o;
  o = align_up(o + (s.dtype == TEMPO_BF16 ? 0 : (size_t)L.row_cap * (s.I / 128) * 4));
  L.h32 = o;
  o = align_up(o + (s.dtype == TEMPO_BF16 ? 0 : (size_t)L.row_cap * s.I * 4));
  L.y_perm = o;
  o = align_up(o + (size_t)L.row_cap * s.H * 2);
  L.apack = o;
  o = align_up(o + std::max(experts_big_pack_bytes(s, L.row_cap), experts_big_f8_pack_bytes(s, L.row_cap)));
  // stage-2 partial tiles: per workgroup of the persistent grid, 8 tiles of
  // m_tile x 128 fp32 (the running sum and the chunks of split work items)
  L.part = o;
  o = align_up(o + (size_t)persistent_grid(1) * 8 * s.m_tile * 128 * 4);
  L.fix = o;  // per workgroup: the split work item it completes (12 int32)
  o = align_up(o + (size_t)persistent_grid(1) * 12 * 4);
  L.total = o;
  return L;
}

int persistent_grid(int per_cu) {
  static std::atomic<int> cached{0};
  int cus = cached.load();
  if (cus <= 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    cached.store(cus);
  }
  return ((cus * per_cu + 7) / 8) * 8;  // a multiple of the 8 XCDs
}

static int check_shape(const tempo_moe_shape* s) {
  if (!s) return TEMPO_EINVAL;
  if (s->T < 1 || s->T_valid < 0 || s->T_valid > s->T || s->K < 1 || s->E < 1 || s->S < 1 || s->H < 128 ||
      s->I < 128)
    return TEMPO_EINVAL;
  if (s->K > kMaxK || s->K > s->E || s->E > kMaxE || s->S > kMaxS) return TEMPO_EINVAL;
  if (s->H % 128 || s->I % 128) return TEMPO_EINVAL;
  if (s->m_tile != 64 && s->m_tile != 128 && s->m_tile != 192 && s->m_tile != 256) return TEMPO_EINVAL;
  if (s->dtype != TEMPO_BF16 && s->dtype != TEMPO_FP8_E4M3 && s->dtype != TEMPO_FP8_E4M3_UE8M0) return TEMPO_EINVAL;
  // row indices and element offsets stay within int32 / the addressable range
  const long long P = (long long)s->T * s->K;
  const long long cap = P + (long long)s->S * (s->m_tile - 1);
  if (P > (1ll << 26) || cap * (long long)s->H > (1ll << 40)) return TEMPO_EUNSUPPORTED;
  return TEMPO_OK;
}

static int check_plan(const tempo_plan* p) {
  if (!p || !p->slot_expert || !p->slot_weight || !p->remote_weight || !p->remote_replicas) return TEMPO_EINVAL;
  if (p->flags & ~(TEMPO_PLAN_SNAP_TILES | TEMPO_PLAN_SAMPLE)) return TEMPO_EINVAL;
  if ((p->flags & TEMPO_PLAN_SNAP_TILES) && (p->flags & TEMPO_PLAN_SAMPLE)) return TEMPO_EINVAL;
  return TEMPO_OK;
}

static int check_disp(const tempo_moe_shape* s, const tempo_dispatch_out* d, bool need_index_outputs) {
  if (!d || !d->slot_counts || !d->slot_offsets || !d->row_token || !d->x_perm) return TEMPO_EINVAL;
  if (need_index_outputs && (!d->expert_counts || !d->pair_row)) return TEMPO_EINVAL;
  if (s->dtype != TEMPO_BF16 && !d->x_perm_scale) return TEMPO_EINVAL;
  return TEMPO_OK;
}

static int check_weights(const tempo_moe_shape* s, const tempo_expert_weights* w) {
  if (!w) return TEMPO_EINVAL;
  if (w->slot_table) return TEMPO_OK;  // the entries are device memory, read by the kernels
  if (!w->w13 || !w->w2) return TEMPO_EINVAL;
  if (s->dtype != TEMPO_BF16 && (!w->w13_scale || !w->w2_scale)) return TEMPO_EINVAL;
  return TEMPO_OK;
}

static int dev_status(hipError_t e) { return e == hipSuccess ? TEMPO_OK : TEMPO_EDEVICE; }


}  // namespace tempo

using namespace tempo;

extern "C" {

int tempo_moe_query(const tempo_moe_shape* shape, size_t* workspace_bytes, int32_t* row_cap,
                    size_t* packed_bytes_per_slot) {
  int rc = check_shape(shape);
  if (rc) return rc;
  const Layout L = make_layout(*shape);
  if (workspace_bytes) *workspace_bytes = L.total;
  if (row_cap) *row_cap = L.row_cap;
  if (packed_bytes_per_slot) {
    const size_t H = shape->H, I = shape->I;
    *packed_bytes_per_slot = shape->dtype == TEMPO_BF16
                                 ? 3 * H * I * 2
                                 : 3 * H * I + ((I / 64) * (H / 128) + (H / 128) * (I / 128)) * 16;
  }
  return TEMPO_OK;
}

int tempo_moe_counter_window(int32_t E, const uint32_t* before, const uint32_t* after, uint32_t* window) {
  if (E < 1 || !before || !after || !window) return TEMPO_EINVAL;
  for (int32_t e = 0; e < E; e++) window[e] = after[e] - before[e];  // unsigned: modulo 2^32
  return TEMPO_OK;
}

int tempo_moe_pack_weights(const tempo_moe_shape* shape, const tempo_expert_weights* natural,
                           const tempo_expert_weights* packed, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!natural || !packed || !natural->w13 || !natural->w2 || !packed->w13 || !packed->w2) return TEMPO_EINVAL;
  if (shape->dtype != TEMPO_BF16 &&
      (!natural->w13_scale || !natural->w2_scale || !packed->w13_scale || !packed->w2_scale))
    return TEMPO_EINVAL;
  const size_t es = shape->dtype == TEMPO_BF16 ? 2 : 1;
  const size_t b13 = (size_t)shape->S * 2 * shape->I * shape->H * es, b2 = (size_t)shape->S * shape->H * shape->I * es;
  auto overlap = [](const void* a, size_t na, const void* b, size_t nb) {
    const char *x = static_cast<const char*>(a), *y = static_cast<const char*>(b);
    return x < y + nb && y < x + na;
  };
  if (overlap(natural->w13, b13, packed->w13, b13) || overlap(natural->w2, b2, packed->w2, b2) ||
      overlap(natural->w13, b13, packed->w2, b2) || overlap(natural->w2, b2, packed->w13, b13) ||
      overlap(packed->w13, b13, packed->w2, b2))
    return TEMPO_EINVAL;
  if (shape->dtype != TEMPO_BF16) {
    const size_t kb = shape->H / 128, ib = shape->I / 128;
    const size_t n13 = (size_t)shape->S * 2 * ib * kb * 4, n2 = (size_t)shape->S * kb * ib * 4;
    const size_t p13 = (size_t)shape->S * (shape->I / 64) * kb * 16, p2 = (size_t)shape->S * kb * ib * 16;
    const void* ns[2] = {natural->w13_scale, natural->w2_scale};
    const size_t nn[2] = {n13, n2};
    const void* ps[2] = {packed->w13_scale, packed->w2_scale};
    const size_t pn[2] = {p13, p2};
    if (overlap(ps[0], pn[0], ps[1], pn[1])) return TEMPO_EINVAL;
    for (int i = 0; i < 2; i++)
      for (int j = 0; j < 2; j++)
        if (overlap(ps[i], pn[i], ns[j], nn[j])) return TEMPO_EINVAL;
  }
  return dev_status(launch_pack(*shape, *natural, *packed, static_cast<hipStream_t>(stream)));
}

int tempo_moe_dispatch(const tempo_moe_shape* shape, const tempo_plan* plan, const int32_t* topk_ids, const void* x,
                       const float* x_scale, const tempo_dispatch_out* out, void* workspace, size_t workspace_bytes,
                       void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_plan(plan)) || (rc = check_disp(shape, out, true))) return rc;
  if ((plan->flags & TEMPO_PLAN_SAMPLE) && !dispatch_sample_supported(*shape)) return TEMPO_EUNSUPPORTED;
  if (!topk_ids || !x || !workspace || (shape->dtype != TEMPO_BF16 && !x_scale)) return TEMPO_EINVAL;
  const Layout L = make_layout(*shape);
  if (workspace_bytes < L.total) return TEMPO_EWORKSPACE;
  return dev_status(launch_dispatch(*shape, *plan, topk_ids, x, x_scale, *out, static_cast<char*>(workspace), L,
                                    false, true, true, static_cast<hipStream_t>(stream)));
}

int tempo_moe_experts(const tempo_moe_shape* shape, const tempo_dispatch_out* disp,
                      const tempo_expert_weights* weights, void* y_perm, void* workspace, size_t workspace_bytes,
                      void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_disp(shape, disp, false)) || (rc = check_weights(shape, weights))) return rc;
  if (!y_perm || !workspace) return TEMPO_EINVAL;
  const Layout L = make_layout(*shape);
  if (workspace_bytes < L.total) return TEMPO_EWORKSPACE;
  if (!experts_supported(*shape)) return TEMPO_EUNSUPPORTED;
  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = shape->dtype == TEMPO_BF16
                           ? launch_experts_bf16(*shape, *disp, *weights, nullptr, y_perm, ws, L, false, nullptr, st)
                           : launch_experts_fp8(*shape, *disp, *weights, nullptr, nullptr, y_perm, ws, L, false, nullptr, st);
  if (e == hipErrorNotSupported) return TEMPO_EUNSUPPORTED;
  return dev_status(e);
}

int tempo_moe_combine(const tempo_moe_shape* shape, const int32_t* pair_row, const float* topk_w,
                      const void* y_perm, void* y, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!pair_row || !topk_w || !y_perm || !y) return TEMPO_EINVAL;
  return dev_status(launch_combine(*shape, pair_row, topk_w, y_perm, y, nullptr, nullptr, nullptr, nullptr,
                                   static_cast<hipStream_t>(stream)));
}

int tempo_moe_forward(const tempo_moe_shape* shape, const tempo_plan* plan, const int32_t* topk_ids,
                      const float* topk_w, const void* x, const float* x_scale, const tempo_expert_weights* weights,
                      const tempo_dispatch_out* disp, void* y, uint64_t* slot_time_ns, void* const* stage_events,
                      void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_plan(plan)) || (rc = check_disp(shape, disp, true)) || (rc = check_weights(shape, weights)))
    return rc;
  if ((plan->flags & TEMPO_PLAN_SAMPLE) && !dispatch_sample_supported(*shape)) return TEMPO_EUNSUPPORTED;
  if (!topk_ids || !topk_w || !x || !y || !workspace || (shape->dtype != TEMPO_BF16 && !x_scale))
    return TEMPO_EINVAL;
  const Layout L = make_layout(*shape);
  if (workspace_bytes < L.total) return TEMPO_EWORKSPACE;
  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool timing = slot_time_ns != nullptr;
  void* y_perm = ws + L.y_perm;
  hipEvent_t ev[TEMPO_STAGE_EVENTS] = {};
  if (stage_events)
    for (int i = 0; i < TEMPO_STAGE_EVENTS; i++) ev[i] = static_cast<hipEvent_t>(stage_events[i]);
  auto mark = [&](int i) { return !ev[i] || hipEventRecord(ev[i], st) == hipSuccess; };
  if (!experts_supported(*shape)) return TEMPO_EUNSUPPORTED;
  if (!mark(0)) return TEMPO_EDEVICE;
  // decode-sized batches and the large-tile kernels: stage 2 gathers the
  // activation rows itself and x_perm stays unwritten (the large-tile fp8
  // kernel also reads the token rows' scales); otherwise stage 1 permutes the
  // rows into x_perm
  const bool gemm_gathers = experts_gather_rows(*shape, L);
  const bool own_scales = gemm_gathers && shape->dtype != TEMPO_BF16 && experts_reads_token_scales(*shape);
  const void* x_rows = gemm_gathers ? x : nullptr;
  hipError_t e =
      launch_dispatch(*shape, *plan, topk_ids, x, x_scale, *disp, ws, L, timing, !gemm_gathers, !own_scales, st);
  if (e != hipSuccess || !mark(1)) return TEMPO_EDEVICE;
  e = shape->dtype == TEMPO_BF16
          ? launch_experts_bf16(*shape, *disp, *weights, x_rows, y_perm, ws, L, timing, ev + 2, st)
          : launch_experts_fp8(*shape, *disp, *weights, x_rows, own_scales ? x_scale : nullptr, y_perm, ws, L,
                                       timing, ev + 2, st);
  if (e == hipErrorNotSupported) return TEMPO_EUNSUPPORTED;
  if (e != hipSuccess || !mark(6)) return TEMPO_EDEVICE;
  e = launch_combine(*shape, disp->pair_row, topk_w, y_perm, y, disp->slot_counts,
                     reinterpret_cast<const uint64_t*>(ws + L.slot_t0),
                     reinterpret_cast<const uint64_t*>(ws + L.slot_t1), slot_time_ns, st);
  if (e != hipSuccess || !mark(7)) return TEMPO_EDEVICE;
  return TEMPO_OK;
}

int tempo_moe_device_error(void* workspace, void* stream, uint32_t* bits) {
  if (!workspace || !bits) return TEMPO_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t v = 0;
  uint32_t* word = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace)) + kHdrSticky;
  if (hipMemcpyAsync(&v, word, sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess) return TEMPO_EDEVICE;
  if (hipStreamSynchronize(st) != hipSuccess) return TEMPO_EDEVICE;
  const uint32_t zero = 0;
  if (hipMemcpyAsync(word, &zero, sizeof(zero), hipMemcpyHostToDevice, st) != hipSuccess) return TEMPO_EDEVICE;
  if (hipStreamSynchronize(st) != hipSuccess) return TEMPO_EDEVICE;
  *bits = v;
  return TEMPO_OK;
}

const char* tempo_moe_strerror(int code) {
  switch (code) {
    case TEMPO_OK: return "ok";
    case TEMPO_EINVAL: return "invalid argument";
    case TEMPO_EWORKSPACE: return "workspace too small";
    case TEMPO_EDEVICE: return "HIP runtime error";
    case TEMPO_EUNSUPPORTED: return "unsupported shape or type";
    default: return "unknown error";
  }
}

}  // extern "C"
