// tempo_moe_forward_static: tempo_moe_forward for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).  Its workspace is `scratch`, a
// file-scope device array of TEMPO_STATIC_SCRATCH_BYTES that every GPU the
// library runs on holds until the process ends; the call allocates nothing.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace {

static __device__ __align__(256) char scratch[TEMPO_STATIC_SCRATCH_BYTES];

// Device address of each GPU's copy of `scratch`, looked up once per device
// with that device current (in host code the array's name is a host-side
// stand-in, not a device address).
constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_scratch[kMaxDevices];
hipError_t g_status[kMaxDevices];

void* scratch_of_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::call_once(g_once[dev], [dev]() {
    void* p = nullptr;
    g_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch[dev] = g_status[dev] == hipSuccess ? p : nullptr;
  });
  return g_status[dev] == hipSuccess ? g_scratch[dev] : nullptr;
}

}  // namespace

extern "C" int tempo_moe_forward_static(const tempo_moe_shape* shape, const tempo_plan* plan,
                                        const int32_t* topk_ids, const float* topk_w, const void* x,
                                        const float* x_scale, const tempo_expert_weights* weights,
                                        const tempo_dispatch_out* disp, void* y, uint64_t* slot_time_ns,
                                        void* const* stage_events, void* stream) {
  // the size check needs no device: shapes beyond the array are refused first
  size_t need = 0;
  const int rc = tempo_moe_query(shape, &need, nullptr, nullptr);
  if (rc != TEMPO_OK) return rc;
  if (need > (size_t)TEMPO_STATIC_SCRATCH_BYTES) return TEMPO_EWORKSPACE;
  void* ws = scratch_of_current_device();
  if (!ws) return TEMPO_EDEVICE;
  return tempo_moe_forward(shape, plan, topk_ids, topk_w, x, x_scale, weights, disp, y, slot_time_ns, stage_events,
                           ws, (size_t)TEMPO_STATIC_SCRATCH_BYTES, stream);
}
