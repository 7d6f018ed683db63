// Stage 2, fp8 e4m3 with fp32 block scales -- not yet implemented; the
// launcher reports the shape as unsupported.
#include "internal.h"

namespace tempo {

bool experts_supported(const tempo_moe_shape& s) { return s.dtype == TEMPO_BF16; }

hipError_t launch_experts_fp8(const tempo_moe_shape&, const tempo_dispatch_out&, const tempo_expert_weights&, void*,
                              char*, const Layout&, bool, hipEvent_t, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace tempo
