// One (d_in, d_out) instantiation of the fused kernel, both modes and both
// activations; compiled once per shape (MOT_FUSED_D_IN, MOT_FUSED_D_OUT set
// by the build) so the instantiations build in parallel.
#include "k_bf16_fused_kernel.h"

#define MOT_CAT3(a, b, c) a##b##_##c
#define MOT_LAUNCH_NAME(a, b) MOT_CAT3(launch_fused_, a, b)

namespace mot {

hipError_t MOT_LAUNCH_NAME(MOT_FUSED_D_IN, MOT_FUSED_D_OUT)(const Problem& p, const UnitTab& ut, bool routed,
                                                           hipStream_t stream) {
    return routed ? launch_t<MOT_FUSED_D_IN, MOT_FUSED_D_OUT, true>(p, ut, stream)
                  : launch_t<MOT_FUSED_D_IN, MOT_FUSED_D_OUT, false>(p, ut, stream);
}

}  // namespace mot
