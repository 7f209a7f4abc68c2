// kan_layer_f32.hip -- instantiation of the fused layer kernels for fp32
// (see kan_layer_kernel.h).
#include "kan_layer_kernel.h"

namespace kan {

hipError_t launch_layer_f32(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a,
                          hipStream_t s) {
    return layer_detail::launch_t<float>(g, c, a, s);
}

}  // namespace kan
