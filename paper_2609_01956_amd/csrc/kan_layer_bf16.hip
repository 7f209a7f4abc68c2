// kan_layer_bf16.hip -- instantiation of the fused layer kernels for bf16
// (see kan_layer_kernel.h).
#include "kan_layer_kernel.h"

namespace kan {

hipError_t launch_layer_bf16(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a,
                          hipStream_t s) {
    return layer_detail::launch_t<uint16_t>(g, c, a, s);
}

}  // namespace kan
