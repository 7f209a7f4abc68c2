// kan_internal.h -- host-side launch interface between the C ABI layer and the
// kernel translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kan_device.h"

namespace kan {

// Launch geometry of the basis-only kernel, chosen on the host.
struct BasisLaunch {
    int tpx;        // threads per input element (power of two, 1..64)
    int xb;         // input elements per 256-thread block (256 / tpx)
    int jc;         // basis functions per thread, ceil(nb / tpx)
    size_t lds;     // dynamic LDS bytes, xb * nb * 4
    int64_t blocks; // ceil(n / xb)
    bool vec;       // output pointer is 16-byte aligned: vector stores allowed
                    // (each workgroup still checks its own run)
};

BasisLaunch plan_basis(int64_t n, int nb, const void* phi);

hipError_t launch_basis_f32(const float* x, int64_t n, float* phi, const GridConst& g,
                            const BasisLaunch& L, hipStream_t s);
hipError_t launch_basis_bf16(const uint16_t* x, int64_t n, uint16_t* phi, const GridConst& g,
                             const BasisLaunch& L, hipStream_t s);

// Fused layer: tile configuration.  A workgroup is four waves arranged
// wm x wn; each wave owns a 32-row x (32 * nt)-column tile of y.
struct LayerTile {
    int nt;  // 32-column MFMA tiles per wave: 1, 2, 4 or 8
    int wm;  // waves along the batch dimension
    int wn;  // waves along the output dimension (wm * wn == 4)
};

// Columns per feature per K-step, upper bound (LDS tile width); the host picks
// cw = min(next power of two >= nbp, this bound).
constexpr int kLayerCwMaxF32 = 16;
constexpr int kLayerCwMaxBf16 = 32;
// MFMA k per lane half: 1 for v_mfma_f32_32x32x2_f32, 8 for 32x32x16 bf16.
constexpr int kLayerKGroupF32 = 1;
constexpr int kLayerKGroupBf16 = 8;

struct LayerArgs {
    const void* x;     // [batch, in]
    const void* coef;  // [out, in, nb]
    const void* wb;    // [out, in]
    void* y;           // [batch, out]
    int64_t batch;
    int in;
    int out;
    int nbp;      // per-feature column count (nb spline + 1 SiLU) padded to the MFMA k-group
    int cw;       // columns per feature per K-step (power of two)
    int nchunks;  // ceil(nbp / cw)
    GridConst g;
};

LayerTile plan_layer_tile(int64_t batch, int out);
bool parse_layer_tile_override(LayerTile* t);

hipError_t launch_layer_f32(const LayerArgs& a, const LayerTile& t, hipStream_t s);
hipError_t launch_layer_bf16(const LayerArgs& a, const LayerTile& t, hipStream_t s);

}  // namespace kan
