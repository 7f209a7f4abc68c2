// kan_api.cpp -- the C ABI declared in include/kan.h: argument validation
// (host only, before any HIP call), grid constants, launch planning and
// dispatch onto the caller's stream.
#include "kan.h"

#include <cmath>
#include <cstdint>

#include "kan_internal.h"

namespace {

constexpr int32_t kMaxGrid = 4000;

size_t dtype_size(kan_dtype dt) { return dt == KAN_BF16 ? 2 : 4; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// [p, p + n) and [q, q + m) (bytes) intersect?
bool overlap(const void* p, size_t n, const void* q, size_t m) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
    return a < b + m && b < a + n;
}

constexpr int32_t kMaxDegree = 7;

// Validates the grid and dtype and fills the grid constants (kan_device.h):
//   nb = G + k; inv_h + inv_lo = G / (hi - lo); a_int + a_frac = (k - 1) / 2 -
//   lo / h, so that v_j = u_j - (k + 1) / 2 = fma(x, inv_h, a_int - j) +
//   (x inv_lo + a_frac).
kan_status check_grid(const kan_grid* grid, kan_dtype dtype, kan::GridConst* gc) {
    if (grid == nullptr) return KAN_ERR_INVALID_ARG;
    const int32_t k = grid->spline_order;
    if (k < 1 || k > kMaxDegree) return KAN_ERR_UNSUPPORTED;
    if (dtype != KAN_F32 && dtype != KAN_BF16) return KAN_ERR_UNSUPPORTED;
    const int32_t G = grid->grid_size;
    if (G < 1 || G > kMaxGrid) return KAN_ERR_INVALID_ARG;
    const double lo = grid->grid_lo, hi = grid->grid_hi;
    if (!std::isfinite(lo) || !std::isfinite(hi) || !(lo < hi)) return KAN_ERR_INVALID_ARG;
    const double inv_h = (double)G / (hi - lo);
    if (!std::isfinite(inv_h) || !std::isfinite((double)(float)inv_h) || (float)inv_h == 0.0f)
        return KAN_ERR_INVALID_ARG;
    // Keep a_int - j (and x * inv_h near the support) inside fp32's exact
    // integer range.
    const double lim = 4194304.0;  // 2^22
    if (std::fabs(lo) * inv_h > lim || std::fabs(hi) * inv_h > lim) return KAN_ERR_INVALID_ARG;
    const double A = 0.5 * (k - 1) - lo * inv_h;
    const double ai = std::nearbyint(A);
    const float ih = (float)inv_h;
    gc->nb = G + k;
    gc->k = k;
    gc->inv_h = ih;
    gc->inv_lo = (float)(inv_h - (double)ih);
    gc->a_int = (float)ai;
    gc->a_frac = (float)(A - ai);
    gc->xlim = (float)(std::fmax(std::fabs(lo), std::fabs(hi)) + (k + 2) * (hi - lo) / G);
    gc->hw = 0.5f * (float)(k + 1);
    double kf = 1.0, binom = 1.0;
    for (int i = 2; i <= k; ++i) kf *= i;
    for (int m = 0; m < 4; ++m) {
        gc->hc[m] = (float)((m & 1 ? -binom : binom) / (2.0 * kf));
        binom = binom * (double)(k + 1 - m) / (double)(m + 1);
    }
    return KAN_OK;
}

kan_status device_status(hipError_t e) { return e == hipSuccess ? KAN_OK : KAN_ERR_DEVICE; }

}  // namespace

extern "C" {

const char* kan_status_string(kan_status status) {
    switch (status) {
        case KAN_OK: return "KAN_OK: success";
        case KAN_ERR_INVALID_ARG: return "KAN_ERR_INVALID_ARG: invalid size, range, pointer, alignment or overlap";
        case KAN_ERR_UNSUPPORTED:
            return "KAN_ERR_UNSUPPORTED: spline_order outside 1..7 (the backward: other than 3), or "
                   "a dtype other than f32/bf16";
        case KAN_ERR_DEVICE: return "KAN_ERR_DEVICE: the HIP runtime rejected a kernel launch";
        case KAN_ERR_SCRATCH_LIMIT:
            return "KAN_ERR_SCRATCH_LIMIT: the layer's packed weights exceed the 16 MiB scratch of "
                   "kan_layer_forward_noalloc (use kan_layer_forward with a workspace)";
    }
    return "unknown kan_status";
}

int32_t kan_abi_version(void) { return KAN_ABI_VERSION; }

// Shared validation of the basis-only entry points.
static kan_status check_basis(const kan_grid* grid, kan_dtype dtype, const void* x, int64_t n,
                              const void* phi, kan::GridConst* gc) {
    const kan_status st = check_grid(grid, dtype, gc);
    if (st != KAN_OK) return st;
    if (n < 0) return KAN_ERR_INVALID_ARG;
    if (n == 0) return KAN_OK;
    if (n > INT64_MAX / gc->nb) return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    if (x == nullptr || phi == nullptr) return KAN_ERR_INVALID_ARG;
    if (!aligned(x, es) || !aligned(phi, es)) return KAN_ERR_INVALID_ARG;
    if ((uint64_t)n > (uint64_t)(SIZE_MAX / es / gc->nb)) return KAN_ERR_INVALID_ARG;
    if (overlap(x, (size_t)n * es, phi, (size_t)n * gc->nb * es)) return KAN_ERR_INVALID_ARG;
    if ((n + 255) / 256 > 0x7fffffffLL) return KAN_ERR_INVALID_ARG;
    return KAN_OK;
}

kan_status kan_basis_eval_cdb(const kan_grid* grid, kan_dtype dtype, const void* x, int64_t n,
                              void* phi, void* stream) {
    kan::GridConst gc;
    const kan_status st = check_basis(grid, dtype, x, n, phi, &gc);
    if (st != KAN_OK || n == 0) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == KAN_F32)
        return device_status(kan::launch_basis_cdb_f32(static_cast<const float*>(x), n,
                                                       static_cast<float*>(phi), gc, s));
    return device_status(kan::launch_basis_cdb_bf16(static_cast<const uint16_t*>(x), n,
                                                    static_cast<uint16_t*>(phi), gc, s));
}

kan_status kan_basis_eval(const kan_grid* grid, kan_dtype dtype, const void* x, int64_t n,
                          void* phi, void* stream) {
    kan::GridConst gc;
    const kan_status st = check_grid(grid, dtype, &gc);
    if (st != KAN_OK) return st;
    if (n < 0) return KAN_ERR_INVALID_ARG;
    if (n == 0) return KAN_OK;
    if (n > INT64_MAX / gc.nb) return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    if (x == nullptr || phi == nullptr) return KAN_ERR_INVALID_ARG;
    if (!aligned(x, es) || !aligned(phi, es)) return KAN_ERR_INVALID_ARG;
    if ((uint64_t)n > (uint64_t)(SIZE_MAX / es / gc.nb)) return KAN_ERR_INVALID_ARG;
    if (overlap(x, (size_t)n * es, phi, (size_t)n * gc.nb * es)) return KAN_ERR_INVALID_ARG;
    const kan::BasisLaunch L = kan::plan_basis(n, gc.nb, phi);
    if (L.blocks > 0x7fffffffLL) return KAN_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == KAN_F32)
        return device_status(kan::launch_basis_f32(static_cast<const float*>(x), n,
                                                   static_cast<float*>(phi), gc, L, s));
    return device_status(kan::launch_basis_bf16(static_cast<const uint16_t*>(x), n,
                                                static_cast<uint16_t*>(phi), gc, L, s));
}

// Shared validation of the layer entry points: grid, dtype, sizes.
static kan_status check_layer(const kan_grid* grid, kan_dtype dtype, int32_t in_features,
                              int32_t out_features, kan::GridConst* gc, kan::LayerGeom* geom) {
    const kan_status st = check_grid(grid, dtype, gc);
    if (st != KAN_OK) return st;
    if (in_features < 1 || out_features < 1) return KAN_ERR_INVALID_ARG;
    if ((int64_t)in_features * (gc->nb + 1) >= 0x80000000LL) return KAN_ERR_INVALID_ARG;
    // The fused kernel reads x through a per-workgroup buffer resource with
    // 32-bit byte offsets over at most kan::kLayerMaxRows rows (of elements of
    // at most 4 bytes), and each N tile of the packed weights likewise.
    if ((int64_t)kan::kLayerMaxRows * in_features * 4 >= 0x100000000LL) return KAN_ERR_INVALID_ARG;
    if ((int64_t)out_features * in_features * gc->nb >= (1LL << 40)) return KAN_ERR_INVALID_ARG;
    if (!kan::layer_geom(gc->nb, gc->k, dtype == KAN_BF16, in_features, out_features, geom))
        return KAN_ERR_INVALID_ARG;
    if (geom->packed_bytes / (size_t)geom->ntiles >= 0x100000000ULL) return KAN_ERR_INVALID_ARG;
    return KAN_OK;
}

kan_status kan_layer_packed_bytes(const kan_grid* grid, kan_dtype dtype, int32_t in_features,
                                  int32_t out_features, size_t* bytes) {
    if (bytes == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    const kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    *bytes = geom.packed_bytes;
    return KAN_OK;
}

kan_status kan_layer_pack(const kan_grid* grid, kan_dtype dtype, int32_t in_features,
                          int32_t out_features, const void* coef, const void* base_w,
                          void* packed, size_t packed_bytes, void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    const kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (coef == nullptr || base_w == nullptr || packed == nullptr) return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    if (!aligned(coef, es) || !aligned(base_w, es) || !aligned(packed, 16))
        return KAN_ERR_INVALID_ARG;
    if (packed_bytes < geom.packed_bytes) return KAN_ERR_INVALID_ARG;
    const size_t c_bytes = (size_t)out_features * in_features * gc.nb * es;
    const size_t w_bytes = (size_t)out_features * in_features * es;
    if (overlap(packed, geom.packed_bytes, coef, c_bytes) ||
        overlap(packed, geom.packed_bytes, base_w, w_bytes))
        return KAN_ERR_INVALID_ARG;
    return device_status(kan::launch_pack(dtype == KAN_BF16, geom, in_features, out_features,
                                          coef, base_w, packed,
                                          static_cast<hipStream_t>(stream)));
}

// Validates the arguments of a packed forward (after check_layer).
static kan_status check_forward_packed(const kan::LayerGeom& geom, kan_dtype dtype, int64_t batch,
                                       int32_t in_features, int32_t out_features, const void* x,
                                       const void* packed, size_t packed_bytes, const void* y) {
    if (x == nullptr || packed == nullptr || y == nullptr) return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    if (!aligned(x, es) || !aligned(y, es) || !aligned(packed, 16)) return KAN_ERR_INVALID_ARG;
    if (packed_bytes < geom.packed_bytes) return KAN_ERR_INVALID_ARG;
    const uint64_t ub = (uint64_t)batch;
    if (ub > SIZE_MAX / es / (uint64_t)in_features || ub > SIZE_MAX / es / (uint64_t)out_features)
        return KAN_ERR_INVALID_ARG;
    const size_t x_bytes = ub * (size_t)in_features * es;
    const size_t y_bytes = ub * (size_t)out_features * es;
    if (overlap(y, y_bytes, x, x_bytes) || overlap(y, y_bytes, packed, geom.packed_bytes))
        return KAN_ERR_INVALID_ARG;
    return KAN_OK;
}

// The shape a forward launches: the planner's, or a forced one that must be
// valid for the layer.
static kan_status layer_shape(const kan::LayerGeom& geom, kan_dtype dtype, int64_t batch,
                              const int32_t* shape, kan::LayerCfg* cfg) {
    if (shape == nullptr) {
        *cfg = kan::plan_layer(geom, dtype == KAN_BF16, batch);
        return KAN_OK;
    }
    const kan::LayerCfg c{shape[0], shape[1], shape[2], shape[3]};
    if (!kan::layer_cfg_valid(geom, c)) return KAN_ERR_INVALID_ARG;
    *cfg = c;
    return KAN_OK;
}

// Enqueues the fused kernel (arguments already validated).
static kan_status launch_forward(const kan::GridConst& gc, const kan::LayerGeom& geom,
                                 const kan::LayerCfg& cfg, kan_dtype dtype, int64_t batch,
                                 int32_t in_features, int32_t out_features, const void* x,
                                 const void* packed, int ks, void* partial, void* y,
                                 hipStream_t s) {
    kan::LayerArgs a;
    a.x = x;
    a.wp = packed;
    a.y = y;
    a.batch = batch;
    a.in = in_features;
    a.out = out_features;
    a.nb = gc.nb;
    a.nsb = geom.nsb;
    a.npairs = geom.npairs;
    a.nblk = geom.nblk;
    a.nblk_pad = geom.nblk_pad;
    a.nchunks = 0;  // set by the launcher (depends on the tile shape)
    a.cps = 0;      // set by the launcher (from ks)
    a.P = nullptr;
    a.inv_h = gc.inv_h;
    a.inv_lo = gc.inv_lo;
    a.xlim = gc.xlim;
    a.a_int = gc.a_int;
    a.a_frac = gc.a_frac;
    a.kdeg = gc.k;
    a.hw = gc.hw;
    for (int m = 0; m < 4; ++m) a.hc[m] = gc.hc[m];
    return device_status(kan::launch_layer(dtype == KAN_BF16, geom, cfg, a, ks, partial, s));
}

kan_status kan_layer_forward_packed(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                    int32_t in_features, int32_t out_features, const void* x,
                                    const void* packed, size_t packed_bytes,
                                    const int32_t* shape, void* workspace,
                                    size_t workspace_bytes, void* y, void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 0) return KAN_ERR_INVALID_ARG;
    // Row tiles of at least 32 rows go in blockIdx.x.
    if (batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    kan::LayerCfg cfg;
    st = layer_shape(geom, dtype, batch < 1 ? 1 : batch, shape, &cfg);
    if (st != KAN_OK) return st;
    if (batch == 0) return KAN_OK;
    st = check_forward_packed(geom, dtype, batch, in_features, out_features, x, packed,
                              packed_bytes, y);
    if (st != KAN_OK) return st;
    // The K split of small batches runs when the workspace holds its partial
    // sums; without one the layer runs unsplit (same result up to the fp32
    // summation order).
    int ks = kan::layer_k_splits(geom, cfg, batch, out_features);
    const size_t pbytes = kan::layer_partial_bytes(geom, cfg, batch, out_features);
    if (ks > 1 && (workspace == nullptr || workspace_bytes < pbytes)) ks = 1;
    if (ks > 1) {
        const size_t es = dtype_size(dtype);
        const uint64_t ub = (uint64_t)batch;
        if (!aligned(workspace, 16) ||
            overlap(workspace, pbytes, x, ub * (size_t)in_features * es) ||
            overlap(workspace, pbytes, packed, geom.packed_bytes) ||
            overlap(workspace, pbytes, y, ub * (size_t)out_features * es))
            return KAN_ERR_INVALID_ARG;
    }
    return launch_forward(gc, geom, cfg, dtype, batch, in_features, out_features, x, packed, ks,
                          ks > 1 ? workspace : nullptr, y, static_cast<hipStream_t>(stream));
}

kan_status kan_layer_forward_packed_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                                    int64_t batch, int32_t in_features,
                                                    int32_t out_features, const int32_t* shape,
                                                    size_t* bytes) {
    if (bytes == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 0 || batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    kan::LayerCfg cfg;
    st = layer_shape(geom, dtype, batch < 1 ? 1 : batch, shape, &cfg);
    if (st != KAN_OK) return st;
    *bytes = batch == 0 ? 0 : kan::layer_partial_bytes(geom, cfg, batch, out_features);
    return KAN_OK;
}

kan_status kan_layer_plan(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                          int32_t in_features, int32_t out_features, const int32_t* shape,
                          int32_t* plan) {
    if (plan == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 1 || batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    kan::LayerCfg cfg;
    st = layer_shape(geom, dtype, batch, shape, &cfg);
    if (st != KAN_OK) return st;
    plan[0] = cfg.rf;
    plan[1] = cfg.wk;
    plan[2] = cfg.nw;
    plan[3] = cfg.cs;
    plan[4] = geom.sparse ? 1 : 0;
    plan[5] = kan::layer_k_splits(geom, cfg, batch, out_features);
    return KAN_OK;
}

kan_status kan_layer_forward_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                             int64_t batch, int32_t in_features,
                                             int32_t out_features, size_t* bytes) {
    if (bytes == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    const kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 0 || batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    // the packed weights, then (small batches) the K split's partial sums
    const kan::LayerCfg cfg = kan::plan_layer(geom, dtype == KAN_BF16, batch < 1 ? 1 : batch);
    const size_t pbytes =
        batch == 0 ? 0 : kan::layer_partial_bytes(geom, cfg, batch, out_features);
    *bytes = pbytes == 0 ? geom.packed_bytes : align256(geom.packed_bytes) + pbytes;
    return KAN_OK;
}

// Validates kan_layer_forward's tensors (after check_layer, batch > 0).
static kan_status check_forward(const kan::GridConst& gc, kan_dtype dtype, int64_t batch,
                                int32_t in_features, int32_t out_features, const void* x,
                                const void* coef, const void* base_w, const void* y) {
    if (x == nullptr || coef == nullptr || base_w == nullptr || y == nullptr)
        return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    if (!aligned(x, es) || !aligned(coef, es) || !aligned(base_w, es) || !aligned(y, es))
        return KAN_ERR_INVALID_ARG;
    if (batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    const uint64_t ub = (uint64_t)batch;
    if (ub > SIZE_MAX / es / (uint64_t)in_features || ub > SIZE_MAX / es / (uint64_t)out_features)
        return KAN_ERR_INVALID_ARG;
    const size_t x_bytes = ub * (size_t)in_features * es;
    const size_t c_bytes = (size_t)out_features * in_features * gc.nb * es;
    const size_t w_bytes = (size_t)out_features * in_features * es;
    const size_t y_bytes = ub * (size_t)out_features * es;
    if (overlap(y, y_bytes, x, x_bytes) || overlap(y, y_bytes, coef, c_bytes) ||
        overlap(y, y_bytes, base_w, w_bytes))
        return KAN_ERR_INVALID_ARG;
    return KAN_OK;
}

kan_status kan_layer_forward(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                             int32_t in_features, int32_t out_features, const void* x,
                             const void* coef, const void* base_w, void* workspace,
                             size_t workspace_bytes, void* y, void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 0) return KAN_ERR_INVALID_ARG;
    if (batch == 0) return KAN_OK;
    st = check_forward(gc, dtype, batch, in_features, out_features, x, coef, base_w, y);
    if (st != KAN_OK) return st;
    if (workspace == nullptr || !aligned(workspace, 16) || workspace_bytes < geom.packed_bytes)
        return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    const uint64_t ub = (uint64_t)batch;
    const size_t ws = geom.packed_bytes;
    // (the whole workspace: past the packed weights it may hold partial sums)
    if (overlap(workspace, workspace_bytes, x, ub * (size_t)in_features * es) ||
        overlap(workspace, workspace_bytes, coef, (size_t)out_features * in_features * gc.nb * es) ||
        overlap(workspace, workspace_bytes, base_w, (size_t)out_features * in_features * es) ||
        overlap(workspace, workspace_bytes, y, ub * (size_t)out_features * es))
        return KAN_ERR_INVALID_ARG;
    st = kan_layer_pack(grid, dtype, in_features, out_features, coef, base_w, workspace, ws,
                        stream);
    if (st != KAN_OK) return st;
    // the rest of the workspace, past the packed weights, for the K split
    const size_t off = align256(ws);
    void* rest = workspace_bytes > off ? static_cast<char*>(workspace) + off : nullptr;
    const size_t rest_bytes = workspace_bytes > off ? workspace_bytes - off : 0;
    return kan_layer_forward_packed(grid, dtype, batch, in_features, out_features, x, workspace,
                                    ws, nullptr, rest, rest_bytes, y, stream);
}

kan_status kan_layer_forward_noalloc(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                     int32_t in_features, int32_t out_features, const void* x,
                                     const void* coef, const void* base_w, void* y,
                                     void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (batch < 0) return KAN_ERR_INVALID_ARG;
    if (geom.packed_bytes > (size_t)KAN_NOALLOC_SCRATCH_BYTES) return KAN_ERR_SCRATCH_LIMIT;
    if (batch == 0) return KAN_OK;
    st = check_forward(gc, dtype, batch, in_features, out_features, x, coef, base_w, y);
    if (st != KAN_OK) return st;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    if (kan::noalloc_scratch(&ws, &ws_bytes) != hipSuccess) return KAN_ERR_DEVICE;
    // (the scratch is the library's own device array: it overlaps no caller
    // tensor)
    st = kan_layer_pack(grid, dtype, in_features, out_features, coef, base_w, ws,
                        geom.packed_bytes, stream);
    if (st != KAN_OK) return st;
    // the scratch past the packed weights holds the K split's partial sums
    // when they fit (else the layer runs unsplit)
    const size_t off = align256(geom.packed_bytes);
    void* rest = ws_bytes > off ? static_cast<char*>(ws) + off : nullptr;
    const size_t rest_bytes = ws_bytes > off ? ws_bytes - off : 0;
    return kan_layer_forward_packed(grid, dtype, batch, in_features, out_features, x, ws,
                                    geom.packed_bytes, nullptr, rest, rest_bytes, y, stream);
}

// Backward geometry (after check_layer): the batch must fit the kernels' grids.
static kan_status backward_geom(const kan::GridConst& gc, kan_dtype dtype, int64_t batch,
                                int32_t in_features, int32_t out_features, kan::BwdGeom* bg) {
    if (batch < 0 || batch > (int64_t)0x7fffffff * 32) return KAN_ERR_INVALID_ARG;
    if (!kan::bwd_geom(gc.nb, dtype == KAN_BF16, batch, in_features, out_features, bg))
        return KAN_ERR_INVALID_ARG;
    return KAN_OK;
}

kan_status kan_layer_backward_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                              int64_t batch, int32_t in_features,
                                              int32_t out_features, size_t* bytes) {
    if (bytes == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (gc.k != 3) return KAN_ERR_UNSUPPORTED;
    kan::BwdGeom bg;
    st = backward_geom(gc, dtype, batch, in_features, out_features, &bg);
    if (st != KAN_OK) return st;
    *bytes = bg.bytes;
    return KAN_OK;
}

kan_status kan_layer_backward(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                              int32_t in_features, int32_t out_features, const void* x,
                              const void* coef, const void* base_w, const void* dy, void* dx,
                              void* dcoef, void* dbase_w, void* workspace,
                              size_t workspace_bytes, void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    if (gc.k != 3) return KAN_ERR_UNSUPPORTED;  // (the backward kernels are cubic)
    kan::BwdGeom bg;
    st = backward_geom(gc, dtype, batch, in_features, out_features, &bg);
    if (st != KAN_OK) return st;
    if ((dcoef == nullptr) != (dbase_w == nullptr)) return KAN_ERR_INVALID_ARG;
    if (dx == nullptr && dcoef == nullptr) return KAN_ERR_INVALID_ARG;
    const bool need_x = batch > 0;
    if (need_x && (x == nullptr || dy == nullptr)) return KAN_ERR_INVALID_ARG;
    if (dx != nullptr && need_x && (coef == nullptr || base_w == nullptr))
        return KAN_ERR_INVALID_ARG;
    if (workspace == nullptr || !aligned(workspace, 16) || workspace_bytes < bg.bytes)
        return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    const uint64_t ub = (uint64_t)batch;
    if (ub > SIZE_MAX / es / (uint64_t)in_features || ub > SIZE_MAX / es / (uint64_t)out_features)
        return KAN_ERR_INVALID_ARG;
    struct Buf { const void* p; size_t n; };
    const size_t x_b = ub * (size_t)in_features * es;
    const size_t y_b = ub * (size_t)out_features * es;
    const size_t c_b = (size_t)out_features * in_features * gc.nb * es;
    const size_t w_b = (size_t)out_features * in_features * es;
    const Buf ins[] = {{need_x ? x : nullptr, x_b}, {dx ? coef : nullptr, c_b},
                       {dx ? base_w : nullptr, w_b}, {need_x ? dy : nullptr, y_b}};
    const Buf outs[] = {{dx, x_b}, {dcoef, c_b}, {dbase_w, w_b}, {workspace, bg.bytes}};
    for (const Buf& o : outs) {
        if (o.p == nullptr || o.n == 0) continue;
        if (!aligned(o.p, es)) return KAN_ERR_INVALID_ARG;
        for (const Buf& i : ins)
            if (i.p != nullptr && i.n > 0 && overlap(o.p, o.n, i.p, i.n)) return KAN_ERR_INVALID_ARG;
        for (const Buf& q : outs)
            if (&q != &o && q.p != nullptr && q.n > 0 && overlap(o.p, o.n, q.p, q.n))
                return KAN_ERR_INVALID_ARG;
    }
    for (const Buf& i : ins)
        if (i.p != nullptr && !aligned(i.p, es)) return KAN_ERR_INVALID_ARG;
    if (batch == 0 && dx != nullptr && dcoef == nullptr) return KAN_OK;
    kan::BwdArgs a;
    a.x = x;
    a.coef = coef;
    a.bw = base_w;
    a.dy = dy;
    a.dx = batch > 0 ? dx : nullptr;
    a.dcoef = dcoef;
    a.dbw = dbase_w;
    a.ws = workspace;
    a.batch = batch;
    a.in = in_features;
    a.out = out_features;
    a.inv_h = gc.inv_h;
    a.inv_lo = gc.inv_lo;
    a.xlim = gc.xlim;
    a.a_int = gc.a_int;
    a.a_frac = gc.a_frac;
    return device_status(kan::launch_backward(dtype == KAN_BF16, bg, a,
                                              static_cast<hipStream_t>(stream)));
}

// Span-sparse geometry (after check_layer).
static kan_status span_geom_of(const kan::GridConst& gc, int64_t batch, int32_t in_features,
                               int32_t out_features, kan::SpanGeom* sg) {
    if (batch < 0 || batch > (int64_t)0x7fffffff * 256) return KAN_ERR_INVALID_ARG;
    if (!kan::span_geom(gc.nb, batch, in_features, out_features, sg)) return KAN_ERR_UNSUPPORTED;
    return KAN_OK;
}

kan_status kan_layer_forward_span_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                                  int64_t batch, int32_t in_features,
                                                  int32_t out_features, size_t* bytes) {
    if (bytes == nullptr) return KAN_ERR_INVALID_ARG;
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    kan::SpanGeom sg;
    st = span_geom_of(gc, batch, in_features, out_features, &sg);
    if (st != KAN_OK) return st;
    *bytes = sg.bytes;
    return KAN_OK;
}

kan_status kan_layer_forward_span(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                  int32_t in_features, int32_t out_features, const void* x,
                                  const void* coef, const void* base_w, void* workspace,
                                  size_t workspace_bytes, void* y, void* stream) {
    kan::GridConst gc;
    kan::LayerGeom geom;
    kan_status st = check_layer(grid, dtype, in_features, out_features, &gc, &geom);
    if (st != KAN_OK) return st;
    kan::SpanGeom sg;
    st = span_geom_of(gc, batch, in_features, out_features, &sg);
    if (st != KAN_OK) return st;
    if (batch == 0) return KAN_OK;
    st = check_forward(gc, dtype, batch, in_features, out_features, x, coef, base_w, y);
    if (st != KAN_OK) return st;
    if (workspace == nullptr || !aligned(workspace, 16) || workspace_bytes < sg.bytes)
        return KAN_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    const uint64_t ub = (uint64_t)batch;
    const size_t ws = sg.bytes;
    if (overlap(workspace, ws, x, ub * (size_t)in_features * es) ||
        overlap(workspace, ws, coef, (size_t)out_features * in_features * gc.nb * es) ||
        overlap(workspace, ws, base_w, (size_t)out_features * in_features * es) ||
        overlap(workspace, ws, y, ub * (size_t)out_features * es))
        return KAN_ERR_INVALID_ARG;
    kan::SpanArgs a;
    a.x = x;
    a.wt = nullptr;
    a.y = y;
    a.ws = workspace;
    a.off_p = sg.off_p;
    a.batch = batch;
    a.in = in_features;
    a.out = out_features;
    a.nb = gc.nb;
    a.outp = sg.outp;
    a.fs = sg.fs;
    a.fpf = sg.fpf;
    a.cs = sg.cs;
    a.inv_h = gc.inv_h;
    a.inv_lo = gc.inv_lo;
    a.xlim = gc.xlim;
    a.a_int = gc.a_int;
    a.a_frac = gc.a_frac;
    a.kdeg = gc.k;
    a.hw = gc.hw;
    for (int m = 0; m < 4; ++m) a.hc[m] = gc.hc[m];
    return device_status(kan::launch_span(dtype == KAN_BF16, sg, a, coef, base_w,
                                          static_cast<hipStream_t>(stream)));
}

}  // extern "C"
