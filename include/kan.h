/*
 * kan.h -- C ABI of the MI355X (gfx950) InKAN KAN layer.
 *
 * The library evaluates uniform B-spline KAN layers with the basis in clamped
 * truncated-power form (paper: Sec. 2 "Step 4", eq. truncated for cubics and
 * eq. general_truncated for other degrees, with the bounded coordinate of
 * eq. bounded) and contracts it with the spline coefficients plus the SiLU
 * base branch (eq. kan_forward); it also computes the layer's gradients.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Pointers named x, phi, coef, base_w, packed, y are DEVICE pointers owned
 *    by the caller.  No entry point allocates device or host memory; where a
 *    call needs scratch memory the caller passes it (a workspace pointer with
 *    a size query).  The library keeps no global state; calls are reentrant
 *    and thread-safe.
 *  * Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is the
 *    null stream) and returns before it finishes.  Results are visible after the
 *    caller synchronises that stream.  A device fault inside a kernel surfaces at
 *    that synchronisation, not in the return code.
 *  * Tensors are dense and row-major.  `dtype` applies to every tensor of a call:
 *    KAN_F32 is IEEE binary32 throughout; KAN_BF16 is bfloat16 storage with
 *    binary32 basis evaluation and accumulation, rounded to nearest-even on
 *    store.
 *  * Grid: G = grid_size intervals of width h = (grid_hi - grid_lo) / G and
 *    degree k = spline_order.  The knot vector is t_j = grid_lo + (j - k) h,
 *    j = 0 .. G + 2k, which gives nb = G + k basis functions; basis j is
 *    supported on [t_j, t_{j+k+1}] (uniform simple knots, Sec. 2 "Step 3";
 *    the extension by k spans on each side of [grid_lo, grid_hi] is this
 *    library's grid convention).  The paper implements k = 3 only (Sec. 5);
 *    this library evaluates eq. general_truncated for 1 <= k <= 7 (the cubic
 *    on its tuned kernels) and the backward for k = 3.  Knots are always
 *    uniform; there is no way to pass a non-uniform knot vector (Sec. 5).
 *  * Accuracy: the basis is evaluated in binary32 as
 *      u_j = x / h - grid_lo / h + k - j   (a fused multiply-add with the fp32
 *                                           1/h, plus x times the rounding
 *                                           residual of 1/h and the fraction
 *                                           of grid_lo / h),
 *      N_j = clamp-based truncated power of u_j     (eq. truncated + eq. bounded),
 *    where the clamp to [0, k + 1] makes every basis exactly 0 off its
 *    support.  The basis is within 1e-6 of the exact value in binary32;
 *    inputs within the coordinate's rounding (about 2^-23 h) of a support end
 *    may land on either side of it.
 *  * Validation happens on the host before any HIP call, and every invalid
 *    argument returns its code without touching the device.  An empty problem
 *    (n == 0 or batch == 0) returns KAN_OK and launches nothing.
 *  * No C++ exception crosses this interface.
 */
#ifndef KAN_H
#define KAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kan_status {
    KAN_OK = 0,
    KAN_ERR_INVALID_ARG = 1, /* bad size, range, pointer, alignment or overlap   */
    KAN_ERR_UNSUPPORTED = 2, /* spline_order outside 1..7 (backward: != 3) or an
                                unknown dtype                                   */
    KAN_ERR_DEVICE = 3,      /* the HIP runtime rejected a launch               */
    KAN_ERR_SCRATCH_LIMIT = 4 /* kan_layer_forward_noalloc: the layer's packed
                                 weights exceed KAN_NOALLOC_SCRATCH_BYTES       */
} kan_status;

typedef enum kan_dtype {
    KAN_F32 = 0,  /* binary32 storage and arithmetic                          */
    KAN_BF16 = 1  /* bfloat16 storage, binary32 arithmetic and accumulation   */
} kan_dtype;

typedef struct kan_grid {
    int32_t grid_size;    /* G, number of grid intervals, 1 <= G <= 4000      */
    int32_t spline_order; /* k, 1 <= k <= 7 (the backward: 3)                   */
    float grid_lo;        /* finite, grid_lo < grid_hi                          */
    float grid_hi;        /* |grid_lo| / h and |grid_hi| / h at most 2^22       */
} kan_grid;

/*
 * kan_basis_eval -- basis-only evaluation (the elementwise truncated-power
 * basis of eq. truncated / eq. general_truncated with the clamp of
 * eq. bounded).
 *
 *   x    [n]           input values, any shape flattened; dtype storage.
 *   phi  [n, G + k]    output, basis index fastest: phi[e * (G+k) + j] = N_j(x[e]).
 *
 * phi must not overlap x.  x and phi must be aligned to the dtype size.
 * A NaN input gives NaN in all G + k outputs of that element; +-Inf gives 0.
 *
 * Returns KAN_OK, KAN_ERR_INVALID_ARG (grid == NULL, bad grid, n < 0,
 * NULL/misaligned/overlapping pointers with n > 0, n * (G + k) overflowing
 * int64), KAN_ERR_UNSUPPORTED (spline_order outside 1..7, unknown dtype) or
 * KAN_ERR_DEVICE (launch rejected).
 */
kan_status kan_basis_eval(const kan_grid* grid, kan_dtype dtype, const void* x,
                          int64_t n, void* phi, void* stream);

/*
 * kan_basis_eval_cdb -- the same basis-only evaluation as kan_basis_eval, by
 * the Cox-de Boor recursion (eq. cdb0, eq. cdbk) over all G + 2k knot
 * intervals (no span lookup), the evaluation the paper compares its
 * truncated-power form against (Sec. 4, Tables 1 and 3).  For measuring that
 * comparison on this hardware; results equal kan_basis_eval's up to the
 * rounding of the recursion (half-open intervals: an input exactly on the last
 * knot gives 0, as the clamped form).
 *
 * Arguments, layout, NaN/Inf behaviour and return codes as kan_basis_eval.
 */
kan_status kan_basis_eval_cdb(const kan_grid* grid, kan_dtype dtype, const void* x,
                              int64_t n, void* phi, void* stream);

/*
 * kan_layer_forward -- one KAN layer (eq. kan_forward):
 *
 *   y[b, o] = sum_i ( sum_j coef[o, i, j] N_j(x[b, i])  +  base_w[o, i] silu(x[b, i]) )
 *
 * with silu(v) = v / (1 + exp(-v)).  coef are the effective spline
 * coefficients (the layer has no separate spline scaler, Sec. 2 "Integration
 * with KAN layers").
 *
 *   x          [batch, in_features]              dtype storage
 *   coef       [out_features, in_features, G+k]  dtype storage
 *   base_w     [out_features, in_features]       dtype storage
 *   workspace  caller-owned device scratch of workspace_bytes >=
 *              kan_layer_forward_workspace_bytes(...) bytes, 16-byte aligned,
 *              overlapping no other argument; its contents are overwritten
 *              (it receives the packed weights) and are of no use afterwards.
 *              It must stay allocated until the enqueued work has finished.
 *   y          [batch, out_features]             dtype storage, fully overwritten
 *
 * The contraction runs on the matrix cores over K = in_features * (G + k + 1)
 * columns (G + k basis values and one SiLU value per input feature); the basis
 * is generated in registers and never written to memory.  The call is
 * kan_layer_pack into the workspace followed by kan_layer_forward_packed,
 * both enqueued on `stream`; the workspace past the packed weights (from the
 * next 256-byte boundary) is the packed forward's workspace.
 *
 * y must not overlap any input.  Every pointer must be aligned to the dtype
 * size.  A NaN in x[b, :] makes y[b, :] NaN (through the SiLU branch).
 *
 * Returns KAN_OK, KAN_ERR_INVALID_ARG (grid == NULL, bad grid, batch < 0,
 * in_features < 1, out_features < 1, in_features * (G + k + 1) >= 2^31,
 * in_features >= 2^24, NULL/misaligned/overlapping pointers or a short
 * workspace with batch > 0), KAN_ERR_UNSUPPORTED (spline_order outside 1..7, unknown
 * dtype) or KAN_ERR_DEVICE (launch rejected).
 */
kan_status kan_layer_forward(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                             int32_t in_features, int32_t out_features,
                             const void* x, const void* coef, const void* base_w,
                             void* workspace, size_t workspace_bytes,
                             void* y, void* stream);

/*
 * kan_layer_forward_workspace_bytes -- size in bytes of the workspace that
 * kan_layer_forward uses for a layer (eq. kan_forward) of this grid, dtype,
 * batch and shape: the packed weights (kan_layer_packed_bytes, the least
 * kan_layer_forward accepts) and, for batches too small to fill the GPU, the
 * fp32 partial sums of the split contraction from the next 256-byte boundary
 * (kan_layer_forward_packed_workspace_bytes).  With only the packed weights'
 * size the layer runs unsplit.
 * Writes *bytes.  Returns KAN_OK, KAN_ERR_INVALID_ARG (bytes == NULL, bad grid
 * or sizes, batch < 0) or KAN_ERR_UNSUPPORTED.
 */
kan_status kan_layer_forward_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                             int64_t batch, int32_t in_features,
                                             int32_t out_features, size_t* bytes);

/*
 * kan_layer_packed_bytes -- size in bytes of the packed weights of a layer
 * (eq. kan_forward) with this grid, dtype and shape; independent of the batch.
 * Writes *bytes.  Returns KAN_OK, KAN_ERR_INVALID_ARG (bytes == NULL, bad grid
 * or sizes) or KAN_ERR_UNSUPPORTED.
 */
kan_status kan_layer_packed_bytes(const kan_grid* grid, kan_dtype dtype, int32_t in_features,
                                  int32_t out_features, size_t* bytes);

/*
 * kan_layer_pack -- rearranges the weights of a layer (eq. kan_forward: the
 * spline coefficients coef[o, i, j] and the SiLU weights base_w[o, i]) into
 * the order in which the matrix cores consume them: for each tile of output
 * columns, feature pair and block of columns, the weights of both features for
 * every output column, the SiLU weight before the G + k spline coefficients of
 * its feature and zeros in the padding (in bf16 with k = 3 and 5 <= G <= 12 a
 * feature's 16 columns are permuted for the structured-sparse matrix
 * instruction).  The
 * layout is private to this library and depends only on (grid, dtype,
 * in_features, out_features).  Weights that do not change can be packed once
 * and reused by any number of kan_layer_forward_packed calls.
 *
 *   coef    [out_features, in_features, G+k]  dtype storage
 *   base_w  [out_features, in_features]       dtype storage
 *   packed  packed_bytes >= kan_layer_packed_bytes(...), 16-byte aligned,
 *           not overlapping coef or base_w; fully overwritten.
 *
 * Enqueued on `stream`.  Returns KAN_OK, KAN_ERR_INVALID_ARG, KAN_ERR_UNSUPPORTED
 * or KAN_ERR_DEVICE, as kan_layer_forward.
 */
kan_status kan_layer_pack(const kan_grid* grid, kan_dtype dtype, int32_t in_features,
                          int32_t out_features, const void* coef, const void* base_w,
                          void* packed, size_t packed_bytes, void* stream);

/*
 * kan_layer_forward_packed -- kan_layer_forward with weights already packed by
 * kan_layer_pack for the same (grid, dtype, in_features, out_features).
 *
 *   x       [batch, in_features]    dtype storage
 *   packed  output of kan_layer_pack, packed_bytes >= kan_layer_packed_bytes(...)
 *   shape   NULL: the workgroup shape the library plans for this layer and
 *           batch (what kan_layer_plan reports).  Otherwise four int32
 *           {rf, wk, nw, cs} as in kan_layer_plan's plan[0..3], forcing that
 *           shape (for testing and tuning; every valid shape gives the same
 *           result up to the fp32 summation order); a shape that is not valid
 *           for the layer is KAN_ERR_INVALID_ARG.
 *   workspace  NULL, or caller-owned device memory of workspace_bytes bytes.
 *           For batches too small to fill the GPU (kan_layer_plan's plan[5]
 *           > 1) the contraction over K is split across workgroups, each
 *           writing fp32 partial sums here, which are then added in a fixed
 *           order (deterministic); that needs workspace_bytes >=
 *           kan_layer_forward_packed_workspace_bytes(...), a 16-byte aligned
 *           workspace overlapping no other argument.  A NULL or smaller
 *           workspace runs the layer unsplit (same result up to the fp32
 *           summation order).
 *   y       [batch, out_features]   dtype storage, fully overwritten; must not
 *           overlap x or packed.
 *
 * Returns as kan_layer_forward.
 */
kan_status kan_layer_forward_packed(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                    int32_t in_features, int32_t out_features, const void* x,
                                    const void* packed, size_t packed_bytes,
                                    const int32_t* shape, void* workspace,
                                    size_t workspace_bytes, void* y, void* stream);

/*
 * kan_layer_forward_packed_workspace_bytes -- size in bytes of the partial
 * sums kan_layer_forward_packed writes when it splits the contraction for
 * this layer, batch and shape (NULL: the planned shape), 0 when it does not
 * split.  Writes *bytes.  Returns KAN_OK, KAN_ERR_INVALID_ARG (bytes == NULL,
 * bad grid or sizes, batch < 0, an invalid forced shape) or
 * KAN_ERR_UNSUPPORTED.
 */
kan_status kan_layer_forward_packed_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                                    int64_t batch, int32_t in_features,
                                                    int32_t out_features, const int32_t* shape,
                                                    size_t* bytes);

/*
 * kan_layer_plan -- the workgroup shape that kan_layer_forward_packed (and
 * kan_layer_forward) launches for a layer of this grid, dtype, shape and
 * batch.  Host only: no HIP call, nothing enqueued.  For testing and tuning.
 *
 *   shape    NULL for the library's own choice, or a forced {rf, wk, nw, cs}
 *            as accepted by kan_layer_forward_packed (validated here the same
 *            way: an invalid one is KAN_ERR_INVALID_ARG)
 *   plan[0]  32-row MFMA tiles per wave (1 or 2), or 0 for the vector-ALU
 *            kernel of narrow layers (below)
 *   plan[1]  waves splitting the contraction (K) of a workgroup (1, 2 or 4)
 *   plan[2]  waves per workgroup (4 or 8)
 *   plan[3]  workgroups splitting the columns of an output tile (1, 2 or 4)
 *   plan[4]  1 if the layer runs on the structured-sparse matrix instruction
 *            (bf16, k = 3, 5 <= G <= 12), else 0
 *   plan[5]  workgroups splitting the contraction (K) of each output tile when
 *            the caller gives kan_layer_forward_packed its workspace (1: no
 *            split).  Only batches that give fewer than 512 workgroups split,
 *            only layers with a long contraction, and into at most as many
 *            splits as keep the fp32 partial sums within 16 MiB; the shape
 *            {2, 1, 8, 1} and the narrow-layer kernel never split.
 *
 * Degrees other than 3 run one shape, {1, 1, 4, 1}.
 *
 * Narrow layers: fp32, k = 3, 1 <= out_features <= 16 and G <= 58 can also
 * run the shape {0, 4, 4, 1}, a kernel without matrix instructions (one batch
 * row per lane, 64 rows per workgroup, four waves each taking a quarter of
 * the features, only the k + 1 nonzero basis values and the SiLU value of
 * each input multiplied into the outputs; the same eq. kan_forward up to the
 * fp32 summation order).  It is planned for batches of 16384 rows or more
 * and never splits (plan[5] = 1).
 *
 * Writes plan[0..5].  Returns KAN_OK, KAN_ERR_INVALID_ARG (plan == NULL, bad
 * grid or sizes, batch < 1, an invalid forced shape) or KAN_ERR_UNSUPPORTED.
 */
kan_status kan_layer_plan(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                          int32_t in_features, int32_t out_features, const int32_t* shape,
                          int32_t* plan);

/*
 * kan_layer_backward -- gradients of one KAN layer (eq. kan_forward) for an
 * upstream gradient dy = dL/dy:
 *
 *   dx[b, i]       = sum_o dy[b, o] ( sum_j coef[o, i, j] N_j'(x[b, i])
 *                                     + base_w[o, i] silu'(x[b, i]) )
 *   dcoef[o, i, j] = sum_b dy[b, o] N_j(x[b, i])
 *   dbase_w[o, i]  = sum_b dy[b, o] silu(x[b, i])
 *
 * N_j' is the derivative in x of the clamped truncated-power basis
 * (eq. general_truncated differentiated: (1/h) (1/2) sum_m (-1)^m C(4, m)
 * (u - m)_+^2 at the clamped coordinate of eq. bounded, 0 off the support).
 * Cubic splines only (spline_order 3; else KAN_ERR_UNSUPPORTED).
 * The paper reports forward timing only and lists backward timing as future
 * work (Sec. 5); these are the chain rule applied to its forward.
 *
 *   x        [batch, in_features]              dtype storage
 *   coef     [out_features, in_features, G+3]  dtype storage (read only for dx)
 *   base_w   [out_features, in_features]       dtype storage (read only for dx)
 *   dy       [batch, out_features]             dtype storage
 *   dx       [batch, in_features]              output, or NULL to skip it
 *   dcoef    [out_features, in_features, G+3]  output, or NULL to skip the
 *   dbase_w  [out_features, in_features]         weight gradients (both NULL
 *                                                or both non-NULL)
 *   workspace  caller-owned device scratch of workspace_bytes >=
 *              kan_layer_backward_workspace_bytes(...), 16-byte aligned,
 *              overlapping no other argument; overwritten.
 *
 * Both contractions run on the matrix cores with fp32 accumulation; the
 * basis values are regenerated in registers, never stored.  For layers of at
 * most 16 outputs from 16384 rows on (when a feature's G + 7 columns, rounded
 * down to even, times its outputs rounded up to a multiple of 4 stay within
 * 256) dx runs instead on the vector ALUs over the SiLU column and the four
 * basis columns whose support holds x (the others' derivatives are exactly 0),
 * one batch row per lane, with a copy of the weights in the workspace (fp32,
 * or in bf16 the weights as given, summed by two-term bf16 dot products with
 * fp32 accumulation): the same sums up to the fp32 summation order.  The weight
 * gradients sum the batch in a fixed order (deterministic).  Outputs are
 * fully overwritten; with batch == 0 the weight gradients are written as 0.
 * Outputs must not overlap each other, any input or the workspace.
 *
 * Returns KAN_OK, KAN_ERR_INVALID_ARG (as kan_layer_forward, plus a NULL dy,
 * no output requested, only one of dcoef / dbase_w, a short or misaligned
 * workspace), KAN_ERR_UNSUPPORTED or KAN_ERR_DEVICE.
 */
kan_status kan_layer_backward(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                              int32_t in_features, int32_t out_features, const void* x,
                              const void* coef, const void* base_w, const void* dy, void* dx,
                              void* dcoef, void* dbase_w, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * kan_layer_backward_workspace_bytes -- size in bytes of the workspace
 * kan_layer_backward needs for this grid, dtype, batch and shape (the packed
 * weights of the dx contraction, dy transposed, and the fp32 partial weight
 * gradients of the batch splits).  Writes *bytes.  Returns KAN_OK,
 * KAN_ERR_INVALID_ARG (bytes == NULL, bad grid or sizes, batch < 0) or
 * KAN_ERR_UNSUPPORTED.
 */
kan_status kan_layer_backward_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                              int64_t batch, int32_t in_features,
                                              int32_t out_features, size_t* bytes);

/*
 * kan_layer_forward_span -- the layer of kan_layer_forward (eq. kan_forward)
 * restricted to its nonzero terms: of each input's G + k basis values only
 * the k + 1 whose support holds the input can be nonzero (the clamp of
 * eq. bounded makes every other one exactly 0), so each (row, feature) adds
 * k + 1 coefficient rows and the SiLU weight row, on the vector ALUs, instead
 * of the G + k + 1 columns of the dense contraction.  Each basis value is
 * still the closed clamped form (no recursion); the result equals
 * kan_layer_forward's up to the fp32 summation order.  For large grids,
 * where the dense contraction multiplies mostly zeros (G = 200: 4 of 203).
 * This goes beyond the paper, whose method evaluates every basis.
 *
 *   x, coef, base_w, y   as kan_layer_forward
 *   workspace            caller-owned, workspace_bytes >=
 *                        kan_layer_forward_span_workspace_bytes(...), 16-byte
 *                        aligned, overlapping no other argument (the weights
 *                        transposed to fp32 [in][G + k + 1][out tile], and
 *                        fp32 partial sums when the features are split over
 *                        workgroups, added in a fixed order).
 *
 * Returns as kan_layer_forward, plus KAN_ERR_UNSUPPORTED for grids too wide
 * for one feature's weight tile in LDS (G + k + 1 > 512).
 */
kan_status kan_layer_forward_span(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                  int32_t in_features, int32_t out_features, const void* x,
                                  const void* coef, const void* base_w, void* workspace,
                                  size_t workspace_bytes, void* y, void* stream);

/* Size in bytes of kan_layer_forward_span's workspace for this layer and batch. */
kan_status kan_layer_forward_span_workspace_bytes(const kan_grid* grid, kan_dtype dtype,
                                                  int64_t batch, int32_t in_features,
                                                  int32_t out_features, size_t* bytes);

/*
 * kan_layer_forward_noalloc -- kan_layer_forward without a workspace argument,
 * for callers that cannot allocate device memory (work under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  The
 * packed weights go to a fixed scratch array of KAN_NOALLOC_SCRATCH_BYTES
 * bytes that the library holds in device memory on every GPU it runs on,
 * until the process ends, followed (from the next 256-byte boundary) by the
 * partial sums of a split contraction when they fit there (else the layer
 * runs unsplit); nothing is allocated or freed by the call.
 *
 *   x, coef, base_w, y   as kan_layer_forward (caller-owned device memory)
 *
 * Every call on one GPU uses that GPU's one scratch array: calls that overlap
 * in time on one GPU (on different streams, or from different host threads
 * without ordering between their streams) race on it and may return wrong
 * results.  Calls ordered on one stream are safe.  The scratch is fully
 * rewritten by each call before it is read, so nothing carries over from an
 * earlier call.  The first call on a device looks up that device's scratch
 * address (hipGetSymbolAddress) and caches it, for the device current at the
 * call.
 *
 * Returns as kan_layer_forward, plus KAN_ERR_SCRATCH_LIMIT when the layer's
 * packed weights (kan_layer_packed_bytes) exceed KAN_NOALLOC_SCRATCH_BYTES;
 * that check runs on the host before any HIP call.
 */
kan_status kan_layer_forward_noalloc(const kan_grid* grid, kan_dtype dtype, int64_t batch,
                                     int32_t in_features, int32_t out_features,
                                     const void* x, const void* coef, const void* base_w,
                                     void* y, void* stream);

/* Size of the per-device scratch array of kan_layer_forward_noalloc: 16 MiB,
 * enough for the packed weights of a 784 -> 256 layer with G = 10 in fp32
 * (11.2 MB) or of a 128 -> 128 layer with G = 200 in fp32 (13.4 MB). */
#define KAN_NOALLOC_SCRATCH_BYTES (16u << 20)

/* Static, NUL-terminated description of a status code (never NULL). */
const char* kan_status_string(kan_status status);

/* Version of this interface; bumped on any incompatible change. */
int32_t kan_abi_version(void);

#define KAN_ABI_VERSION 4

#ifdef __cplusplus
}
#endif

#endif /* KAN_H */
