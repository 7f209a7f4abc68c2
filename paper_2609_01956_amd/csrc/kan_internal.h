// kan_internal.h -- host-side launch interface between the C ABI layer and the
// kernel translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kan_device.h"

namespace kan {

// ---------------------------------------------------------------- basis only

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
// The same basis by the Cox-de Boor recursion over every knot interval.
hipError_t launch_basis_cdb_f32(const float* x, int64_t n, float* phi, const GridConst& g,
                                hipStream_t s);
hipError_t launch_basis_cdb_bf16(const uint16_t* x, int64_t n, uint16_t* phi, const GridConst& g,
                                 hipStream_t s);

// ---------------------------------------------------------------- fused layer
//
// The contraction runs over K = in * (nb + 1) columns: for every input feature
// its nb basis values and its SiLU value.  Features are taken in pairs, one
// per half of a wave (the two k halves of the MFMA operands), and each pair's
// nb + 1 columns are cut into "blocks" of kj columns (8 for bf16, one
// v_mfma_f32_32x32x16_bf16 k-step; 2 for fp32, two v_mfma_f32_32x32x2_f32
// k-steps), the last block of a pair zero-padded.  The packed weight buffer
// holds, per N tile of 32 * nf output columns, the blocks in order:
//
//   packed[tile][pair][block][h][n][kj]      (h = feature within the pair)
//
// i.e. 2 * (32 * nf) * kj elements per block, kj consecutive per (h, n), so a
// wave reads one block's B operand for 32 columns with one conflict-free 16-
// or 8-byte LDS load per lane, and a workgroup stages consecutive blocks with
// plain contiguous copies.
// Weights move global -> registers -> LDS in chunks of whole blocks: a chunk
// is up to 16 KB (at most 8 blocks) and a multiple of 4 KB (one 16-byte load
// per thread of a 256-thread workgroup).
__host__ __device__ constexpr int layer_block_bytes(bool bf16, int nf) {
    return 2 * 32 * nf * (bf16 ? 8 * 2 : 2 * 4);  // [h][n][kj] elements
}
__host__ __device__ constexpr int layer_chunk_blocks(bool bf16, int nf) {
    return 16384 / layer_block_bytes(bf16, nf) < 8 ? 16384 / layer_block_bytes(bf16, nf) : 8;
}

struct LayerGeom {
    int nb;       // G + k
    int kdeg;     // spline degree k
    int kj;       // columns per block (8 bf16, 2 fp32)
    int nsb;      // blocks per feature pair, ceil((nb + 1) / kj)
    int npairs;   // ceil(in / 2)
    int nblk;     // blocks per N tile holding data, npairs * nsb
    int nblk_pad; // blocks per N tile in the packed buffer (whole chunks; the
                  // padding blocks are zero)
    int kb;       // blocks per chunk
    int nf;       // 32-column MFMA fragments per N tile (1, 2, 4 or 8)
    int ntiles;   // ceil(out / (32 * nf))
    int out;      // output features
    // bf16 with two blocks per feature (5 <= G <= 12): packed for the
    // structured-sparse MFMA (block = feature of the pair, half = column
    // half, element e of half w = column 4 (e % 4) + 2 w + e / 4), and only
    // the shapes without a K split run on it (layer_cfg_valid).
    bool sparse;
    size_t packed_bytes;
};

// Returns false when the sizes do not fit the index types of the kernels.
bool layer_geom(int nb, int kdeg, bool bf16, int in, int out, LayerGeom* g);

// Workgroup shape of the fused kernel: nw waves, each holding rf 32-row MFMA
// tiles of nf / cs 32-column fragments; wk waves split the blocks (K) of a
// chunk and are summed through LDS at the end, the other nw / wk waves take
// different rows; cs workgroups split the columns of an N tile (each stages
// only its columns of every packed block).
// On the sparse layout eight waves of two row tiles (rf = 2, nw = 8) pair up:
// the two waves of a 64-row group take the two column halves of the tile and
// pass each other the A of one row tile each.
// rf = 0 (wk = nw = 4, cs = 1) is instead the vector-ALU kernel of narrow
// fp32 layers (kan_narrow.hip): one batch row per lane, 64 rows per
// workgroup, the four waves splitting the features.
struct LayerCfg {
    int rf;  // 1 or 2 (0: the narrow-layer kernel)
    int wk;  // 1, 2 or 4
    int nw;  // waves per workgroup: 4, or 8 (wk = 1, cs = 1; rf = 2 sparse only)
    int cs;  // column slices per N tile: 1, 2 or 4 (rf = 1, nw = 4 only)
};
// Most rows any workgroup shape covers (x is addressed per workgroup with
// 32-bit byte offsets, so kLayerMaxRows * in * 4 must stay below 2^32).
constexpr int kLayerMaxRows = 256;
// Rows per workgroup and most outputs of the narrow-layer kernel.
constexpr int kNarrowRows = 64;
constexpr int kNarrowMaxOut = 16;
// Rows per workgroup of a shape.
inline int64_t layer_cfg_rows(const LayerCfg& c) {
    if (c.rf == 0) return kNarrowRows;
    return 32LL * c.rf * (c.nw / c.wk) / (c.rf == 2 && c.nw == 8 ? 2 : 1);
}

// The shapes the fused kernel is instantiated for, given the packed tile of
// nfl fragments: the chunk the slice stages must be whole 16-byte loads of
// every thread, its blocks must split evenly over the wk waves, and wk > 1
// keeps rf * (nfl / cs) <= 4 (the partial sums fit in LDS).
__host__ __device__ constexpr bool layer_shape_ok(bool bf16, int nfl, int rf, int wk, int nw,
                                                 int cs) {
    if ((rf != 1 && rf != 2) || (wk != 1 && wk != 2 && wk != 4) || (nw != 4 && nw != 8) ||
        (cs != 1 && cs != 2 && cs != 4) || nfl % cs != 0 || (!bf16 && nfl > 4))
        return false;
    const int nf = nfl / cs;
    const int kb = layer_chunk_blocks(bf16, nfl);
    const int chb = kb * layer_block_bytes(bf16, nf);
    if (chb % (1024 * nw) != 0 || kb % wk != 0) return false;
    // (eight waves of two row tiles: the sparse shared-A shape, bf16 256-column
    // tiles only; eight waves splitting K: sparse tiles of one or two
    // fragments only)
    if (nw == 8)
        return cs == 1 && ((wk == 1 && (rf == 1 || (bf16 && nfl == 8))) ||
                           (wk > 1 && rf == 1 && bf16 && nfl <= 2));
    if (cs > 1) return rf == 1;
    return wk == 1 || rf * nf <= 4;
}

// bf16 x can be read as the aligned 32-bit words holding its elements: x is
// 4-byte aligned and batch * in is even, so no word reaches past the tensor.
inline bool layer_x_words(const void* x, int64_t batch, int in) {
    return reinterpret_cast<uintptr_t>(x) % 4 == 0 && (batch * (int64_t)in) % 2 == 0;
}
LayerCfg plan_layer(const LayerGeom& g, bool bf16, int64_t batch);
// Whether a shape (planned or forced by the caller) is instantiated and valid
// for the geometry.
bool layer_cfg_valid(const LayerGeom& g, const LayerCfg& c);

struct LayerArgs {
    const void* x;    // [batch, in]
    const void* wp;   // packed weights
    void* y;          // [batch, out]
    int64_t batch;
    int in;
    int out;
    int nb;
    int nsb;
    int npairs;       // ceil(in / 2)
    int nblk;         // blocks holding data
    int nblk_pad;     // blocks per N tile in the packed buffer
    int nchunks;      // nblk_pad / blocks-per-chunk
    int cps;          // chunks per K split (workgroup z takes chunks [z cps, (z + 1) cps))
    float* P;         // K splits > 1: fp32 partial sums [split][batch][out] (else null)
    float inv_h;      // see GridConst
    float inv_lo;
    float xlim;
    float a_int;
    float a_frac;
    int kdeg;         // spline degree (3: the cubic kernels; else the run-time degree form)
    float hw;
    float hc[4];
};

// Device address and size of the calling thread's current device's copy of
// the fixed scratch array used by kan_layer_forward_noalloc (looked up once
// per device, then cached).
hipError_t noalloc_scratch(void** ptr, size_t* bytes);

hipError_t launch_pack(bool bf16, const LayerGeom& g, int in, int out, const void* coef,
                       const void* base_w, void* packed, hipStream_t s);
// K splits across workgroups for a shape and batch: small batches give too
// few workgroups to fill the chip, so each of ks workgroups per output tile
// takes a range of the K chunks and writes fp32 partial sums, which a second
// kernel adds in a fixed order (1: no split).
int layer_k_splits(const LayerGeom& g, const LayerCfg& c, int64_t batch, int out);
// Bytes of those partial sums (0 for one split).
size_t layer_partial_bytes(const LayerGeom& g, const LayerCfg& c, int64_t batch, int out);
// The fused forward; ks > 1 needs `partial` of layer_partial_bytes bytes
// (16-byte aligned), else it may be null.
hipError_t launch_layer(bool bf16, const LayerGeom& g, const LayerCfg& c, LayerArgs a, int ks,
                        void* partial, hipStream_t s);
// Per-dtype kernel launches (one translation unit each).
hipError_t launch_layer_bf16(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a,
                             hipStream_t s);
hipError_t launch_layer_f32(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a,
                            hipStream_t s);
// The narrow-layer kernel: fp32, k = 3, 1 <= out <= kNarrowMaxOut, G <= 58.
bool narrow_ok(const LayerGeom& g);
hipError_t launch_narrow(const LayerGeom& g, const LayerArgs& a, hipStream_t s);

// ------------------------------------------------------------- backward
//
// Gradients of the layer for an upstream gradient dy [batch, out]:
//   dx[b, i]  = sum_o dy[b, o] (sum_j C[o, i, j] N_j'(x[b, i]) + Wb[o, i] silu'(x[b, i]))
//   dC[o,i,j] = sum_b dy[b, o] N_j(x[b, i]),   dWb[o, i] = sum_b dy[b, o] silu(x[b, i])
// Both contractions run over "K rows": feature f owns rows [f cp, (f+1) cp),
// row f cp + c holding column c of the feature (0: SiLU, 1..nb: basis c - 1,
// beyond: zero padding).  cp is 16 when a feature's nb + 1 columns fit in 16,
// else a multiple of 32; rows are cut into tiles of 32 (two features each
// when cp = 16, part of one feature otherwise).
struct BwdGeom {
    int nb;         // G + 3
    int cp;         // K rows per feature
    int ntiles;     // 32-row K tiles
    int kr;         // 32 ntiles
    int out32;      // out rounded up to 32 (rows of the transposed dy)
    int groups;     // dx: k-step groups over all outputs (16 outputs bf16, 8 fp32)
    int gmax;       // dx: groups per output chunk held in registers (256 outputs)
    int nchunk;     // dx: output chunks (partial dx summed by a reduce when > 1)
    int dx_rf;      // dx: 32-row batch tiles per wave
    int dx_bm;      // dx: batch rows per workgroup
    int dx_ksplit;  // dx: workgroups splitting the K tiles of a row block
    int dx_tiles_per_split;  // dx: K tiles per such workgroup (whole features)
    bool nx;        // dx on the vector-ALU kernel of narrow layers (else the MFMA kernel)
    int ncw, nrs;   // nx: columns per feature and floats per column of its weight table
    int nfeat;      // nx: features of the table (in rounded up to 8)
    int oh, nfw;    // dW: waves across outputs, 32-output fragments per wave
    int kt;         // dW: K rows per workgroup (256)
    int ktiles;     // dW: K tiles of kt rows
    int otiles;     // dW: output tiles of 32 oh nfw columns
    int split;      // dW: batch splits (partials summed by the reduce kernel)
    int rows_per_split;  // multiple of 32
    int64_t bpad;   // batch rounded up to 32 (columns of the transposed dy)
    size_t off_wt, off_dyt, off_xt, off_p, off_dxp, bytes;  // workspace layout
};

// Returns false when the sizes do not fit the kernels' index types.
bool bwd_geom(int nb, bool bf16, int64_t batch, int in, int out, BwdGeom* g);

struct BwdArgs {
    const void* x;     // [batch, in]
    const void* coef;  // [out, in, nb]
    const void* bw;    // [out, in]
    const void* dy;    // [batch, out]
    void* dx;          // [batch, in] or null
    void* dcoef;       // [out, in, nb] or null (then dbw is null too)
    void* dbw;         // [out, in]
    void* ws;          // workspace of BwdGeom::bytes
    int64_t batch;
    int in;
    int out;
    float inv_h, inv_lo, xlim, a_int, a_frac;
};

hipError_t launch_backward(bool bf16, const BwdGeom& g, const BwdArgs& a, hipStream_t s);

// ------------------------------------------------------------ span-sparse
//
// The layer forward restricted to the k + 1 bases whose support holds each
// input (and the SiLU term), on the vector ALUs with one feature's weights
// staged in LDS at a time (kan_span.hip).
struct SpanGeom {
    int opt, ng, nr; // outputs per thread, output groups per workgroup, rows per thread
    int otiles;      // output tiles of opt * ng columns
    int outp;        // out padded to whole tiles (columns of the transposed weights)
    int fs, fpf;     // feature splits (partials summed when > 1), features per split
    int cs;          // LDS stride of one weight column in floats (tile width, padded)
    int64_t rblocks; // row blocks of 256 nr / ng rows
    size_t off_w, off_p, bytes;  // workspace: transposed fp32 weights, partial sums
};
bool span_geom(int nb, int64_t batch, int in, int out, SpanGeom* g);

struct SpanArgs {
    const void* x;    // [batch, in]
    const float* wt;  // transposed weights [in][nb + 1][outp] (set by the launcher)
    void* y;          // [batch, out]
    void* ws;         // workspace of SpanGeom::bytes
    size_t off_p;
    int64_t batch;
    int in, out, nb, outp, fs, fpf, cs;
    float inv_h, inv_lo, xlim, a_int, a_frac;
    int kdeg;
    float hw;
    float hc[4];
};
hipError_t launch_span(bool bf16, const SpanGeom& g, const SpanArgs& a, const void* coef,
                       const void* bw, hipStream_t s);

}  // namespace kan
