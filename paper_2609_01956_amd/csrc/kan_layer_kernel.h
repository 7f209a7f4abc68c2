// kan_layer_kernel.h -- fused KAN-layer forward on MFMA (eq. kan_forward):
//
//   y[b, o] = sum_i sum_{j <= nb} A[b, (i, j)] * W[o, (i, j)]
//   A[b, (i, j)] = N_j(x[b, i]) for j < nb,   silu(x[b, i]) for j = nb
//   W[o, (i, j)] = coef[o, i, j]   for j < nb,   base_w[o, i]  for j = nb
//
// a dense [batch, in * (nb + 1)] x [in * (nb + 1), out] contraction whose
// left operand is never stored: every lane generates its own A elements in
// registers, directly in the MFMA operand layout, from one x value per block.
//
// layer_kernel: 4 or 8 waves per workgroup.  The workgroup walks the blocks
// of packed weights (kan_internal.h) in chunks of up to 16 KB: each chunk is
// loaded into registers two chunks ahead, written to one of two LDS stages
// while the previous chunk is multiplied, and read from LDS by every wave.
// Each wave owns rf 32-row tiles of nf 32-column fragments, so every
// generated A element feeds nf MFMAs and every B fragment read from LDS feeds
// rf MFMAs.  With two waves per SIMD a wave generates the next block's A and
// then issues the current block's MFMAs, so one wave's VALU work overlaps the
// other's matrix work; with one wave per SIMD the two interleave within the
// wave.
//
// Basis values are N_j / 2 = P^3 - Q^3 (half_basis, kan_device.h).  The MFMA
// operands are N_j / 2 and silu / 2, and the epilogue doubles y: scaling by a
// power of two is exact, so the operands are exactly bf16(N_j) / 2 and
// bf16(silu) / 2 on the bf16 path and the result is the contraction of the
// rounded N_j and silu values.
//
// fp32: A and W fp32, v_mfma_f32_32x32x2_f32 (one k per lane half, two
//       k-steps per block).
// bf16: x, W bf16 in memory; A generated in fp32, rounded to bf16 (RNE);
//       v_mfma_f32_32x32x16_bf16 (eight k per lane half), fp32 accumulation;
//       y rounded to bf16 on store.
//
// Included by kan_layer.hip (weight packing, planning) and by one
// translation unit per dtype that instantiates the fused kernels
// (kan_layer_bf16.hip, kan_layer_f32.hip), so they compile in parallel.
#pragma once

#include "kan_internal.h"

#include <type_traits>

namespace kan {
namespace layer_detail {

constexpr int kThreads = 256;
// silu(x) / 2 = x / (2 + 2 exp(-x)).
__device__ __forceinline__ float half_silu(float x) {
    return x * __builtin_amdgcn_rcpf(__builtin_fmaf(__expf(-x), 2.0f, 2.0f));
}

// Two floats to bf16 (round to nearest even), packed low then high.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}
// bf16(v) (RNE) in the low half, 0 in the high half: one conversion (written
// through pack_bf16x2(v, 0) the compiler converts with an arbitrary high
// operand and then clears the high half with a second instruction).
__device__ __forceinline__ uint32_t bf16_lo(float v) {
    uint32_t r;
    asm("v_cvt_pk_bf16_f32 %0, %1, 0" : "=v"(r) : "v"(v));
    return r;
}

template <typename T> struct Tr;

template <> struct Tr<float> {
    static constexpr int KJ = 2;  // columns per block
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ uint32_t raw(const float* p) {
        return __float_as_uint(*p);
    }
    static __device__ __forceinline__ float value(uint32_t u) { return __uint_as_float(u); }
    static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};

template <> struct Tr<uint16_t> {
    static constexpr int KJ = 8;
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ uint32_t raw(const uint16_t* p) { return *p; }
    static __device__ __forceinline__ float value(uint32_t u) { return __uint_as_float(u << 16); }
    static __device__ __forceinline__ void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// ---------------------------------------------------------- A generation
//
// Within a feature the columns are ordered [silu, N_0, N_1, ..., N_{nb-1}]
// and zero-padded to a whole number of blocks, so column c of the feature is
// basis c - 1 for c >= 1.  Block b, element e is column KJ * b + e: a basis
// value at v = s_b - e with s_b = v of basis KJ * b - 1, except column 0 (the
// SiLU value).  fp32 (and bf16 with one wave per SIMD) generates every block
// with the same straight-line code: columns past nb are evaluated like any
// other basis (finite values that meet zero weights) and element 0 of block 0
// is replaced.  bf16 with two waves per SIMD picks the code by the block's
// place in its pair (gen_split).
template <typename T, int RF> struct AFrag;
template <int RF> struct AFrag<uint16_t, RF> { bf16x8 a[RF]; };
template <int RF> struct AFrag<float, RF> { float a[RF][2]; };

template <int RF>
__device__ __forceinline__ void zero_frag(AFrag<uint16_t, RF>& A, int rf) {
#pragma unroll
    for (int e = 0; e < 8; ++e) A.a[rf][e] = (__bf16)0.0f;
}
template <int RF>
__device__ __forceinline__ void zero_frag(AFrag<float, RF>& A, int rf) {
    A.a[rf][0] = 0.0f;
    A.a[rf][1] = 0.0f;
}

// Position of a wave's block: global block index, feature pair and block
// within the pair.  A wave visits blocks wk, wk + WK, wk + 2 WK, ...
struct Pos {
    int blk, pair, bsub;
};

// Advance a position by STEP blocks (compile-time STEP <= 8, nsb >= 1):
// straight-line selects, so no loop (and no basic-block split) in the main
// loop.
template <int STEP>
__device__ __forceinline__ Pos advance(Pos p, int nsb) {
    p.blk += STEP;
    p.bsub += STEP;
#pragma unroll
    for (int i = 0; i < STEP; ++i) {
        // wrap = (bsub >= nsb) as plain integer arithmetic (no lane masks,
        // so the scalar unit does it)
        const int wrap = (int)((uint32_t)(nsb - 1 - p.bsub) >> 31);
        p.bsub -= nsb & -wrap;
        p.pair += wrap;
    }
    return p;
}

// Advance by a runtime step < 4.
__device__ __forceinline__ Pos advance_n(Pos p, int step, int nsb) {
    p.blk += step;
    p.bsub += step;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int wrap = (int)((uint32_t)(nsb - 1 - p.bsub) >> 31);
        p.bsub -= nsb & -wrap;
        p.pair += wrap;
    }
    return p;
}

// ------------------------------------------------------------- main kernel

// Waves per SIMD the register budget is sized for: two when the accumulators
// take at most 128 registers (so a second wave's MFMAs fill the matrix core
// while one wave runs its basis VALU work), otherwise one.
template <int RF, int NF>
struct Occ {
    static constexpr int waves = RF * NF * 16 <= 128 ? 2 : 1;
};

// NFL: 32-column fragments per N tile of the packed layout; NF: fragments of
// the tile this workgroup computes (a column slice, NFL / NF slices per tile).
// NSBC: blocks per feature when fixed at compile time (0: a.nsb at run time).
// XP (bf16): x read as the aligned 32-bit word holding the element (x 4-byte
// aligned and batch * in even, so the word never leaves the tensor).
// SP: the structured-sparse MFMA on the sparse packed layout (LayerGeom::sparse).
// XA (SP, two row tiles per wave, eight waves): the two waves of a row group
// take the two column halves of the tile, and each generates the A of one of
// the group's two row tiles and passes it to the other through LDS (half the
// LDS bytes of B per MFMA of one-row-tile waves, still two waves per SIMD).
// GD: a spline degree other than 3, evaluated with the run-time degree form
// (half_basis_deg) instead of the cubic's two-term form.
template <typename T, int RF, int NFL, int NF, int WK, int NW, int NSBC = 0, bool XP = false,
          bool SP = false, bool XA = false, bool GD = false>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(Occ<RF, XA ? NF / 2 : NF>::waves)))
void layer_kernel(LayerArgs a) {
    constexpr bool BF16 = sizeof(T) == 2;
    constexpr int KJ = Tr<T>::KJ;
    constexpr int NT = 64 * NW;                  // threads per workgroup
    constexpr int CH = XA ? 2 : 1;               // waves sharing a row group's columns
    constexpr int NFW = NF / CH;                 // 32-column fragments per wave
    constexpr int GRF = XA ? 1 : RF;             // row tiles whose A a wave generates
    constexpr int WM = NW / WK / CH;
    constexpr int CS = NFL / NF;                 // column slices per N tile
    constexpr int NTILE = 32 * NF;               // columns of the slice
    constexpr int LANEB = KJ * (int)sizeof(T);  // B bytes per lane per block (16 / 8)
    constexpr int BLKBL = layer_block_bytes(BF16, NFL);  // packed block: [h][n][KJ]
    constexpr int BLKB = layer_block_bytes(BF16, NF);    // the slice's part of it (in LDS)
    constexpr int KB = layer_chunk_blocks(BF16, NFL);    // blocks per chunk
    constexpr int CHB = KB * BLKB;               // bytes per chunk in LDS
    constexpr int DPW = CHB / (1024 * NW);       // 16-byte loads per lane per chunk
    constexpr int KBW = KB / WK;                 // blocks per wave per chunk
    constexpr int BM = 32 * RF * WM;             // rows per workgroup
    // Weights of chunk c are loaded into registers L chunks ahead (register
    // set c % L), written to LDS stage c % 2 while chunk c - 1 is multiplied,
    // and read from there during chunk c.  (Two chunks ahead measured faster
    // than three: the loop body, unrolled by lcm(2, L), stays small.)
    // PRE (the shared-A shape, one feature pair per chunk): four LDS stages
    // and four register sets; loads four chunks ahead, weights stored to LDS
    // two chunks after their loads and two chunks before their use, and the
    // B of chunk c + 1 read into registers during chunk c, so every chunk's
    // MFMAs start right after its barrier.  (784 -> 256: 298 us against 308
    // with three stages and 304-306 with five or six.  The other 256-column
    // sparse shapes hold twice the B registers and spill with it.)
    constexpr bool PRE = XA;
    constexpr int NST = PRE ? 4 : 2;             // LDS stages
    constexpr int L = PRE ? 4 : 2;
    constexpr int U = PRE ? 4 : (L % 2 == 0 ? L : 2 * L);  // chunk-loop unroll, lcm(NST, L)
    constexpr int PART = WK > 1 ? 32 * RF * NTILE * 4 : 0;  // one wave's partial sums
    constexpr int SMEM = NST * CHB > NW * PART ? NST * CHB : NW * PART;
    static_assert(CHB % (1024 * NW) == 0 && KB % WK == 0 && KB >= WK, "chunk shape");
    static_assert(NW == 4 || (NW == 8 && (WK == 1 || SP)), "waves per workgroup");
    static_assert(SMEM <= 64 * 1024, "LDS budget");
    // With a compile-time block count per feature that divides the wave's
    // blocks per chunk (and no K split), every chunk starts a feature: the
    // place of each step's block in its feature is a compile-time constant.
    constexpr bool ALIGNED = NSBC > 0 && (WK == 1 || SP) && KBW % NSBC == 0;
    // Sparse with a K split (SPK): wave slice wk takes the chunk's feature
    // pairs wk, wk + WK, ... (pairs per chunk PPC), i.e. pair
    // c PPC + wk + WK q as the wave's q-th pair of chunk c, blocks
    // 2 (wk + WK q) and 2 (wk + WK q) + 1 of the chunk.
    constexpr bool SPK = SP && WK > 1;
    constexpr int PPC = KB / 2;
    static_assert(NSBC == 0 || ALIGNED, "compile-time blocks per feature");
    const int nsb = NSBC > 0 ? NSBC : a.nsb;
    static_assert(BLKB == 2 * NTILE * LANEB && NFL % NF == 0, "block layout");
    static_assert(!XA || (SP && RF == 2 && NW == 8 && WK == 1 && NF == 8 && NFL == 8),
                  "shared-A shape");
    // LDS: two chunk stages; after the main loop the K-split partial sums.
    __shared__ u32x4 smem[SMEM / 16];
    // XA: two stages of every wave's generated A (values, positions), one
    // slot per lane
    __shared__ u32x4 xa_a[XA ? 2 * NW * 64 : 1];
    __shared__ uint32_t xa_i[XA ? 2 * NW * 64 : 1];
    // (gfx950: 160 KB of LDS per workgroup; XA takes 84 KB, one workgroup per CU)
    static_assert(SMEM + (XA ? 2 * NW * 64 * 20 : 0) <= 96 * 1024, "LDS budget");
    auto stage = [&](auto kk) -> u32x4* {
        return smem + (decltype(kk)::value % NST) * (CHB / 16);
    };

    const T* __restrict__ x = static_cast<const T*>(a.x);
    T* __restrict__ y = static_cast<T*>(a.y);
    static_assert(!GD || (!SP && !XA), "the structured-sparse operand is cubic");
    // a basis value N / 2 at v = u - (k + 1) / 2
    auto hb = [&](float v) -> float {
        if constexpr (GD) return half_basis_deg(v, a.kdeg, a.hw, a.hc);
        else return half_basis(v);
    };

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int lane = tid & 63;
    const int r = lane & 31;
    const int h = lane >> 5;
    const int wm = wave % WM;
    const int wk = XA ? 0 : wave / WM;
    // XA: the wave's column half, also the row tile whose A it generates
    // (its partner, wave wm + WM (1 - ch), generates the other)
    const int ch = XA ? wave / WM : 0;
    const int64_t row0 = (int64_t)blockIdx.x * BM + wm * 32 * RF;
    const int nt = blockIdx.y / CS;     // N tile
    const int slice = blockIdx.y % CS;  // column slice of the tile
    // K split (workgroup z): chunks [c_beg, c_beg + nch) of the tile; the
    // loop below counts chunks from c_beg (one split: the whole tile).
    const int c_beg = blockIdx.z * a.cps;
    const int nch = min(a.cps, a.nchunks - c_beg);
    // Packed weights of this N tile (nblk_pad blocks = nchunks whole chunks),
    // from the split's first chunk.
    const char* __restrict__ wpt = static_cast<const char*>(a.wp) +
                                   (size_t)nt * (size_t)a.nblk_pad * BLKBL +
                                   (size_t)c_beg * (KB * BLKBL);

    // x and the N tile's packed weights are read through buffer resources
    // with 32-bit byte offsets: x from a per-workgroup base (the host rejects
    // layers with kLayerMaxRows * in * 4 >= 2^32, and N tiles of 2^32 packed
    // bytes or more).  Each lane's offset within a pair or chunk is fixed, so
    // it is computed once here; the pair's or chunk's offset is wave-uniform
    // and goes in the scalar operand.  Rows past the batch read row batch - 1
    // (their results are not stored).
    const int64_t wg_row0 = (int64_t)blockIdx.x * BM;
    const T* __restrict__ xw = x + wg_row0 * (int64_t)a.in;
    const uint64_t x_left = (uint64_t)(a.batch - wg_row0) * (uint64_t)a.in * sizeof(T);
    const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(xw), (short)0, (int)(x_left < 0xffffffffull ? x_left : 0xffffffffull),
        kBufferWord3);
    uint32_t xoff[GRF];  // element offset of (row, feature h of pair 0)
#pragma unroll
    for (int rf = 0; rf < GRF; ++rf) {
        int64_t row = row0 + (XA ? ch : rf) * 32 + r;
        row = row < a.batch ? row : a.batch - 1;
        xoff[rf] = (uint32_t)((row - wg_row0) * a.in + h);
    }
    // With an odd feature count the last pair has a phantom second feature
    // (zero weights): its lanes read the real last feature and use x = 0.
    const int last_pair_odd = (a.in & 1) ? a.in / 2 : -1;
    // XP: byte selector that moves the lane's half of the loaded word to the
    // top of a float (the half is the parity of its element offset, the same
    // for every pair; the phantom lanes' value is replaced by 0 anyway).
    static_assert(!XP || sizeof(T) == 2, "paired x reads are for bf16");
    uint32_t xsel[GRF];
#pragma unroll
    for (int rf = 0; rf < GRF; ++rf) xsel[rf] = (xoff[rf] & 1u) ? 0x03020c0cu : 0x01000c0cu;
    // Byte offsets of the lane's x at pair 0 (XP: of the aligned word holding
    // it), and at the last pair of an odd feature count, where the phantom
    // lanes step back one feature; pair p adds 2 p elements (XP: p words).
    uint32_t xvo[GRF], xvo_odd[GRF];
#pragma unroll
    for (int rf = 0; rf < GRF; ++rf) {
        const uint32_t eb = xoff[rf] - (uint32_t)h;
        if constexpr (XP) {
            xvo[rf] = (xoff[rf] >> 1) * 4u;
            xvo_odd[rf] = (eb >> 1) * 4u;
        } else {
            xvo[rf] = xoff[rf] * (uint32_t)sizeof(T);
            xvo_odd[rf] = eb * (uint32_t)sizeof(T);
        }
    }

    // ---- loads of chunk c into register set j, for the wave's blocks from
    // position p on: first the x of each block and row tile (per lane: the
    // lane's row, the feature of its half in the block's pair; positions past
    // the end read the last pair, the phantom lanes step back one feature),
    // then the weights (wave w, load i holds bytes [i 1024 NW + w 1024,
    // + 1024) of the chunk as staged in LDS, 16 per lane).  In LDS a chunk
    // holds the slice's columns only: each block is [h][n][KJ] over the
    // slice's NTILE columns, read from the two matching runs of the packed
    // block (goff: the packed offset of each of the lane's loads).  Chunks
    // past the last re-load the last chunk.  Raw x bits are kept: conversion
    // and masking happen where the values are used, so nothing waits for a
    // load when it is issued.
    typedef uint32_t XSet[KBW][GRF];
    constexpr bool X_FIRST_ONLY = ALIGNED && BF16 && (SP || Occ<RF, NF>::waves == 2);
    typedef u32x4 WSet[DPW];
    const uint32_t wlane = (uint32_t)(wave * 1024 + lane * 16);
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(wpt), (short)0, (int)((uint32_t)nch * (uint32_t)(KB * BLKBL)),
        kBufferWord3);
    uint32_t goff[CS == 1 ? 1 : DPW];
    if constexpr (CS > 1) {
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const uint32_t o = wlane + (uint32_t)(i * 1024 * NW);  // byte in the LDS chunk
            const uint32_t blk = o / BLKB, rem = o % BLKB;
            const uint32_t half = rem / (BLKB / 2), within = rem % (BLKB / 2);
            goff[i] = blk * BLKBL + half * (BLKBL / 2) + (uint32_t)slice * (BLKB / 2) + within;
        }
    }
    auto issue = [&](int c, Pos p, XSet& xs, WSet& ws) {
#pragma unroll
        for (int t = 0; t < KBW; ++t) {
            int pr = p.pair;
            if constexpr (SPK) pr = (c_beg + c) * PPC + wk + WK * (t / 2);
            pr = pr < a.npairs ? pr : a.npairs - 1;
            const bool odd = pr == last_pair_odd;  // wave-uniform
            // The split generation reads x only at a feature's first block.
            if (!(X_FIRST_ONLY && t % NSBC != 0)) {
#pragma unroll
                for (int rf = 0; rf < GRF; ++rf) {
                    const uint32_t vo = odd ? xvo_odd[rf] : xvo[rf];
                    if constexpr (XP)
                        xs[t][rf] = __builtin_amdgcn_raw_buffer_load_b32(xrs, vo, 4 * pr, 0);
                    else if constexpr (sizeof(T) == 4)
                        xs[t][rf] = __builtin_amdgcn_raw_buffer_load_b32(
                            xrs, vo, 2 * (int)sizeof(T) * pr, 0);
                    else
                        xs[t][rf] = __builtin_amdgcn_raw_buffer_load_b16(
                            xrs, vo, 2 * (int)sizeof(T) * pr, 0);
                }
            } else {
#pragma unroll
                for (int rf = 0; rf < GRF; ++rf) xs[t][rf] = 0u;
            }
            p = advance<WK>(p, nsb);
        }
        const int cc = c < nch ? c : nch - 1;
        const int cofs = (int)((uint32_t)cc * (uint32_t)(KB * BLKBL));  // the chunk's bytes
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const uint32_t vo = CS == 1 ? wlane + (uint32_t)(i * 1024 * NW) : goff[i];
            ws[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wrs, vo, cofs, 0));
        }
    };
    // Register set -> LDS stage kk (the same byte offsets as in the chunk).
    auto store = [&](auto kk, const WSet& ws) {
        char* l = reinterpret_cast<char*>(stage(kk));
#pragma unroll
        for (int i = 0; i < DPW; ++i)
            *reinterpret_cast<u32x4*>(l + wlane + i * 1024 * NW) = ws[i];
    };
    // Value of raw x bits for the lane's feature at position p (the phantom
    // feature of an odd feature count gives 0).
    auto x_value = [&](const Pos& p, uint32_t raw, int rf) {
        float v;
        if constexpr (XP)
            v = __uint_as_float(__builtin_amdgcn_perm(raw, raw, xsel[rf]));
        else
            v = Tr<T>::value(raw);
        // (one condition: the wave-uniform pair test and the lane's half
        // combine into one lane mask, so this is a single select)
        return (p.pair == last_pair_odd && h != 0) ? 0.0f : v;
    };

    // acc[rf]: row tile rf ^ ch of the wave's row group (XA: the tile whose A
    // the wave generates first), its NFW fragments from column half ch
    floatx16 acc[RF][NFW];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf)
#pragma unroll
        for (int nf = 0; nf < NFW; ++nf)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[rf][nf][q] = 0.0f;

    // ---- B fragments of one block (LDS block `bi` of stage `st`)
    typedef typename std::conditional<BF16, bf16x8, floatx2>::type BVec;
    struct BFrag { BVec b[NFW]; };
    auto read_b = [&](BFrag& B, const u32x4* st, int bi) {
        const char* lb = reinterpret_cast<const char*>(st) + bi * BLKB;
#pragma unroll
        for (int nf = 0; nf < NFW; ++nf) {
            const char* q = lb + (h * NTILE + (ch * NFW + nf) * 32 + r) * LANEB;
            if constexpr (BF16)
                B.b[nf] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(q));
            else
                B.b[nf] = *reinterpret_cast<const floatx2*>(q);
        }
    };

    // MFMA number i of a block (NMFMA per block): bf16 (nf, rf); fp32 also
    // the k-step t of the block's two columns.
    constexpr int NMFMA = (BF16 ? 1 : 2) * RF * NFW;
    auto do_mfma = [&](int i, const AFrag<T, RF>& A, const BFrag& B) {
        const int rf = i % RF;
        const int nf = (i / RF) % NFW;
        if constexpr (BF16) {
            acc[rf][nf] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.a[rf], B.b[nf], acc[rf][nf], 0, 0, 0);
        } else {
            const int t = i / (RF * NFW);
            acc[rf][nf] = __builtin_amdgcn_mfma_f32_32x32x2f32(A.a[rf][t], B.b[nf][t],
                                                               acc[rf][nf], 0, 0, 0);
        }
    };

    // One step: the NMFMA MFMAs of the current block (A, B) together with the
    // generation of the next block's A (block pg from x values xv, slv the
    // silu of its pair) and, with one wave per SIMD, the LDS reads of the next
    // block's B (PREF: block bi_n of stage st).  After MFMA i come the VALU
    // ops of A elements [i NE / NMFMA, (i + 1) NE / NMFMA).
    constexpr int NE = RF * KJ;  // A elements generated per lane per block
    constexpr bool SCHED_PINGPONG = Occ<RF, NF>::waves == 2;
    auto step = [&](const AFrag<T, RF>& A, const BFrag& B, const Pos& pg,
                    const float (&xv)[RF], const float (&slv)[RF], AFrag<T, RF>& An,
                    auto pref_tag, BFrag& Bn, const u32x4* st, int bi_n) {
        constexpr bool PREF = decltype(pref_tag)::value;
        float s[RF];
        const float c = a.a_int + 1.0f - (float)(KJ * pg.bsub);
#pragma unroll
        for (int rf = 0; rf < RF; ++rf)
            s[rf] = __builtin_fmaf(xv[rf], a.inv_h, c) + coord_lo(xv[rf], a.xlim, a.inv_lo, a.a_frac);
        // (xv: x values of block pg, already converted)
        const bool first = pg.bsub == 0;
        float v[RF][KJ];
        auto gen_elem = [&](int k) {
            const int rf = k / KJ;
            const int e = k % KJ;
            const float bv = hb(s[rf] - (float)e);
            v[rf][e] = (e == 0 && first) ? slv[rf] : bv;
            if constexpr (BF16) {
                if (e & 1) {
                    An.a[rf][e - 1] = (__bf16)v[rf][e - 1];
                    An.a[rf][e] = (__bf16)v[rf][e];
                }
            } else {
                An.a[rf][e] = v[rf][e];
            }
        };
        if constexpr (SCHED_PINGPONG) {
            // Two waves per SIMD: the whole basis generation (VALU), then the
            // MFMAs back to back at raised priority.  While one wave runs its
            // VALU phase the other's MFMA phase keeps the matrix core busy,
            // and the priority makes the MFMA phase win when both want to
            // issue.
#pragma unroll
            for (int k = 0; k < NE; ++k) gen_elem(k);
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int i = 0; i < NMFMA; ++i) do_mfma(i, A, B);
            __builtin_amdgcn_s_setprio(0);
            __builtin_amdgcn_sched_barrier(0);
        } else {
            // One wave per SIMD: after MFMA i come the VALU ops of elements
            // [i NE / NMFMA, (i + 1) NE / NMFMA).
#pragma unroll
            for (int i = 0; i < NMFMA; ++i) {
                do_mfma(i, A, B);
                if constexpr (PREF) {
                    if (i == 0) read_b(Bn, st, bi_n);
                }
#pragma unroll
                for (int k = i * NE / NMFMA; k < (i + 1) * NE / NMFMA; ++k) gen_elem(k);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    // bf16 with two waves per SIMD: the A of a block is generated by code
    // chosen by the block's place in its feature pair (uniform branches).
    //   first block:  x, the coordinate and the SiLU value (element 0), then
    //                 basis values 1 .. 7;
    //   middle block: the coordinate steps down by 8 (one wave visits the
    //                 blocks of a pair in order when WK = 1; with WK > 1 it is
    //                 recomputed from x), then 8 basis values;
    //   last block:   as a middle block, but only the real columns of the
    //                 feature (rounded up to even) are evaluated and the
    //                 padding columns are set to 0.
    // Stepping the coordinate by 8 is exact wherever a basis value of the
    // block is nonzero (there |s| < 17 and s - 8 is computed exactly).
    constexpr bool GEN_SPLIT = BF16 && Occ<RF, NF>::waves == 2;
    constexpr bool DIRECT = WK > 1;
    float sc[RF];  // coordinate of the wave's current block (element 0)
    // real columns in the last block of a feature, rounded up to even
    const int last_cols = a.nb + 1 - KJ * (nsb - 1);
    const int last_even = (last_cols + 1) & ~1;
    auto gen_split = [&](const Pos& pg, const uint32_t (&xr)[RF], AFrag<T, RF>& An) {
      if constexpr (GEN_SPLIT) {
        auto basis = [&](int rf, int e0, int e1) {
#pragma unroll
            for (int e = e0; e < e1; ++e) An.a[rf][e] = (__bf16)hb(sc[rf] - (float)e);
        };
        auto zero = [&](int rf, int e0) {
#pragma unroll
            for (int e = e0; e < KJ; ++e) An.a[rf][e] = (__bf16)0.0f;
        };
        if (pg.bsub == 0) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) {
                const float xv = x_value(pg, xr[rf], rf);
                sc[rf] = __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f) +
                         coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
                // keep the coordinate itself for the feature's later blocks
                // (recomputing it there from x would hold the raw x register,
                // and a copy of it could wait on a load still in flight)
                asm volatile("" : "+v"(sc[rf]));
                An.a[rf][0] = (__bf16)half_silu(xv);
                basis(rf, 1, KJ);
            }
            return;
        }
        if constexpr (DIRECT) {
            const float c = a.a_int + 1.0f - (float)(KJ * pg.bsub);
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) {
                const float xv = x_value(pg, xr[rf], rf);
                sc[rf] = __builtin_fmaf(xv, a.inv_h, c) + coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
            }
        } else {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) sc[rf] -= (float)KJ;
        }
        if (pg.bsub != nsb - 1 || last_even == KJ) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) basis(rf, 0, KJ);
        } else if (last_even == 6) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) { basis(rf, 0, 6); zero(rf, 6); }
        } else if (last_even == 4) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) { basis(rf, 0, 4); zero(rf, 4); }
        } else {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) { basis(rf, 0, 2); zero(rf, 2); }
        }
      }
    };
    // Step with split generation: the next block's A, then the MFMAs of the
    // current block (while one wave generates, the other's MFMAs keep the
    // matrix core busy; the compiler is left to schedule within the step,
    // which measured as fast as a fixed phase order with raised MFMA
    // priority, and faster for the 256 -> 256 layer).
    // SP: the A of a whole feature pair for one v_smfmac_f32_32x32x32_bf16
    // per 32-column fragment.  Its 32 K slots are four groups of four per
    // feature; a lane holds its row's feature (the feature of its half), two
    // values per group, each at the position its 2-bit index gives (values at
    // one position add up).  Group G holds the columns c = G (mod 4), at
    // position c / 4.  Every nonzero basis column lies in the four columns
    // c0 .. c0 + 3 with c0 = floor(s) - 1 (R20); clamped to [1, 12], the
    // window stays inside columns 1 .. 15 and the columns it then takes in
    // are at |v| >= 2, where the form is exactly 0.  Its columns fall one per
    // group: value 2G is the basis at column c0 + ((G - c0) mod 4), at
    // position c0 / 4, plus 1 for G < c0 mod 4; value 1 is the SiLU value at
    // column 0 (group 0, position 0); values 3, 5, 7 are zero.
    static_assert(!SP || (BF16 && NSBC == 2 && KBW % 2 == 0 && (WK == 1 || (!XA && RF == 1))),
                  "sparse MFMA shape");
    auto gen_sparse = [&](const float (&xf)[GRF], AFrag<T, RF>& As, uint32_t (&idx)[RF]) {
      if constexpr (SP) {
#pragma unroll
        for (int rf = 0; rf < GRF; ++rf) {
            const float sv = __builtin_fmaf(xf[rf], a.inv_h, a.a_int + 1.0f) +
                             coord_lo(xf[rf], a.xlim, a.inv_lo, a.a_frac);
            // c0 + 1 = floor(s) within [2, 13] (a NaN coordinate gives c0 = 1
            // and NaN values, as it should)
            const float f1 = __builtin_amdgcn_fmed3f(__builtin_floorf(sv), 2.0f, 13.0f);
            const int c0 = (int)f1 - 1;
            const int r = c0 & 3;
            const float d = sv - (f1 - 1.0f);  // v of column c0
            // (G - c0) mod 4 is byte G of 0x03020100 rotated left by 8 c0
            // bits, i.e. right by 24 c0 (mod 32), which is 0x00030201 rotated
            // right by 24 (c0 + 1) = 24 f1 (exact in fp32; an integer
            // multiply here compiles to the quarter-rate v_mul_lo_u32)
            const uint32_t kg = __builtin_amdgcn_alignbit(0x00030201u, 0x00030201u,
                                                          (uint32_t)(24.0f * f1));
            float bv[4];
#pragma unroll
            for (int G = 0; G < 4; ++G) bv[G] = half_basis(d - (float)((kg >> (8 * G)) & 0xffu));
            idx[rf] = __umul24((uint32_t)(c0 >> 2), 0x1111u) + (0x1111u & ((1u << (4 * r)) - 1u));
            const u32x4 w = {pack_bf16x2(bv[0], half_silu(xf[rf])), bf16_lo(bv[1]),
                             bf16_lo(bv[2]), bf16_lo(bv[3])};
            As.a[rf] = __builtin_bit_cast(bf16x8, w);
        }
      }
    };
    auto step_split = [&](const AFrag<T, RF>& A, const BFrag& B, const Pos& pg,
                          const uint32_t (&xr)[RF], AFrag<T, RF>& An) {
        gen_split(pg, xr, An);
#pragma unroll
        for (int i = 0; i < NMFMA; ++i) do_mfma(i, A, B);
        // The next block's A must be complete here: otherwise code sinking
        // moves its generation past the next barrier, next to the MFMAs that
        // read it, and neither step overlaps generation with multiplication.
        if constexpr (BF16) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) {
                u32x4 w = __builtin_bit_cast(u32x4, An.a[rf]);
                asm volatile("" : "+v"(w));
                An.a[rf] = __builtin_bit_cast(bf16x8, w);
            }
        }
    };

    auto silu_of = [&](const float (&xv)[RF], float (&sl)[RF]) {
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) sl[rf] = half_silu(xv[rf]);
    };

    // ---- pipeline
    // Chunk c: at its top a barrier (every wave has written chunk c to stage
    // c % 2 and finished reading chunk c - 1 from the other stage), then the
    // loads of chunk c + L are issued into register set c % L (free: its
    // weights went to LDS during chunk c - 1, its x were copied out), the
    // weights of chunk c + 1 (set (c + 1) % L) are written to stage
    // (c + 1) % 2, and the chunk's blocks are multiplied.  The chunk loop is
    // unrolled by U so that stages and register sets are compile-time
    // choices (a register move of a load still in flight would wait for
    // it).  Chunks past the last one (to fill the unrolled group) load
    // clamped inputs and multiply zero A.
    // PRE: stage c % 4 holds chunk c, written during chunk c - 2 and read
    // into registers during chunk c - 1; chunk c issues the loads of chunk
    // c + 4 into set c % 4, writes the weights of chunk c + 2 (set
    // (c + 2) % 4, loaded two chunks earlier) to stage (c + 2) % 4 (last
    // read during chunk c - 3), multiplies chunk c and then reads the B of
    // chunk c + 1 from stage (c + 1) % 4 (written during chunk c - 1).  XA's
    // A exchange alternates between its two stages by the parity of c.
    static_assert(WK <= 4, "wave block stride");
    constexpr int WAIT_LDS = 0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14);  // lgkmcnt(0) only
    // XA (PRE): lgkmcnt(2 NFW), every LDS operation but the chunk's last 2 NFW
    // (the B reads of the next chunk, issued after all of the chunk's LDS
    // writes; LDS operations complete in order and the loop has no scalar
    // memory loads, which would also count)
    constexpr int WAIT_XA = 0xF | (0x7 << 4) | ((2 * NFW) << 8) | (0x3 << 14);
    static_assert(!PRE || 2 * NFW <= 15, "lgkmcnt field");
    // real blocks of the split, and of this wave; SP: the end of the split's
    // feature pairs (a chunk holds KB / 2 of them)
    const int nblk_s = min(a.nblk - c_beg * KB, nch * KB);
    const int pair_end = min(a.npairs, (c_beg + nch) * (KB / 2));
    const int nq = wk < nblk_s ? (nblk_s - wk + WK - 1) / WK : 0;

    XSet xq[L];
    WSet wq[L];
    float sl[RF];
    AFrag<T, RF> A_cur, A_nxt;
    uint32_t idx_cur[RF], idx_nxt[RF];  // SP: positions of the compressed A values
    // XA: the wave's generated A (tile 0 of A) to stage stg of its slot; the
    // partner's from stage stg to tile 1
    auto xa_put = [&](int stg, const AFrag<T, RF>& A, const uint32_t (&idx)[RF]) {
      if constexpr (XA) {
        const int o = stg * NW * 64 + wave * 64 + lane;
        xa_a[o] = __builtin_bit_cast(u32x4, A.a[0]);
        xa_i[o] = idx[0];
      }
    };
    auto xa_get = [&](int stg, AFrag<T, RF>& A, uint32_t (&idx)[RF]) {
      if constexpr (XA) {
        const int o = stg * NW * 64 + (wm + WM * (1 - ch)) * 64 + lane;
        A.a[1] = __builtin_bit_cast(bf16x8, xa_a[o]);
        idx[1] = xa_i[o];
      }
    };
    BFrag bq[2];
    // first block of the current chunk (SPK: the first block of pair wk)
    Pos pos_c;
    {
        const int b0 = c_beg * KB;  // the split's first block (a whole pair when SPK)
        pos_c = SPK ? Pos{b0 + 2 * wk, b0 / 2 + wk, 0}
                    : advance_n(Pos{b0, b0 / nsb, b0 % nsb}, wk, nsb);
    }
    Pos pos_l = pos_c;                               // first block of the next chunk to load

    // prologue: loads of chunks 0 .. L - 1, chunk 0 to stage 0
    auto prologue = [&](auto jj) {
        constexpr int j = decltype(jj)::value;
        issue(j, pos_l, xq[j], wq[j]);
        pos_l = advance<KB>(pos_l, nsb);
    };
    StaticFor<0, L>::run(prologue);
    store(std::integral_constant<int, 0>{}, wq[0]);
    if constexpr (PRE) store(std::integral_constant<int, 1>{}, wq[1]);
    // A of the wave's first block (nothing to interleave with yet); XA
    // generates it before the barrier, to pass it on.
    auto gen_first_sparse = [&]() {
        float x0[GRF];
#pragma unroll
        for (int rf = 0; rf < GRF; ++rf) x0[rf] = x_value(pos_c, xq[0][0][rf], rf);
        gen_sparse(x0, A_cur, idx_cur);
    };
    if constexpr (XA) {
        gen_first_sparse();
        xa_put(0, A_cur, idx_cur);
    }
    __builtin_amdgcn_s_waitcnt(WAIT_LDS);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);

    if constexpr (SP) {
        if constexpr (PRE) {
            read_b(bq[0], stage(std::integral_constant<int, 0>{}), 0);
            read_b(bq[1], stage(std::integral_constant<int, 0>{}), 1);
        }
        if constexpr (!XA) gen_first_sparse();
    } else if constexpr (GEN_SPLIT) {
        if constexpr (!DIRECT) {
            // A K split across workgroups can start inside a feature: seed the
            // carried coordinate with that of the block before the first (the
            // generation subtracts KJ from it).  Wave-uniform branch.
            if (pos_c.bsub != 0) {
                const float c = a.a_int + 1.0f - (float)(KJ * (pos_c.bsub - 1));
#pragma unroll
                for (int rf = 0; rf < RF; ++rf) {
                    const float xv = x_value(pos_c, xq[0][0][rf], rf);
                    sc[rf] = __builtin_fmaf(xv, a.inv_h, c) +
                             coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
                }
            }
        }
        gen_split(pos_c, xq[0][0], A_cur);
    } else {
        float x0[RF];
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) x0[rf] = x_value(pos_c, xq[0][0][rf], rf);
        silu_of(x0, sl);
        const float c0 = a.a_int + 1.0f - (float)(KJ * pos_c.bsub);
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) {
            const float s0 = __builtin_fmaf(x0[rf], a.inv_h, c0) +
                             coord_lo(x0[rf], a.xlim, a.inv_lo, a.a_frac);
#pragma unroll
            for (int e = 0; e < KJ; ++e) {
                const float bv = hb(s0 - (float)e);
                const float v = (e == 0 && pos_c.bsub == 0) ? sl[rf] : bv;
                if constexpr (BF16) A_cur.a[rf][e] = (__bf16)v;
                else A_cur.a[rf][e] = v;
            }
        }
    }

    // Chunk c with K = c % U (compile-time).
    auto chunk = [&](int c, auto kk, auto last_tag) {
        constexpr int K = decltype(kk)::value;
        constexpr bool LASTG = decltype(last_tag)::value;  // in the final group
        constexpr int J = K % L;          // register set of chunk c (and of c + L)
        constexpr int JN = (K + 1) % L;   // register set of chunk c + 1
        if constexpr (ALIGNED) {
            pos_c.bsub = 0;
            pos_l.bsub = 0;
        }
        if (c > 0) {  // (chunk 0's barrier is in the prologue)
            __builtin_amdgcn_s_waitcnt(PRE ? WAIT_XA : WAIT_LDS);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
        }
        // x of the blocks whose A this chunk generates: blocks 1 .. KBW - 1
        // of this chunk, then block 0 of the next one
        uint32_t xr[KBW][GRF];
#pragma unroll
        for (int t = 0; t < KBW; ++t)
#pragma unroll
            for (int rf = 0; rf < GRF; ++rf)
                xr[t][rf] = t + 1 < KBW ? xq[J][t + 1][rf] : xq[JN][0][rf];
        __builtin_amdgcn_sched_barrier(0);
        issue(c + L, pos_l, xq[J], wq[J]);
        pos_l = advance<KB>(pos_l, nsb);
        __builtin_amdgcn_sched_barrier(0);
        // The next chunk's weights go to the other LDS stage before the next
        // barrier.  With the split generation they are stored after the
        // first step, which gives their loads that step's time to land.
        if constexpr (!GEN_SPLIT && !SP) {
            store(std::integral_constant<int, K + 1>{}, wq[JN]);
            __builtin_amdgcn_sched_barrier(0);
        }

        const u32x4* st = stage(kk);
        if constexpr (!PRE) read_b(bq[0], st, SP ? 2 * wk : wk);
        if constexpr (SP) {
            // the chunk's feature pairs, one step each: the B of the pair's two
            // blocks (XA: and the partner's A), at the first pair the next
            // chunk's weights to the other LDS stage, the next pair's A (its x
            // was loaded a chunk or more ago), the MFMAs of this pair
            constexpr int NPC = KBW / 2;  // pairs per chunk of this wave
            auto pair_step = [&](auto qq) {
                constexpr int q = decltype(qq)::value;
                if constexpr (!PRE) {
                    // (blocks of the wave's q-th pair of the chunk)
                    if constexpr (q > 0) read_b(bq[0], st, 2 * (wk + WK * q));
                    read_b(bq[1], st, 2 * (wk + WK * q) + 1);
                }
                xa_get(c & 1, A_cur, idx_cur);  // (XA: one pair per chunk)
                if constexpr (q == 0) {
                    // the next chunk's weights to the other LDS stage, before
                    // this pair's generation and MFMAs (their loads were
                    // issued a chunk ago; stored after the MFMAs instead, the
                    // writes and their wait end the chunk, just before its
                    // barrier)
                    __builtin_amdgcn_sched_barrier(0);
                    if constexpr (PRE)
                        store(std::integral_constant<int, K + 2>{}, wq[(K + 2) % L]);
                    else
                        store(std::integral_constant<int, K + 1>{}, wq[JN]);
                    __builtin_amdgcn_sched_barrier(0);
                }
                Pos pn = pos_c;  // the wave's next pair
                pn.pair += WK * (q + 1);
                // (x of the next pair's first block, copied before this
                // chunk's loads reused its register set)
                float xf[GRF];
#pragma unroll
                for (int rf = 0; rf < GRF; ++rf) xf[rf] = x_value(pn, xr[2 * q + 1][rf], rf);
                if constexpr (LASTG) {
                    // a pair past the split's range (padding of the layer,
                    // or the next split's) contributes 0
                    if (pos_c.pair + WK * q >= pair_end) {
#pragma unroll
                        for (int rf = 0; rf < RF; ++rf) zero_frag(A_cur, rf);
                    }
                }
                gen_sparse(xf, A_nxt, idx_nxt);
                auto smfmac = [&](int rf, int nf) {
                    const bf16x16 b = __builtin_shufflevector(bq[0].b[nf], bq[1].b[nf], 0, 1, 2, 3,
                                                              4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14,
                                                              15);
                    acc[rf][nf] = __builtin_amdgcn_smfmac_f32_32x32x32_bf16(
                        A_cur.a[rf], b, acc[rf][nf], (int)idx_cur[rf], 0, 0);
                };
                if constexpr (XA) {
                    // the wave's own tile first: the partner's A comes from LDS
#pragma unroll
                    for (int rf = 0; rf < RF; ++rf)
#pragma unroll
                        for (int nf = 0; nf < NFW; ++nf) smfmac(rf, nf);
                } else {
#pragma unroll
                    for (int nf = 0; nf < NFW; ++nf)
#pragma unroll
                        for (int rf = 0; rf < RF; ++rf) smfmac(rf, nf);
                }
                // (the next A complete here, so code sinking cannot move its
                // generation past the next barrier)
#pragma unroll
                for (int rf = 0; rf < GRF; ++rf) {
                    u32x4 w = __builtin_bit_cast(u32x4, A_nxt.a[rf]);
                    asm volatile("" : "+v"(w), "+v"(idx_nxt[rf]));
                    A_nxt.a[rf] = __builtin_bit_cast(bf16x8, w);
                }
                if constexpr (XA) {
                    xa_put((c + 1) & 1, A_nxt, idx_nxt);
                    __builtin_amdgcn_sched_barrier(0);
                }
                if constexpr (PRE) {
                    // the next chunk's B (stored during the previous chunk),
                    // the chunk's last LDS operations: the barrier waits only
                    // for the LDS writes before them (WAIT_XA)
                    read_b(bq[0], stage(std::integral_constant<int, K + 1>{}), 0);
                    read_b(bq[1], stage(std::integral_constant<int, K + 1>{}), 1);
                }
                if constexpr (XA) {
                    A_cur.a[0] = A_nxt.a[0];
                    idx_cur[0] = idx_nxt[0];
                } else {
                    A_cur = A_nxt;
#pragma unroll
                    for (int rf = 0; rf < RF; ++rf) idx_cur[rf] = idx_nxt[rf];
                }
            };
            StaticFor<0, NPC>::run(pair_step);
            pos_c = advance<KB>(pos_c, nsb);
        } else {
            Pos p = pos_c;
            auto one = [&](auto tt) {
                constexpr int t = decltype(tt)::value;
                // position of the next block: the next step's, or the first block
                // of the next chunk
                const Pos pnext = advance<WK>(p, nsb);
                float xv[RF];
                if constexpr (!GEN_SPLIT) {
#pragma unroll
                    for (int rf = 0; rf < RF; ++rf) xv[rf] = x_value(pnext, xr[t][rf], rf);
                    if (pnext.bsub == 0) silu_of(xv, sl);
                }
                if constexpr (LASTG) {
                    if (c * KBW + t >= nq) {  // past the wave's last real block: contribute 0
#pragma unroll
                        for (int rf = 0; rf < RF; ++rf) zero_frag(A_cur, rf);
                    }
                }
                // One wave per SIMD: the next block's B is read during this step.
                // Two waves: B is read at the start of each step; the other wave
                // covers the latency, and the registers of a second B set are
                // saved.
                constexpr bool PREF = Occ<RF, NF>::waves == 1 && t + 1 < KBW;
                if constexpr (Occ<RF, NF>::waves == 2 && t > 0) read_b(bq[t & 1], st, wk + WK * t);
                if constexpr (GEN_SPLIT)
                    step_split(A_cur, bq[t & 1], pnext, xr[t], A_nxt);
                else
                    step(A_cur, bq[t & 1], pnext, xv, sl, A_nxt,
                         std::integral_constant<bool, PREF>{}, bq[(t + 1) & 1], st,
                         wk + WK * (t + 1));
                A_cur = A_nxt;
                p = pnext;
                if constexpr (GEN_SPLIT && t == 0) {
                    __builtin_amdgcn_sched_barrier(0);
                    store(std::integral_constant<int, K + 1>{}, wq[JN]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            StaticFor<0, KBW>::run(one);
            pos_c = p;
        }
    };

    // Every wave's blocks are all real in every group but the final one.
    const int ngroups = (nch + U - 1) / U;
#pragma unroll 1
    for (int gi = 0; gi + 1 < ngroups; ++gi) {
        auto group = [&](auto kk) {
            chunk(gi * U + decltype(kk)::value, kk, std::false_type{});
        };
        StaticFor<0, U>::run(group);
    }
    {
        const int gi = ngroups - 1;
        auto group = [&](auto kk) {
            chunk(gi * U + decltype(kk)::value, kk, std::true_type{});
        };
        StaticFor<0, U>::run(group);
    }
    __syncthreads();

    // ---- epilogue: y = 2 acc (the operands carry N / 2 and silu / 2)
    const int col0 = nt * (32 * NFL) + slice * NTILE;
    // The shared-A shape (bf16, 256-column tiles; never K-split) stores y
    // through LDS (the weight stages are free now): in two rounds, each wave
    // writes one of its row tiles there as bf16, so a round holds 128 rows x
    // 256 columns of the workgroup's tile (64 KB), and every thread then
    // stores 16-byte row segments (element stores where out % 8 != 0 or y is
    // not 16-byte aligned).  The accumulator layout alone gives 2-byte
    // stores of 32 columns (784 -> 256 at batch 65536: 8.9 us of stores, about 5
    // at the HBM write rate).
    if constexpr (XA) {
        static_assert(BF16 && NST * CHB >= 128 * 256 * 2, "staged epilogue");
        const bool vec = (a.out & 7) == 0 && (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
        uint16_t* st = reinterpret_cast<uint16_t*>(smem);  // [128][256]
        const int64_t wg_row0 = (int64_t)blockIdx.x * BM;
        // round R: every wave writes its row tile R (workgroup rows 64 wm +
        // 32 (R ^ ch) + (0 .. 31), columns 128 ch + (0 .. 127)) at LDS rows
        // 32 wm + (0 .. 31); the column half thus tells a unit's row tile.
        // (acc is indexed by compile-time constants only: a tile chosen by
        // ch at run time would move acc out of registers.)
        auto out_round = [&](auto rr) __attribute__((always_inline)) {
            constexpr int R = decltype(rr)::value;
#pragma unroll
            for (int nf = 0; nf < NFW; ++nf)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int rl = wm * 32 + 8 * (q / 4) + 4 * h + (q % 4);
                    const int cl = (ch * NFW + nf) * 32 + r;
                    st[rl * 256 + cl] = f32_to_bf16(2.0f * acc[R][nf][q]);
                }
            __syncthreads();
#pragma unroll
            for (int m = 0; m < 128 * 32 / NT; ++m) {
                const int u = tid + NT * m;  // 16-byte unit: 32 per LDS row
                const int rl = u >> 5;
                const int cu = (u & 31) * 8;
                const int col = col0 + cu;
                const int k = cu < 128 ? R : 1 - R;  // the row tile of this column half
                const int64_t row = wg_row0 + (rl >> 5) * 64 + k * 32 + (rl & 31);
                if (row >= a.batch || col >= a.out) continue;
                const uint16_t* src = st + rl * 256 + cu;
                if (vec) {
                    *reinterpret_cast<u32x4*>(y + row * a.out + col) =
                        *reinterpret_cast<const u32x4*>(src);
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (col + e < a.out) y[row * a.out + col + e] = src[e];
                }
            }
            __syncthreads();
        };
        StaticFor<0, 2>::run(out_round);
    } else if constexpr (WK == 1) {
        const bool full = row0 + 32 * RF <= a.batch && col0 + NTILE <= a.out;
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) {
#pragma unroll
            for (int nf = 0; nf < NFW; ++nf) {
                const int col = col0 + (ch * NFW + nf) * 32 + r;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int64_t row = row0 + (rf ^ ch) * 32 + 8 * (q / 4) + 4 * h + (q % 4);
                    if (full || (row < a.batch && col < a.out)) {
                        if (a.P != nullptr)
                            a.P[((int64_t)blockIdx.z * a.batch + row) * a.out + col] =
                                2.0f * acc[rf][nf][q];
                        else
                            Tr<T>::store(y + row * a.out + col, 2.0f * acc[rf][nf][q]);
                    }
                }
            }
        }
    } else {
        // Waves with the same wm hold partial sums of the same rows: write all
        // partials to LDS (the weight buffers are free after the last
        // barrier), then every thread sums WK partials of some elements and
        // stores them row-major (coalesced).
        constexpr int TILE = 32 * RF * NTILE;  // floats per wave
        auto red = [&](int w) -> float* { return reinterpret_cast<float*>(smem) + w * TILE; };
        float* mine = red(wave);
#pragma unroll
        for (int rf = 0; rf < RF; ++rf)
#pragma unroll
            for (int nf = 0; nf < NFW; ++nf)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int rl = rf * 32 + 8 * (q / 4) + 4 * h + (q % 4);
                    mine[rl * NTILE + nf * 32 + r] = acc[rf][nf][q];
                }
        __syncthreads();
        const int64_t bm0 = (int64_t)blockIdx.x * BM;
        for (int idx = tid; idx < WM * TILE; idx += NT) {
            const int g = idx / TILE;
            const int rem = idx % TILE;
            const int rl = rem / NTILE;
            const int cl = rem % NTILE;
            float sum = 0.0f;
#pragma unroll
            for (int w = 0; w < WK; ++w) sum += red(g + WM * w)[rem];
            const int64_t row = bm0 + g * 32 * RF + rl;
            const int col = col0 + cl;
            if (row < a.batch && col < a.out) {
                if (a.P != nullptr)
                    a.P[((int64_t)blockIdx.z * a.batch + row) * a.out + col] = 2.0f * sum;
                else
                    Tr<T>::store(y + row * a.out + col, 2.0f * sum);
            }
        }
    }
}

template <typename T, int RF, int NFL, int NF, int WK, int NW>
hipError_t launch_cfg(const LayerGeom& g, LayerArgs a, hipStream_t s) {
    // Eight waves of two row tiles: the sparse shared-A shape (layer_shape_ok)
    constexpr bool XA = RF == 2 && NW == 8;
    constexpr int BM = 32 * RF * (NW / WK) / (XA ? 2 : 1);
    static_assert(BM <= kLayerMaxRows, "rows per workgroup (32-bit x byte offsets)");
    a.nblk_pad = g.nblk_pad;
    a.nchunks = g.nblk_pad / g.kb;
    const unsigned ks = (unsigned)((a.nchunks + a.cps - 1) / a.cps);
    const dim3 grid((unsigned)((a.batch + BM - 1) / BM), (unsigned)(g.ntiles * (NFL / NF)), ks);
    // The sparse packed layout (bf16, two blocks per feature, 5 <= G <= 12)
    // runs only on the structured-sparse MFMA: no K split, whole feature
    // pairs per chunk (every block's place in its feature is a compile-time
    // constant), x read as aligned 32-bit words where that stays inside the
    // tensor.
    constexpr bool BF16 = sizeof(T) == 2;
    if (g.sparse) {
        // (K splits: narrow tiles, whole feature pairs per wave slice)
        constexpr int KBL = layer_chunk_blocks(BF16, NFL);
        if constexpr (BF16 && KBL % 2 == 0 &&
                      ((WK == 1 && (RF == 1 ? (NW == 8 || NF < 8)
                                            : (NF == NFL && (NW == 4 || NF == 8)))) ||
                       (WK > 1 && RF == 1 && NF == NFL && NFL <= 2 && (KBL / 2) % WK == 0))) {
            if (layer_x_words(a.x, a.batch, a.in))
                hipLaunchKernelGGL((layer_kernel<T, RF, NFL, NF, WK, NW, 2, true, true, XA>),
                                   grid, dim3(64 * NW), 0, s, a);
            else
                hipLaunchKernelGGL((layer_kernel<T, RF, NFL, NF, WK, NW, 2, false, true, XA>),
                                   grid, dim3(64 * NW), 0, s, a);
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;
        }
    }
    if constexpr (XA || (NW == 8 && WK > 1)) {  // (sparse-only shapes)
        return hipErrorInvalidValue;
    } else {
        if (g.kdeg != 3) {
            // other degrees: one shape, the run-time degree form
            if constexpr (RF == 1 && WK == 1 && NW == 4 && NF == NFL) {
                hipLaunchKernelGGL(
                    (layer_kernel<T, RF, NFL, NF, WK, NW, 0, false, false, false, true>), grid,
                    dim3(64 * NW), 0, s, a);
                return hipGetLastError();
            } else {
                return hipErrorInvalidValue;
            }
        }
        hipLaunchKernelGGL((layer_kernel<T, RF, NFL, NF, WK, NW>), grid, dim3(64 * NW), 0, s, a);
        return hipGetLastError();
    }
}

// Launches the configuration c if it is this (RF, WK, NW, CS) and the shape
// is instantiated (layer_shape_ok); *hit tells whether it was.
template <typename T, int NFL, int RF, int WK, int NW, int CS>
hipError_t try_cfg(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s,
                   bool* hit) {
    if constexpr (layer_shape_ok(sizeof(T) == 2, NFL, RF, WK, NW, CS)) {
        if (c.rf == RF && c.wk == WK && c.nw == NW && c.cs == CS) {
            *hit = true;
            return launch_cfg<T, RF, NFL, NFL / CS, WK, NW>(g, a, s);
        }
    }
    return hipSuccess;
}

template <typename T, int NFL, int RF, int WK, int NW>
hipError_t try_cs(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s,
                  bool* hit) {
    hipError_t e = try_cfg<T, NFL, RF, WK, NW, 1>(g, c, a, s, hit);
    if (!*hit) e = try_cfg<T, NFL, RF, WK, NW, 2>(g, c, a, s, hit);
    if (!*hit) e = try_cfg<T, NFL, RF, WK, NW, 4>(g, c, a, s, hit);
    return e;
}

template <typename T, int NFL, int RF, int WK>
hipError_t try_nw(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s,
                  bool* hit) {
    hipError_t e = try_cs<T, NFL, RF, WK, 4>(g, c, a, s, hit);
    if (!*hit) e = try_cs<T, NFL, RF, WK, 8>(g, c, a, s, hit);
    return e;
}

template <typename T, int NFL, int RF>
hipError_t try_wk(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s,
                  bool* hit) {
    hipError_t e = try_nw<T, NFL, RF, 1>(g, c, a, s, hit);
    if (!*hit) e = try_nw<T, NFL, RF, 2>(g, c, a, s, hit);
    if (!*hit) e = try_nw<T, NFL, RF, 4>(g, c, a, s, hit);
    return e;
}

template <typename T, int NFL>
hipError_t launch_nfl(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s) {
    bool hit = false;
    hipError_t e = try_wk<T, NFL, 1>(g, c, a, s, &hit);
    if (!hit) e = try_wk<T, NFL, 2>(g, c, a, s, &hit);
    return hit ? e : hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_t(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s) {
    switch (g.nf) {
        case 1: return launch_nfl<T, 1>(g, c, a, s);
        case 2: return launch_nfl<T, 2>(g, c, a, s);
        case 4: return launch_nfl<T, 4>(g, c, a, s);
        case 8:
            if constexpr (sizeof(T) == 2) return launch_nfl<T, 8>(g, c, a, s);
            return hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

}  // namespace layer_detail
}  // namespace kan
