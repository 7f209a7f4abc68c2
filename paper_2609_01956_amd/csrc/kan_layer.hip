// kan_layer.hip -- fused KAN-layer forward on MFMA (eq. kan_forward):
//
//   y[b, o] = sum_i sum_{j <= nb} A[b, (i, j)] * W[o, (i, j)]
//   A[b, (i, j)] = N_j(x[b, i]) for j < nb,   silu(x[b, i]) for j = nb
//   W[o, (i, j)] = coef[o, i, j]   for j < nb,   base_w[o, i]  for j = nb
//
// a dense [batch, in * (nb + 1)] x [in * (nb + 1), out] contraction whose
// left operand is never stored: every lane generates its own A elements in
// registers, directly in the MFMA operand layout, from one x value per block.
//
// Two kernels:
//   pack_kernel    rearranges coef / base_w into the block order described in
//                  kan_internal.h (a few MB, read once per call);
//   layer_kernel   4 waves per workgroup.  The workgroup walks the blocks in
//                  chunks of 32 KB of packed weights, double-buffered in LDS
//                  (global loads of chunk c + 1 are in flight while chunk c is
//                  multiplied).  Each wave owns rf 32-row tiles of all nf
//                  32-column fragments of the N tile, so every generated A
//                  element feeds nf MFMAs and every B fragment read from LDS
//                  feeds rf MFMAs.  A is generated one block ahead of the MFMAs
//                  that consume it, so VALU work and matrix work interleave.
//
// Basis values.  With v = u - 2 (u the coordinate of eq. truncated), the clamp
// of eq. bounded and the symmetry of the stencil {1, -4, 6, -4, 1} give
//     6 N = w^3 - 4 b^3,   w = 2 - min(|v|, 2),  b = max(1 - |v|, 0),
// and with P = w / 2 = clamp01(1 - |v| / 2) and Q = (2/3)^(1/3) b =
// clamp01((2/3)^(1/3) (1 - |v|)):
//     N = (4/3) P^3 - Q^3.
// Each value is then one subtraction, two clamped fused multiply-adds (the
// clamp and |v| fold into the instruction), four multiplies and one fused
// multiply-add.  Off the support both P and Q are 0 and the value is exactly
// 0.  The MFMA operands are exactly N_j and silu (rounded to bf16 on the bf16
// path), so the result is the contraction of those rounded operands.
//
// fp32: A and W fp32, v_mfma_f32_32x32x2_f32 (one k per lane half, two
//       k-steps per block).
// bf16: x, W bf16 in memory; A generated in fp32, rounded to bf16 (RNE);
//       v_mfma_f32_32x32x16_bf16 (eight k per lane half), fp32 accumulation;
//       y rounded to bf16 on store.
#include "kan_internal.h"

#include <cstdio>
#include <cstdlib>
#include <type_traits>

namespace kan {

namespace {

constexpr int kThreads = 256;
constexpr float kCbrtTwoThirds = 0.87358046473629571f;  // (2/3)^(1/3)

// N(u) at v = u - 2 (see the header comment).
__device__ __forceinline__ float basis(float v) {
    const float av = __builtin_fabsf(v);
    const float P = __builtin_amdgcn_fmed3f(__builtin_fmaf(av, -0.5f, 1.0f), 0.0f, 1.0f);
    const float Q = __builtin_amdgcn_fmed3f(
        __builtin_fmaf(av, -kCbrtTwoThirds, kCbrtTwoThirds), 0.0f, 1.0f);
    return __builtin_fmaf(P * P, P * (4.0f / 3.0f), -(Q * Q * Q));
}

// silu(x) = x / (1 + exp(-x)).
__device__ __forceinline__ float silu_fast(float x) {
    return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}

template <typename T> struct Tr;

template <> struct Tr<float> {
    static constexpr int KJ = 2;  // columns per block
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};

template <> struct Tr<uint16_t> {
    static constexpr int KJ = 8;
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// --------------------------------------------------------------- pack kernel

// One unit of the packed buffer per thread: the kj weights of columns
// [kj * blk, kj * blk + kj) of feature 2 * pair + h for output column n, the
// columns of a feature ordered [base_w, coef[.., 0], ..., coef[.., nb - 1]]
// and zero-padded.
template <typename T>
__global__ __launch_bounds__(kThreads) void pack_kernel(const T* __restrict__ coef,
                                                        const T* __restrict__ bw,
                                                        T* __restrict__ packed, int in, int out,
                                                        int nb, int nsb, int npairs, int ntile,
                                                        int64_t units) {
    constexpr int KJ = Tr<T>::KJ;
    const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (u >= units) return;
    int64_t rest = u;
    const int n = (int)(rest % ntile); rest /= ntile;
    const int h = (int)(rest % 2); rest /= 2;
    const int blk = (int)(rest % nsb); rest /= nsb;
    const int pair = (int)(rest % npairs);
    const int tile = (int)(rest / npairs);
    const int ng = tile * ntile + n;
    const int f = 2 * pair + h;
    T v[KJ];
#pragma unroll
    for (int e = 0; e < KJ; ++e) v[e] = T(0);
    if (ng < out && f < in) {
        const int64_t row = (int64_t)ng * in + f;
#pragma unroll
        for (int e = 0; e < KJ; ++e) {
            const int c = blk * KJ + e;  // column within the feature: [silu, N_0..N_{nb-1}]
            if (c == 0) v[e] = bw[row];
            else if (c <= nb) v[e] = coef[row * nb + c - 1];
        }
    }
    T* dst = packed + u * KJ;
#pragma unroll
    for (int e = 0; e < KJ; ++e) dst[e] = v[e];
}

// ---------------------------------------------------------- A generation
//
// Within a feature the columns are ordered [silu, N_0, N_1, ..., N_{nb-1}]
// and zero-padded to a whole number of blocks, so column c of the feature is
// basis c - 1 for c >= 1.  Block b, element e is column KJ * b + e: a basis
// value at v = s_b - e with s_b = v of basis KJ * b - 1, except column 0 (the
// SiLU value).  Columns past nb are evaluated like any other basis (finite
// values) and meet zero weights.  Every block is therefore generated by the
// same straight-line code; only element 0 of block 0 is replaced.
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

template <int RF>
__device__ __forceinline__ void gen(const float (&s)[RF], const float (&sl)[RF], bool first,
                                    AFrag<uint16_t, RF>& A) {
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        const float v0 = basis(s[rf]);
        A.a[rf][0] = (__bf16)(first ? sl[rf] : v0);
#pragma unroll
        for (int e = 1; e < 8; ++e) A.a[rf][e] = (__bf16)basis(s[rf] - (float)e);
    }
}

template <int RF>
__device__ __forceinline__ void gen(const float (&s)[RF], const float (&sl)[RF], bool first,
                                    AFrag<float, RF>& A) {
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        const float v0 = basis(s[rf]);
        A.a[rf][0] = first ? sl[rf] : v0;
        A.a[rf][1] = basis(s[rf] - 1.0f);
    }
}

// Position of a wave's block: global block index, feature pair and block
// within the pair.  A wave visits blocks wk, wk + WK, wk + 2 WK, ...
struct Pos {
    int blk, pair, bsub;
};

// Straight-line for step <= 4 (no loop, so no basic-block split in the main
// loop); nsb >= 1.
__device__ __forceinline__ Pos advance(Pos p, int step, int nsb) {
    p.blk += step;
    p.bsub += step;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const bool wrap = p.bsub >= nsb;
        p.bsub = wrap ? p.bsub - nsb : p.bsub;
        p.pair = wrap ? p.pair + 1 : p.pair;
    }
    return p;
}

// ------------------------------------------------------------- main kernel

template <typename T, int RF, int NF, int WK>
__global__ __launch_bounds__(kThreads) void layer_kernel(LayerArgs a) {
    constexpr bool BF16 = sizeof(T) == 2;
    constexpr int KJ = Tr<T>::KJ;
    constexpr int WM = 4 / WK;
    constexpr int NTILE = 32 * NF;
    constexpr int LANEB = KJ * (int)sizeof(T);  // B bytes per lane per block (16 / 8)
    constexpr int BLKB = 2 * NTILE * LANEB;      // bytes per block: [h][n][KJ]
    constexpr int KB = (32768 / BLKB) < 8 ? (32768 / BLKB) : 8;  // blocks per chunk
    constexpr int CHB = KB * BLKB;               // bytes per chunk (<= 32 KB)
    constexpr int CHU = CHB / 16;                // 16-byte units per chunk
    constexpr int SPT = CHU / kThreads;          // staged units per thread
    constexpr int KBW = KB / WK;                 // blocks per wave per chunk
    constexpr int BM = 32 * RF * WM;             // rows per workgroup
    constexpr int RED = WK > 1 ? 4 * 32 * RF * NTILE * 4 : 0;  // K-split reduction bytes
    constexpr int LDSB = 2 * CHB > RED ? 2 * CHB : RED;
    static_assert(CHU % kThreads == 0 && KB % WK == 0 && KB >= WK, "chunk shape");
    static_assert(LDSB <= 65536, "LDS budget");
    __shared__ u32x4 lds[LDSB / 16];

    const T* __restrict__ x = static_cast<const T*>(a.x);
    T* __restrict__ y = static_cast<T*>(a.y);

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int lane = tid & 63;
    const int r = lane & 31;
    const int h = lane >> 5;
    const int wm = wave % WM;
    const int wk = wave / WM;
    const int64_t row0 = (int64_t)blockIdx.x * BM + wm * 32 * RF;
    const int nt = blockIdx.y;
    const u32x4* __restrict__ wp =
        static_cast<const u32x4*>(a.wp) + (size_t)nt * (size_t)a.nblk * (BLKB / 16);
    const int64_t last_unit = (int64_t)a.nblk * (BLKB / 16) - 1;

    // Rows past the batch read row batch - 1 (their results are not stored).
    const T* xr[RF];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        int64_t row = row0 + rf * 32 + r;
        row = row < a.batch ? row : a.batch - 1;
        xr[rf] = x + row * (int64_t)a.in;
    }

    // ---- staging of packed weights (global -> registers -> LDS).  Units past
    // the end re-read the last unit; they land in LDS blocks nobody reads.
    u32x4 stg[SPT];
    auto stage_load = [&](int c) {
        const int64_t base = (int64_t)c * CHU + tid;
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            int64_t u = base + i * kThreads;
            u = u < last_unit ? u : last_unit;
            stg[i] = wp[u];
        }
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < SPT; ++i) lds[buf * CHU + tid + i * kThreads] = stg[i];
    };

    // x of this lane's rows for the feature of its half in pair p.pair; the
    // phantom feature of an odd feature count (and positions past the end)
    // give 0.
    auto load_x = [&](const Pos& p, float (&xv)[RF]) {
        const int f = 2 * p.pair + h;
        const int fc = f < a.in ? f : a.in - 1;
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) {
            const float v = Tr<T>::load(xr[rf] + fc);
            xv[rf] = f < a.in ? v : 0.0f;
        }
    };

    floatx16 acc[RF][NF];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf)
#pragma unroll
        for (int nf = 0; nf < NF; ++nf)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[rf][nf][q] = 0.0f;

    // ---- the MFMAs of one block, B read from LDS block `bi` of buffer `buf`
    auto mfma_block = [&](const AFrag<T, RF>& A, int buf, int bi) {
        const char* lb = reinterpret_cast<const char*>(lds) + buf * CHB + bi * BLKB;
        if constexpr (BF16) {
            bf16x8 b[NF];
#pragma unroll
            for (int nf = 0; nf < NF; ++nf)
                b[nf] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4*>(lb + (h * NTILE + nf * 32 + r) * 16));
#pragma unroll
            for (int nf = 0; nf < NF; ++nf)
#pragma unroll
                for (int rf = 0; rf < RF; ++rf)
                    acc[rf][nf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.a[rf], b[nf],
                                                                         acc[rf][nf], 0, 0, 0);
        } else {
            floatx2 b[NF];
#pragma unroll
            for (int nf = 0; nf < NF; ++nf)
                b[nf] = *reinterpret_cast<const floatx2*>(lb + (h * NTILE + nf * 32 + r) * 8);
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int nf = 0; nf < NF; ++nf)
#pragma unroll
                    for (int rf = 0; rf < RF; ++rf)
                        acc[rf][nf] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            A.a[rf][t], b[nf][t], acc[rf][nf], 0, 0, 0);
        }
    };

    // A of block p from x values xv; sl holds silu of the same x, computed
    // when the pair starts.
    auto gen_block = [&](const Pos& p, const float (&xv)[RF], const float (&sl)[RF],
                         AFrag<T, RF>& A) {
        const float c = a.a_int + 1.0f - (float)(KJ * p.bsub);
        float s[RF];
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) s[rf] = __builtin_fmaf(xv[rf], a.inv_h, c) + a.a_frac;
        gen<RF>(s, sl, p.bsub == 0, A);
    };
    auto silu_of = [&](const float (&xv)[RF], float (&sl)[RF]) {
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) sl[rf] = silu_fast(xv[rf]);
    };

    // ---- pipeline
    // Chunk c (KB blocks, CHB bytes of packed weights) is multiplied from LDS
    // buffer c & 1.  At the start of chunk c the wave issues the x loads of
    // chunk c + 1 and then the weight loads of chunk c + 1; the weights go to
    // LDS at the end of chunk c.  Loads complete in issue order, so waiting for
    // x never waits for weights still in flight.  Within a chunk (unrolled),
    // each step generates A of the next block (VALU) and multiplies the
    // current block (MFMA) in one basic block.
    static_assert(WK <= 4, "advance() steps at most 4");
    const int nq = wk < a.nblk ? (a.nblk - wk + WK - 1) / WK : 0;  // blocks of this wave
    float xc[KBW][RF], xn[KBW][RF], sl[RF];
    AFrag<T, RF> A_cur, A_nxt;

    // x of the KBW blocks of chunk c for this wave, starting at position p.
    auto load_chunk_x = [&](Pos p, float (&xv)[KBW][RF]) {
#pragma unroll
        for (int t = 0; t < KBW; ++t) {
            load_x(p, xv[t]);
            p = advance(p, WK, a.nsb);
        }
    };

    Pos pc = advance(Pos{0, 0, 0}, wk, a.nsb);  // first block of the current chunk
    load_chunk_x(pc, xc);
    stage_load(0);
    stage_store(0);
    __syncthreads();
    silu_of(xc[0], sl);
    gen_block(pc, xc[0], sl, A_cur);

    // One chunk.  LAST: no next chunk (no prefetch, no generation past the
    // end), and blocks past the wave's last one multiply zeros.
    auto chunk = [&](int c, auto last_tag) {
        constexpr bool LAST = decltype(last_tag)::value;
        const int buf = c & 1;
        Pos pn = pc;
#pragma unroll
        for (int t = 0; t < KBW; ++t) pn = advance(pn, WK, a.nsb);  // first block of c + 1
        if constexpr (!LAST) {
            load_chunk_x(pn, xn);
            stage_load(c + 1);
        }
        Pos p = pc;
#pragma unroll
        for (int t = 0; t < KBW; ++t) {
            const Pos pnext = t + 1 < KBW ? advance(p, WK, a.nsb) : pn;
            const bool gen_next = !LAST || t + 1 < KBW;
            if (gen_next) {
                const float(&xv)[RF] = t + 1 < KBW ? xc[t + 1 < KBW ? t + 1 : 0] : xn[0];
                if (pnext.bsub == 0) silu_of(xv, sl);
                gen_block(pnext, xv, sl, A_nxt);
            }
            if constexpr (LAST) {
                if (c * KBW + t >= nq) {  // past the wave's last block: contribute 0
#pragma unroll
                    for (int rf = 0; rf < RF; ++rf) zero_frag(A_cur, rf);
                }
            }
            mfma_block(A_cur, buf, wk + WK * t);
            if (gen_next) A_cur = A_nxt;
            p = pnext;
        }
        if constexpr (!LAST) {
            stage_store((c + 1) & 1);
            __syncthreads();
#pragma unroll
            for (int t = 0; t < KBW; ++t)
#pragma unroll
                for (int rf = 0; rf < RF; ++rf) xc[t][rf] = xn[t][rf];
        }
        pc = pn;
    };

#pragma unroll 1
    for (int c = 0; c + 1 < a.nchunks; ++c) chunk(c, std::false_type{});
    chunk(a.nchunks - 1, std::true_type{});
    __syncthreads();

    // ---- epilogue
    const int col0 = nt * NTILE;
    if constexpr (WK == 1) {
        const bool full = row0 + 32 * RF <= a.batch && col0 + NTILE <= a.out;
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) {
#pragma unroll
            for (int nf = 0; nf < NF; ++nf) {
                const int col = col0 + nf * 32 + r;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int64_t row = row0 + rf * 32 + 8 * (q / 4) + 4 * h + (q % 4);
                    if (full || (row < a.batch && col < a.out))
                        Tr<T>::store(y + row * a.out + col, acc[rf][nf][q]);
                }
            }
        }
    } else {
        // Waves with the same wm hold partial sums of the same rows: write all
        // partials to LDS (the weight buffers are free after the last
        // barrier), then every thread sums WK partials of some elements and
        // stores them row-major (coalesced).
        constexpr int TILE = 32 * RF * NTILE;  // floats per wave
        float* red = reinterpret_cast<float*>(lds);
#pragma unroll
        for (int rf = 0; rf < RF; ++rf)
#pragma unroll
            for (int nf = 0; nf < NF; ++nf)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int rl = rf * 32 + 8 * (q / 4) + 4 * h + (q % 4);
                    red[wave * TILE + rl * NTILE + nf * 32 + r] = acc[rf][nf][q];
                }
        __syncthreads();
        const int64_t bm0 = (int64_t)blockIdx.x * BM;
        for (int idx = tid; idx < WM * TILE; idx += kThreads) {
            const int g = idx / TILE;
            const int rem = idx % TILE;
            const int rl = rem / NTILE;
            const int cl = rem % NTILE;
            float sum = 0.0f;
#pragma unroll
            for (int w = 0; w < WK; ++w) sum += red[(g + WM * w) * TILE + rem];
            const int64_t row = bm0 + g * 32 * RF + rl;
            const int col = col0 + cl;
            if (row < a.batch && col < a.out) Tr<T>::store(y + row * a.out + col, sum);
        }
    }
}

template <typename T, int RF, int NF, int WK>
hipError_t launch_cfg(const LayerGeom& g, LayerArgs a, hipStream_t s) {
    constexpr int WM = 4 / WK;
    constexpr int BM = 32 * RF * WM;
    constexpr int BLKB = 2 * 32 * NF * Tr<T>::KJ * (int)sizeof(T);
    constexpr int KB = (32768 / BLKB) < 8 ? (32768 / BLKB) : 8;
    a.nchunks = (a.nblk + KB - 1) / KB;
    const dim3 grid((unsigned)((a.batch + BM - 1) / BM), (unsigned)g.ntiles);
    hipLaunchKernelGGL((layer_kernel<T, RF, NF, WK>), grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <typename T, int NF>
hipError_t launch_nf(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s) {
    if (c.wk == 1) {
        if (c.rf == 1) return launch_cfg<T, 1, NF, 1>(g, a, s);
        if (c.rf == 2) return launch_cfg<T, 2, NF, 1>(g, a, s);
    }
    if constexpr (NF <= 4) {
        if (c.rf == 1 && c.wk == 2) return launch_cfg<T, 1, NF, 2>(g, a, s);
        if (c.rf == 1 && c.wk == 4) return launch_cfg<T, 1, NF, 4>(g, a, s);
    }
    if constexpr (NF <= 2) {
        if (c.rf == 2 && c.wk == 2) return launch_cfg<T, 2, NF, 2>(g, a, s);
        if (c.rf == 2 && c.wk == 4) return launch_cfg<T, 2, NF, 4>(g, a, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_t(const LayerGeom& g, const LayerCfg& c, const LayerArgs& a, hipStream_t s) {
    switch (g.nf) {
        case 1: return launch_nf<T, 1>(g, c, a, s);
        case 2: return launch_nf<T, 2>(g, c, a, s);
        case 4: return launch_nf<T, 4>(g, c, a, s);
        case 8:
            if constexpr (sizeof(T) == 2) return launch_nf<T, 8>(g, c, a, s);
            return hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// ------------------------------------------------------------------ planning

bool layer_geom(int nb, bool bf16, int in, int out, LayerGeom* g) {
    g->nb = nb;
    g->kj = bf16 ? 8 : 2;
    g->nsb = (nb + 1 + g->kj - 1) / g->kj;
    g->npairs = (in + 1) / 2;
    const int64_t nblk = (int64_t)g->npairs * g->nsb;
    // fp32 tiles are at most 128 columns wide (fp32 MFMA time dwarfs the basis
    // generation, so regenerating it per tile is cheap); bf16 tiles up to 256
    // so each basis value is generated once per row for out <= 256.
    const int nfmax = bf16 ? 8 : 4;
    const int need = (out + 31) / 32;
    int nf = 1;
    while (nf < nfmax && nf < need) nf *= 2;
    g->nf = nf;
    g->ntiles = (out + 32 * nf - 1) / (32 * nf);
    const int64_t blk_bytes = 2LL * 32 * nf * g->kj * (bf16 ? 2 : 4);  // [h][n][kj]
    if (nblk > 0x7fffffffLL / 8 || g->ntiles > 65535) return false;
    g->nblk = (int)nblk;
    g->packed_bytes = (size_t)g->ntiles * (size_t)nblk * (size_t)blk_bytes;
    return true;
}

bool layer_cfg_valid(const LayerGeom& g, const LayerCfg& c) {
    if (c.rf != 1 && c.rf != 2) return false;
    if (c.wk != 1 && c.wk != 2 && c.wk != 4) return false;
    return c.wk == 1 || c.rf * g.nf <= 4;
}

LayerCfg plan_layer(const LayerGeom& g, bool bf16, int64_t batch) {
    auto wgs = [&](const LayerCfg& c) {
        const int64_t bm = 32LL * c.rf * (4 / c.wk);
        return ((batch + bm - 1) / bm) * g.ntiles;
    };
    // bf16 with the widest tile: 64 rows per wave (one wave per SIMD, 256
    // accumulator registers) halves the LDS traffic per MFMA; one workgroup per
    // CU is enough.  Otherwise one 32-row tile per wave, two workgroups per CU
    // wanted, and the K split inside the workgroup when rows run out.
    if (bf16 && g.nf == 8) {
        LayerCfg c{2, 1};
        if (wgs(c) >= 256) return c;
        return LayerCfg{1, 1};
    }
    const LayerCfg cands[] = {{1, 1}, {1, 2}, {1, 4}};
    for (const LayerCfg& c : cands)
        if (wgs(c) >= 512) return c;
    return LayerCfg{1, 4};
}

bool parse_layer_cfg_override(const LayerGeom& g, LayerCfg* c) {
    const char* s = std::getenv("KAN_LAYER_CFG");
    if (!s || !*s) return false;
    LayerCfg t{0, 0};
    if (std::sscanf(s, "%d,%d", &t.rf, &t.wk) != 2) return false;
    if (!layer_cfg_valid(g, t)) return false;
    *c = t;
    return true;
}

// ------------------------------------------------------------------ launches

hipError_t launch_pack(bool bf16, const LayerGeom& g, int in, int out, const void* coef,
                       const void* base_w, void* packed, hipStream_t s) {
    const int ntile = 32 * g.nf;
    const int64_t units = (int64_t)g.ntiles * g.nblk * 2 * ntile;
    const unsigned blocks = (unsigned)((units + kThreads - 1) / kThreads);
    if (bf16)
        hipLaunchKernelGGL(pack_kernel<uint16_t>, dim3(blocks), dim3(kThreads), 0, s,
                           static_cast<const uint16_t*>(coef),
                           static_cast<const uint16_t*>(base_w), static_cast<uint16_t*>(packed),
                           in, out, g.nb, g.nsb, g.npairs, ntile, units);
    else
        hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(kThreads), 0, s,
                           static_cast<const float*>(coef), static_cast<const float*>(base_w),
                           static_cast<float*>(packed), in, out, g.nb, g.nsb, g.npairs, ntile,
                           units);
    return hipGetLastError();
}

hipError_t launch_layer(bool bf16, const LayerGeom& g, const LayerCfg& c, LayerArgs a,
                        hipStream_t s) {
    if (!layer_cfg_valid(g, c)) return hipErrorInvalidValue;
    return bf16 ? launch_t<uint16_t>(g, c, a, s) : launch_t<float>(g, c, a, s);
}

}  // namespace kan
