// kan_backward.hip -- gradients of the KAN layer (eq. kan_forward
// differentiated) for an upstream gradient dy [batch, out]:
//
//   dx[b, i]  = sum_o dy[b, o] ( sum_j C[o, i, j] N_j'(x[b, i]) + Wb[o, i] silu'(x[b, i]) )
//   dC[o,i,j] = sum_b dy[b, o] N_j(x[b, i])
//   dWb[o, i] = sum_b dy[b, o] silu(x[b, i])
//
// Both are contractions over a dense operand and run on the matrix cores:
//
//   dx:  Gm = dy W^T over the outputs (Gm[b, (i, c)] for every column c of
//        every feature), then per (row, feature) the dot product of its
//        columns with (silu'(x), N_0'(x), ..., N_{nb-1}'(x)).  The MFMA puts
//        the K rows in the A operand (the packed weights, staged in LDS and
//        shared by the workgroup's eight waves) and the batch rows in the B
//        operand (a wave's 32 rows of dy, held in registers for the whole
//        kernel); the A rows are permuted so that each lane's 16 accumulators
//        are 16 consecutive columns of one feature for one batch row, and the
//        derivative contraction runs in the lane with no cross-lane step
//        (features of more than 16 columns add the two lane halves).
//   dW:  dW^T = A^T dy over the batch, A the forward's basis / SiLU matrix
//        regenerated in registers (never stored), dy transposed once into
//        the workspace so that both MFMA operands hold consecutive batch rows
//        per lane.  The batch is split over workgroups; their fp32 partials
//        are summed in a fixed order by a reduce kernel (deterministic).
//
// The derivative of the clamped cubic (eq. truncated with eq. bounded) at
// v = u - 2 is, with a = min(|v|, 2), w = 2 - a and b = max(1 - a, 0),
//     N'(u) = sign(v) (2 b^2 - w^2 / 2),
// the term-by-term derivative of the reflected two-term form 6 N = w^3 - 4 b^3
// (w = 2 - |v| on the support): exactly 0 off the support, where the clamp
// holds the coordinate constant.
#include "kan_internal.h"

#include <algorithm>

namespace kan {

namespace {

constexpr int kThreads = 512;  // eight waves

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// silu(x) / 2 and silu'(x).
__device__ __forceinline__ float half_silu_b(float x) {
    return x * __builtin_amdgcn_rcpf(__builtin_fmaf(__expf(-x), 2.0f, 2.0f));
}
__device__ __forceinline__ float silu_deriv(float x) {
    const float s = __builtin_amdgcn_rcpf(1.0f + __expf(-x));
    return s * __builtin_fmaf(x, 1.0f - s, 1.0f);
}

// N'(u) at v = u - 2 (see the header comment).  m = 2 b^2 - w^2 / 2 <= 0, so
// N' = sign(v) m = copysign(m, -v).  A NaN coordinate gives 0 (the SiLU
// derivative carries the NaN).
__device__ __forceinline__ float dbasis(float v) {
    const float a = __builtin_fminf(__builtin_fabsf(v), 2.0f);
    const float w = 2.0f - a;
    const float b = __builtin_fmaxf(1.0f - a, 0.0f);
    const float m = __builtin_fmaf(2.0f * b, b, -0.5f * w * w);
    return __builtin_copysignf(m, -v);
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, bf16x2_t{(__bf16)lo, (__bf16)hi});
}

template <typename T> struct B;  // storage helpers
template <> struct B<float> {
    static __device__ __forceinline__ float ld(const float* p) { return *p; }
    static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
    // two consecutive elements, p aligned to both
    static __device__ __forceinline__ void st2(float* p, float v0, float v1) {
        *reinterpret_cast<floatx2*>(p) = floatx2{v0, v1};
    }
    static constexpr int E = 4;   // elements per 16-byte unit
};
template <> struct B<uint16_t> {
    static __device__ __forceinline__ float ld(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void st(uint16_t* p, float v) { *p = f32_to_bf16(v); }
    static __device__ __forceinline__ void st2(uint16_t* p, float v0, float v1) {
        *reinterpret_cast<uint32_t*>(p) = pack2_bf16(v0, v1);
    }
    static constexpr int E = 8;
};

// Local K row of A-operand row i of a 32-row dx tile: rows with (i / 4) % 2 == h
// land in lane half h of the accumulators, as local rows 16 h .. 16 h + 15.
__host__ __device__ constexpr int dx_local_row(int i) {
    return 16 * ((i / 4) % 2) + 4 * (i / 8) + i % 4;
}

// -------------------------------------------------------------- transposes

// dst[c][pos(b)] = src[b][c] for a row-major src [rows, cols], zero-padded to
// ceil(cols / 32) * 32 rows and rpad columns (rpad a multiple of 32).  With
// PERM each 32-row chunk of b is stored as its even rows then its odd rows
// (position 16 (b % 2) + b / 2 in the chunk): a 32x32x2 fp32 k-step takes rows
// 2 j and 2 j + 1 in its two lane halves, so a lane's rows of a chunk are then
// consecutive.  Used for dy (the B operand of dW) and x (read per feature for
// 32 consecutive batch rows by both backward kernels).
template <typename T, bool PERM>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ src,
                                                        T* __restrict__ dst, int64_t rows,
                                                        int cols, int64_t rpad) {
    __shared__ T tile[32][33];
    const int64_t b0 = (int64_t)blockIdx.x * 32;
    const int c0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 8 rows of 32
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int bl = ty + 8 * k;
        const int64_t b = b0 + bl;
        const int c = c0 + tx;
        tile[bl][tx] = (b < rows && c < cols) ? src[b * cols + c] : T(0);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int cl = ty + 8 * k;
        const int bl = tx;
        const int pos = PERM ? 16 * (bl & 1) + (bl >> 1) : bl;
        dst[(int64_t)(c0 + cl) * rpad + b0 + pos] = tile[bl][cl];
    }
}

// The same transposition (without PERM) in 64 x 64 tiles with 16-byte
// accesses, for bf16: four threads read a tile row's 64 elements (a 128-byte
// run of src) and four write an output row's 64 (a run of dst), each moving
// 16 elements.  vec: src and cols allow 16-byte loads (else element loads);
// drows = ceil(cols / 32) * 32 rows of dst are written, columns up to rpad.
template <typename T>
__global__ __launch_bounds__(256) void transpose64_kernel(const T* __restrict__ src,
                                                          T* __restrict__ dst, int64_t rows,
                                                          int cols, int64_t rpad, int drows,
                                                          bool vec) {
    constexpr int V = 16 / (int)sizeof(T);  // elements per 16-byte access
    constexpr int PER = 16;                 // elements per thread
    constexpr int PAD = V;                  // keeps tile rows 16-byte aligned
    __shared__ __align__(16) T tile[64][64 + PAD];
    const int64_t b0 = (int64_t)blockIdx.x * 64;
    const int c0 = blockIdx.y * 64;
    const int part = threadIdx.x & 3;
    {
        const int bl = threadIdx.x >> 2;
        const int64_t b = b0 + bl;
#pragma unroll
        for (int v = 0; v < PER / V; ++v) {
            const int cl = part * PER + v * V;
            const int c = c0 + cl;
            u32x4 w = {0u, 0u, 0u, 0u};
            if (b < rows) {
                if (vec && c + V <= cols) {
                    w = *reinterpret_cast<const u32x4*>(src + b * cols + c);
                } else {
                    T e[V];
#pragma unroll
                    for (int i = 0; i < V; ++i) e[i] = c + i < cols ? src[b * cols + c + i] : T(0);
                    w = __builtin_bit_cast(u32x4, e);
                }
            }
            *reinterpret_cast<u32x4*>(&tile[bl][cl]) = w;
        }
    }
    __syncthreads();
    const int cl = threadIdx.x >> 2;
    const int c = c0 + cl;
    if (c >= drows) return;
#pragma unroll
    for (int v = 0; v < PER / V; ++v) {
        const int bl = part * PER + v * V;
        const int64_t b = b0 + bl;
        if (b >= rpad) continue;  // (rpad is a multiple of V)
        T e[V];
#pragma unroll
        for (int i = 0; i < V; ++i) e[i] = tile[bl + i][cl];
        *reinterpret_cast<u32x4*>(dst + (int64_t)c * rpad + b) = __builtin_bit_cast(u32x4, e);
    }
}

// -------------------------------------------------------------- dx packing

// wtp[t][g][lane][e]: for lane (r, h) of 32-row K tile t and k-step group g,
// the weights W[o][K row of A row r] of the group's outputs o of the lane half:
// bf16 o = 16 g + 8 h + e (one 32x32x16 k-step), fp32 o = 8 g + 2 e + h (four
// 32x32x2 k-steps).  W[o][(f, c)] is Wb[o][f] for c = 0, coef[o][f][c - 1] for
// 1 <= c <= nb, else 0; rows of features past `in` and outputs past `out` are 0.
template <typename T>
__global__ __launch_bounds__(256) void pack_dx_kernel(const T* __restrict__ coef,
                                                      const T* __restrict__ bw,
                                                      T* __restrict__ wtp, int in, int out, int nb,
                                                      int cp, int groups, int64_t units) {
    constexpr int E = B<T>::E;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= units) return;
    const int lane = (int)(u % 64);
    const int g = (int)((u / 64) % groups);
    const int64_t t = u / (64LL * groups);
    const int r = lane & 31, h = lane >> 5;
    const int64_t R = 32 * t + dx_local_row(r);
    const int f = (int)(R / cp);
    const int c = (int)(R % cp);
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int o = sizeof(T) == 2 ? 16 * g + 8 * h + e : 8 * g + 2 * e + h;
        T w = T(0);
        if (o < out && f < in) {
            const int64_t row = (int64_t)o * in + f;
            if (c == 0) w = bw[row];
            else if (c <= nb) w = coef[row * nb + c - 1];
        }
        v[e] = w;
    }
    T* d = wtp + u * E;
#pragma unroll
    for (int e = 0; e < E; ++e) d[e] = v[e];
}

// ------------------------------------------------------------------ dx

template <typename T>
struct DxArgs {
    const T* xt;       // x transposed: [in][bpad]
    int64_t bpad;
    const T* dy;
    const u32x4* wtp;  // packed weights, 16-byte units
    T* dx;
    float* dxp;        // per-chunk partials when the outputs take several chunks
    int64_t batch;
    int in, out, nb, cp, ntiles, groups, gmax;
    int tiles_per_split;  // K tiles of a workgroup (blockIdx.z), whole features
    float inv_h, inv_lo, xlim, a_int, a_frac;
};

// One workgroup: 8 RF 32 batch rows (eight waves of RF 32-row tiles) against
// the K tiles of split blockIdx.z, for output chunk blockIdx.y (up to gmax
// k-step groups, 256 outputs).  SM bounds the groups of a chunk at compile
// time.  Every A fragment read from LDS feeds RF MFMAs.
//
// Pipeline (two LDS stages, two register sets, loop unrolled by two so the
// sets are compile-time choices): LDS stage t % 2 holds tile t; during tile t
// the MFMAs and the epilogue run, then the loads of tile t + 2 (weights, and
// x of the lane's rows for its epilogue) go into register set t % 2 and
// register set (t + 1) % 2, loaded a whole tile earlier, is stored to stage
// (t + 1) % 2 before the barrier.
template <typename T, int SM, int RF, int NW>
__global__ __launch_bounds__(64 * NW) void dx_kernel(DxArgs<T> a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int NT = 64 * NW;
    constexpr int UPT = (SM * 64 + NT - 1) / NT;  // 16-byte units per thread per tile
    __shared__ u32x4 lds[2][SM * 64];
    // per wave: a lane's 16 accumulators after 4 zero floats (stride 80 bytes,
    // so the 16-byte writes of 16 lanes fall in distinct banks; the next
    // lane's zeros, and 4 after the last lane, follow them), read back at the
    // four columns the clamped derivative can make nonzero
    __shared__ u32x4 gat[NW][64 * 5 + 1];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, r = lane & 31, h = lane >> 5;
    const int64_t row0 = (int64_t)blockIdx.x * (NW * 32 * RF) + wave * (32 * RF) + r;
    int64_t rowc[RF];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        const int64_t row = row0 + 32 * rf;
        rowc[rf] = row < a.batch ? row : a.batch - 1;
    }
    const int ch = blockIdx.y;
    const int g0 = ch * a.gmax;
    const int S = min(a.gmax, a.groups - g0);
    const int t_begin = blockIdx.z * a.tiles_per_split;
    const int t_end = min(t_begin + a.tiles_per_split, a.ntiles);

    // B operands: the lane's batch rows of dy for every k-step group of the chunk
    u32x4 dyr[RF][SM];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        const T* dyrow = a.dy + rowc[rf] * a.out;
#pragma unroll
        for (int s = 0; s < SM; ++s) {
            float v[B<T>::E];
#pragma unroll
            for (int e = 0; e < B<T>::E; ++e) {
                const int o = BF ? (g0 + s) * 16 + 8 * h + e : (g0 + s) * 8 + 2 * e + h;
                v[e] = (s < S && o < a.out) ? B<T>::ld(dyrow + o) : 0.0f;
            }
            if constexpr (BF)
                dyr[rf][s] = u32x4{pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]),
                                   pack2_bf16(v[4], v[5]), pack2_bf16(v[6], v[7])};
            else
                dyr[rf][s] = u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]),
                                   __float_as_uint(v[2]), __float_as_uint(v[3])};
        }
    }

    typedef u32x4 WSet[UPT];
    typedef T XSet[RF];
    // Tile t's rows are features f0(t) + h of 16 columns each (cp = 16), or
    // columns 16 h .. 16 h + 15 of feature f0(t) (cp a multiple of 32):
    // f0(t) is the same for the whole wave.
    const bool cp16 = a.cp == 16;
    auto feat0 = [&](int t) -> int { return cp16 ? 2 * t : (32 * t) / a.cp; };
    // per-lane offsets fixed for the whole kernel: units of the weight loads,
    // x rows (in x transposed, relative to feature f0), dx rows
    int wl[UPT];
#pragma unroll
    for (int k = 0; k < UPT; ++k) wl[k] = min(tid + k * NT, S * 64 - 1);
    int64_t xl[RF], dxo[RF];
    bool rowok[RF];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
        const int64_t row = row0 + 32 * rf;
        xl[rf] = rowc[rf] + (cp16 && h ? a.bpad : 0);
        rowok[rf] = row < a.batch;
        dxo[rf] = (a.dxp != nullptr ? (int64_t)ch * a.batch + row : row) * a.in;
    }
    // Register sets: tile t's loads go to set t % L, issued L tiles before
    // the tile and stored to LDS one tile before it, so each store waits for
    // loads issued L - 1 tiles earlier (a tile is short: with one tile of
    // distance the stores wait on most of a memory round trip).
    constexpr int L = SM >= 32 ? 2 : 4;  // (32 k-steps of fp32 dy already fill the registers)
    WSet wq[L];
    XSet xq[L];
    // Loads of tile t: unconditional (tiles past the split's last, units past
    // the chunk's and features past `in` re-read valid addresses; their
    // values are not used), so the compiler's wait before a register set is
    // used counts only the loads issued after it.  x comes from its
    // transpose: a lane half reads 32 consecutive rows of one feature.
    auto issue = [&](int t, WSet& w, XSet& xs) {
        const int tc = min(t, t_end - 1);
        const u32x4* src = a.wtp + ((int64_t)tc * a.groups + g0) * 64;
#pragma unroll
        for (int k = 0; k < UPT; ++k) w[k] = src[wl[k]];
        const T* xb = a.xt + (int64_t)feat0(tc) * a.bpad;  // (the lane half's rows: xl)
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) xs[rf] = xb[xl[rf]];
    };
    auto put = [&](int buf, const WSet& w) {
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + k * NT;
            if (u < S * 64) lds[buf][u] = w[k];
        }
    };
    auto to_f = [&](T v) -> float {
        if constexpr (BF) return bf16_to_f32(v);
        else return v;
    };
    auto store_dx = [&](int rf, int f, float v) {
        if (rowok[rf] && f < a.in) {
            if (a.dxp != nullptr)
                a.dxp[dxo[rf] + f] = v;
            else
                B<T>::st(a.dx + dxo[rf] + f, v);
        }
    };

    const int tpf = a.cp / 32;  // tiles per feature (cp >= 32)
    float dxacc[RF];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) dxacc[rf] = 0.0f;

    // The MFMAs of the tile in LDS stage `buf`: acc[rf][q] = Gm[row][K row of
    // the tile's local row q (lane half h)].  Groups past S multiply zeros
    // (the LDS rows past the chunk's are zero, and so is dyr there), so the
    // loop has no branch and its LDS reads can run ahead of the MFMAs.
    auto mma = [&](int buf, floatx16 (&acc)[RF]) {
#pragma unroll
        for (int rf = 0; rf < RF; ++rf)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[rf][q] = 0.0f;
        const u32x4* st = lds[buf];
        // every A fragment of the tile read before the first MFMA (bf16: the
        // group barriers below keep them there; left to itself the compiler
        // keeps two reads in flight and each pair of MFMAs waits on the LDS:
        // 784 -> 256 dx 596 -> 534 us)
        u32x4 wv[SM];
#pragma unroll
        for (int s = 0; s < SM; ++s) wv[s] = st[s * 64 + lane];
#pragma unroll
        for (int s = 0; s < SM; ++s) {
            const u32x4 w = wv[s];
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) {
                if constexpr (BF) {
                    acc[rf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, w), __builtin_bit_cast(bf16x8, dyr[rf][s]),
                        acc[rf], 0, 0, 0);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[rf] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            __uint_as_float(w[j]), __uint_as_float(dyr[rf][s][j]), acc[rf], 0, 0,
                            0);
                }
            }
        }
        if constexpr (BF) {
            __builtin_amdgcn_sched_group_barrier(0x100, SM, 0);       // the LDS reads
            __builtin_amdgcn_sched_group_barrier(0x008, SM * RF, 0);  // then the MFMAs
        }
    };

    // The epilogue of tile t, without stores: acc[rf][q] = Gm[row][feature f,
    // column c0 + q].  Of the basis columns only the four with |v| < 2 have a
    // nonzero derivative: with s the coordinate of column 0 of the feature,
    // tau = s - floor(s) and clo = floor(s) - 1, column clo + k has u = tau +
    // 3 - k, where the derivative of the cubic (its segment form on the span)
    // is
    //   k = 0: -(1 - tau)^2 / 2      k = 1: (3 tau^2 - 4 tau) / 2
    //   k = 2: (1 + 2 tau - 3 tau^2) / 2   k = 3: tau^2 / 2.
    // Column 0 carries the SiLU derivative.  The four accumulators are read
    // back from a wave-private LDS copy (their index differs per lane).  xvs:
    // the lane's x of the tile's feature, per row tile.  Returns the tile's
    // contribution to dx per row tile in sum.
    auto epi_sum = [&](int t, const floatx16 (&acc)[RF], const float (&xvs)[RF],
                       float (&sum)[RF]) {
        const int fu = feat0(t);
        const int f = cp16 ? fu + h : fu;
        const int c0 = cp16 ? 0 : 32 * t - fu * a.cp + 16 * h;
        char* gl = reinterpret_cast<char*>(gat[wave]) + lane * 80;
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) {
            const float xv = f < a.in ? xvs[rf] : 0.0f;
            // coordinate of column c0 (its integer offset folded into the fma),
            // clamped to keep the window index small for far-out inputs; +-Inf
            // lands outside every column, NaN is carried by the SiLU term
            const float sc = __builtin_amdgcn_fmed3f(
                __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f - (float)c0) +
                    coord_lo(xv, a.xlim, a.inv_lo, a.a_frac),
                -8.0f, 24.0f);
            const float fl = __builtin_floorf(sc);
            const float tau = sc - fl;
            const float t2 = tau * tau;
            float d[4];
            d[0] = -0.5f * (1.0f - tau) * (1.0f - tau);
            d[1] = __builtin_fmaf(1.5f, t2, -2.0f * tau);
            d[2] = __builtin_fmaf(-1.5f, t2, __builtin_fmaf(tau, 1.0f, 0.5f));
            d[3] = 0.5f * t2;
            // the lane's 16 columns after its 4 zeros; the SiLU column (c = 0)
            // is not a basis column and reads as 0 too
#pragma unroll
            for (int m = 0; m < 4; ++m)
                *reinterpret_cast<floatx4*>(gl + 16 + 16 * m) =
                    floatx4{m == 0 && c0 == 0 ? 0.0f : acc[rf][4 * m], acc[rf][4 * m + 1],
                            acc[rf][4 * m + 2], acc[rf][4 * m + 3]};
            // window columns q = qlo .. qlo + 3 relative to c0: columns outside
            // the lane's 16 read the zeros around them (padding columns past
            // nb hold exact zeros: their weights are 0), and a window wholly
            // outside is moved onto 4 zeros
            const int qlo = min(max((int)fl - 1, -4), 16);
            const float* gw = reinterpret_cast<const float*>(gl + 16 + 4 * qlo);
            float sb = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) sb = __builtin_fmaf(gw[k], d[k], sb);
            sum[rf] = __builtin_fmaf(c0 == 0 ? acc[rf][0] : 0.0f, silu_deriv(xv), a.inv_h * sb);
        }
    };
    // The tile's stores: dx of its feature, or (features of two tiles) the
    // running sum, stored at the feature's last tile.
    auto epi_store = [&](int t, const float (&sum)[RF]) {
        const int f = cp16 ? feat0(t) + h : feat0(t);
        if (a.cp == 16) {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) store_dx(rf, f, sum[rf]);
        } else {
#pragma unroll
            for (int rf = 0; rf < RF; ++rf) dxacc[rf] += sum[rf];
            if ((t + 1) % tpf == 0) {  // the feature's last tile: add the two halves
#pragma unroll
                for (int rf = 0; rf < RF; ++rf) {
                    const float tot = dxacc[rf] + __shfl_xor(dxacc[rf], 32);
                    if (h == 0) store_dx(rf, f, tot);
                    dxacc[rf] = 0.0f;
                }
            }
        }
    };
    auto xfloat = [&](const XSet& xs, float (&xv)[RF]) {
#pragma unroll
        for (int rf = 0; rf < RF; ++rf) xv[rf] = to_f(xs[rf]);
    };

    // LDS rows of groups past the chunk's are never written by put: zero them
    // once (the MFMAs of those groups then add exact zeros).  Likewise the
    // zeros around each lane's gather slot, never written after this.
    for (int u = S * 64 + tid; u < SM * 64; u += NT) {
        lds[0][u] = u32x4{0u, 0u, 0u, 0u};
        lds[1][u] = u32x4{0u, 0u, 0u, 0u};
    }
    {
        char* gw0 = reinterpret_cast<char*>(gat[wave]);
        *reinterpret_cast<u32x4*>(gw0 + lane * 80) = u32x4{0u, 0u, 0u, 0u};
        if (lane == 63) *reinterpret_cast<u32x4*>(gw0 + 64 * 80) = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < L; ++j) issue(t_begin + j, wq[j], xq[j]);
    put(0, wq[0]);
    __syncthreads();
    if constexpr (BF) {
        // bf16 (a tile's MFMAs are short next to its epilogue): software
        // pipelined over two accumulator sets.  The iteration of tile t issues
        // its MFMAs and computes tile t - 1's epilogue in the same straight-line
        // code, so that VALU and LDS work overlaps the MFMAs; the stores
        // follow.  x of tile t is kept as floats (xp) before its register set
        // is reloaded.  Tile t_begin + i uses LDS stage i % 2, register set
        // i % L and accumulator set i % 2 (L is even).
        floatx16 acc[2][RF];
        float xp[2][RF];
        float sum[RF];
        if (t_begin < t_end) {  // the first tile: MFMAs only
            mma(0, acc[0]);
            xfloat(xq[0], xp[0]);
            issue(t_begin + L, wq[0], xq[0]);
            if (t_begin + 1 < t_end) put(1, wq[1 % L]);
            __syncthreads();
        }
#pragma unroll 1
        for (int tb = t_begin + 1; tb < t_end; tb += L) {
            bool done = false;
            StaticFor<0, L>::run([&](auto jj) {
                constexpr int j = decltype(jj)::value;
                constexpr int i = j + 1;  // t - t_begin, mod L
                constexpr int p = i & 1;
                const int t = tb + j;
                if (done || t >= t_end) {
                    done = true;
                    return;
                }
                mma(p, acc[p]);
                epi_sum(t - 1, acc[p ^ 1], xp[p ^ 1], sum);
                epi_store(t - 1, sum);
                xfloat(xq[i % L], xp[p]);
                issue(t + L, wq[i % L], xq[i % L]);
                if (t + 1 < t_end) put((i + 1) & 1, wq[(i + 1) % L]);
                __syncthreads();
                __builtin_amdgcn_sched_barrier(0);
            });
        }
        const int tl = t_end - 1;  // the last tile's epilogue
        if (tl >= t_begin) {
            if (((tl - t_begin) & 1) == 0) epi_sum(tl, acc[0], xp[0], sum);
            else epi_sum(tl, acc[1], xp[1], sum);
            epi_store(tl, sum);
        }
    } else {
        // tile t = t_begin + L i + j: LDS stage j % 2, register set j
#pragma unroll 1
        for (int tb = t_begin; tb < t_end; tb += L) {
            bool done = false;
            StaticFor<0, L>::run([&](auto jj) {
                constexpr int j = decltype(jj)::value;
                const int t = tb + j;
                if (done || t >= t_end) {
                    done = true;
                    return;
                }
                floatx16 acc[RF];
                float xv[RF], sum[RF];
                mma(j & 1, acc);
                xfloat(xq[j], xv);
                epi_sum(t, acc, xv, sum);
                epi_store(t, sum);
                issue(t + L, wq[j], xq[j]);
                if (t + 1 < t_end) put((j + 1) & 1, wq[(j + 1) % L]);
                __syncthreads();
                __builtin_amdgcn_sched_barrier(0);  // (tiles are not interleaved)
            });
        }
    }
}

// dx = sum over output chunks of the partials, in chunk order.
template <typename T>
__global__ __launch_bounds__(256) void dx_reduce_kernel(const float* __restrict__ dxp,
                                                        T* __restrict__ dx, int64_t n,
                                                        int nchunk) {
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= n) return;
    float s = 0.0f;
    for (int c = 0; c < nchunk; ++c) s += dxp[(int64_t)c * n + u];
    B<T>::st(dx + u, s);
}

// ------------------------------------------------------------------ dW

template <typename T>
struct DwArgs {
    const T* xt;    // x transposed: [in][bpad]
    const T* dyt;   // [out32][bpad]
    float* P;       // [split][out32][kr] partial sums of dW^T / 2
    int64_t batch, bpad;
    int in, out32, nb, cp, kr, rows_per_split;
    float inv_h, inv_lo, xlim, a_int, a_frac;
};

// Workgroup: the 256 K rows [kt0, kt0 + 256) x outputs [ot0, ot0 + OT) over
// the batch rows of split blockIdx.y.  Wave (kg, oh) holds RF = OH 32-row K
// tiles by NFW 32-output fragments (8 / OH K groups of RF tiles: 256 rows).
//
// Per chunk of 32 batch rows the workgroup stages in LDS, double-buffered:
//   * the transposed dy of its outputs (plain copies of contiguous runs);
//   * the chunk of the A operand (K rows x 32 batch rows: N_c(x) / 2 and
//     silu(x) / 2), built once per workgroup: each thread owns (batch row,
//     feature) pairs and writes only the four columns the clamped form can
//     make nonzero (c = floor(s) - 1 .. floor(s) + 2, s the coordinate of
//     column 0) and the SiLU column, after clearing the four it wrote two
//     chunks earlier in the same stage.  Every other entry stays 0 (the
//     stages start cleared), which is the value of the clamped form there.
// Each wave then reads its A and B fragments from LDS: every A fragment
// feeds NFW MFMAs and every B fragment RF.
template <typename T, int OH, int NFW>
__global__ __launch_bounds__(kThreads) void dw_kernel(DwArgs<T> a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int RF = OH;
    constexpr int KG = 8 / OH;
    constexpr int KT = KG * RF * 32;            // 256
    constexpr int OT = OH * NFW * 32;
    constexpr int NFEAT = KT / 16 + 2;          // features a workgroup's K rows touch, at most
    constexpr int UR = BF ? 4 : 8;              // 16-byte units of a chunk's 32 batch values
    constexpr int ROWU = UR + 1;                // LDS row stride in units (one unit of padding)
    constexpr int ES = sizeof(T);
    constexpr int DU = (OT * UR + kThreads - 1) / kThreads;     // dy units per thread
    constexpr int XU = (32 * NFEAT + kThreads - 1) / kThreads;  // (row, feature) pairs per thread
    static_assert(KT == 256, "K rows per workgroup");
    __shared__ u32x4 dys[2][OT * ROWU];
    // (row KT of each stage: a dummy row that takes the writes of lanes with
    // nothing to write, so that building the A chunk has no branch)
    __shared__ u32x4 as[2][(KT + 1) * ROWU];
    // features with a NaN input in this workgroup's rows: their basis
    // gradients are NaN (N_j(NaN) is NaN; the clamped form would give 0)
    __shared__ int nanf[NFEAT];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, r = lane & 31, h = lane >> 5;
    const int kg = wave / OH, oh = wave % OH;
    const int kt0 = blockIdx.x * KT;
    const int ot0 = blockIdx.z * OT;
    const int F0 = kt0 / a.cp;
    const int F1 = min((kt0 + KT - 1) / a.cp, (a.kr - 1) / a.cp);
    const int nfeat = F1 - F0 + 1;
    const int64_t b_begin = (int64_t)blockIdx.y * a.rows_per_split;
    const int64_t b_end = min(b_begin + a.rows_per_split, a.bpad);
    const int nchunks = (int)((b_end - b_begin) / 32);

    for (int i = tid; i < NFEAT; i += kThreads) nanf[i] = 0;
    for (int i = tid; i < 2 * (KT + 1) * ROWU; i += kThreads)
        (&as[0][0])[i] = u32x4{0u, 0u, 0u, 0u};

    typedef u32x4 DSet[DU];
    typedef T XSet[XU];
    DSet dq[2];
    XSet xq[2];
    int prev[2][XU];  // first window column written two chunks ago in each stage (or -8)
    bool nanx[XU];    // a NaN input seen in the thread's (batch row, feature) pairs
#pragma unroll
    for (int k = 0; k < XU; ++k) {
        prev[0][k] = prev[1][k] = -8;
        nanx[k] = false;
    }

    // Loads of chunk ck: unconditional (chunks past the split's last, units
    // past the tile's and features past `in` re-read valid addresses; their
    // values are not used or are replaced), so the compiler's wait before a
    // register set is used counts only the loads issued after it.  Rows past
    // the batch are zero in both transposes.
    auto issue = [&](int ck, DSet& d, XSet& xs) {
        const int64_t b0 = b_begin + 32 * (int64_t)min(ck, nchunks - 1);
#pragma unroll
        for (int k = 0; k < DU; ++k) {
            const int u = min(tid + k * kThreads, OT * UR - 1);
            const int o = min(ot0 + u / UR, a.out32 - 1), w = u % UR;
            d[k] = *reinterpret_cast<const u32x4*>(
                reinterpret_cast<const char*>(a.dyt + (int64_t)o * a.bpad + b0) + 16 * w);
        }
#pragma unroll
        for (int k = 0; k < XU; ++k) {
            const int idx = min(tid + k * kThreads, 32 * nfeat - 1);
            const int bl = idx % 32, f = min(F0 + idx / 32, a.in - 1);
            xs[k] = a.xt[(int64_t)f * a.bpad + b0 + bl];
        }
    };
    // one A entry: K row R (absolute), batch row bl of the chunk; with ok
    // false, or R outside the workgroup's K rows, the dummy row takes it
    auto put_a = [&](int buf, int R, int bl, float v, bool ok) {
        const int lr = R - kt0;
        const int lre = ok && lr >= 0 && lr < KT ? lr : KT;
        const int pos = BF ? bl : 16 * (bl & 1) + (bl >> 1);
        char* p = reinterpret_cast<char*>(&as[buf][lre * ROWU]) + pos * ES;
        if constexpr (BF)
            *reinterpret_cast<uint16_t*>(p) = f32_to_bf16(v);
        else
            *reinterpret_cast<float*>(p) = v;
    };
    // Stage chunk data: dy by plain copies, and the A chunk: per (batch row,
    // feature) pair of the thread the SiLU column and the four window columns,
    // after clearing the four written two chunks earlier in this stage.
    // Straight-line code (no branch on lanes), so that the compiler can
    // interleave it with the MFMAs of the other stage.
    auto stage = [&](int buf, const DSet& d, const XSet& xs, int (&pv)[XU]) {
#pragma unroll
        for (int k = 0; k < DU; ++k) {
            const int u = tid + k * kThreads;
            if ((OT * UR) % kThreads == 0 || u < OT * UR)
                dys[buf][(u / UR) * ROWU + u % UR] = d[k];
        }
#pragma unroll
        for (int k = 0; k < XU; ++k) {
            if (k > 0 && k * kThreads >= 32 * nfeat) break;  // (the same for every lane)
            const int idx = tid + k * kThreads;
            const bool valid = idx < 32 * nfeat;
            const int bl = idx % 32, fl = idx / 32;
            const int Rf = (F0 + fl) * a.cp;  // K row of the feature's column 0
            float xv;
            if constexpr (BF) xv = bf16_to_f32(xs[k]);
            else xv = xs[k];
            xv = F0 + fl >= a.in ? 0.0f : xv;  // (a padding feature)
            const bool isn = xv != xv;
            nanx[k] = nanx[k] || (valid && isn);
            // clear the window written two chunks ago in this stage
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int c = pv[k] + m;
                put_a(buf, Rf + c, bl, 0.0f, valid && c >= 1 && c <= a.nb);
            }
            put_a(buf, Rf, bl, half_silu_b(xv), valid);
            // coordinate of column 0 (clamped so that the column index stays
            // small for far-out or infinite inputs), the window's first
            // column, then each value with its column folded into the fma's
            // exact integer addend; a NaN input writes no basis value
            const float lot = coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
            const float s0 = __builtin_amdgcn_fmed3f(
                __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f) + lot, -8.0f, (float)(a.nb + 8));
            const int clo = isn ? -8 : (int)__builtin_floorf(s0) - 1;
            pv[k] = clo;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int c = clo + m;
                const float v = __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f - (float)c) + lot;
                put_a(buf, Rf + c, bl, half_basis(v), valid && c >= 1 && c <= a.nb);
            }
        }
    };

    floatx16 acc[RF][NFW];
#pragma unroll
    for (int rt = 0; rt < RF; ++rt)
#pragma unroll
        for (int nf = 0; nf < NFW; ++nf)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[rt][nf][q] = 0.0f;

    auto chunk = [&](int buf) {
        const char* dl = reinterpret_cast<const char*>(dys[buf]);
        const char* al = reinterpret_cast<const char*>(as[buf]);
        if constexpr (BF) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {  // k-steps of 16 batch rows
                bf16x8 A[RF];
#pragma unroll
                for (int rt = 0; rt < RF; ++rt) {
                    const int lr = 32 * (kg * RF + rt) + r;
                    A[rt] = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u32x4*>(al + lr * ROWU * 16 + 32 * s + 16 * h));
                }
#pragma unroll
                for (int nf = 0; nf < NFW; ++nf) {
                    const int o = (oh * NFW + nf) * 32 + r;
                    const bf16x8 Bv = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u32x4*>(dl + o * ROWU * 16 + 32 * s + 16 * h));
#pragma unroll
                    for (int rt = 0; rt < RF; ++rt)
                        acc[rt][nf] =
                            __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[rt], Bv, acc[rt][nf], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int jg = 0; jg < 4; ++jg) {  // groups of four 32x32x2 k-steps
                floatx4 A[RF];
#pragma unroll
                for (int rt = 0; rt < RF; ++rt) {
                    const int lr = 32 * (kg * RF + rt) + r;
                    A[rt] = *reinterpret_cast<const floatx4*>(al + lr * ROWU * 16 + 64 * h + 16 * jg);
                }
#pragma unroll
                for (int nf = 0; nf < NFW; ++nf) {
                    const int o = (oh * NFW + nf) * 32 + r;
                    const floatx4 Bv =
                        *reinterpret_cast<const floatx4*>(dl + o * ROWU * 16 + 64 * h + 16 * jg);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int rt = 0; rt < RF; ++rt)
                            acc[rt][nf] = __builtin_amdgcn_mfma_f32_32x32x2f32(A[rt][e], Bv[e],
                                                                              acc[rt][nf], 0, 0, 0);
                }
            }
        }
    };

    // Pipeline: stage ck % 2 holds chunk ck; register set ck % 2 is loaded two
    // chunks ahead, staged one chunk before its use.  The loop takes two
    // chunks per trip (the stages and sets are compile-time choices); it
    // stages one chunk past the last (the loads are clamped to the last
    // chunk; that stage is never multiplied), and an odd last chunk follows.
    __syncthreads();  // (stages cleared, flags reset)
    issue(0, dq[0], xq[0]);
    issue(1, dq[1], xq[1]);
    if (nchunks > 0) {
        stage(0, dq[0], xq[0], prev[0]);
        __syncthreads();
        int ck = 0;
        for (; ck + 1 < nchunks; ck += 2) {
            chunk(0);
            issue(ck + 2, dq[0], xq[0]);
            stage(1, dq[1], xq[1], prev[1]);
            __syncthreads();
            chunk(1);
            issue(ck + 3, dq[1], xq[1]);
            stage(0, dq[0], xq[0], prev[0]);
            __syncthreads();
        }
        if (ck < nchunks) chunk(0);
    }
#pragma unroll
    for (int k = 0; k < XU; ++k)
        if (nanx[k]) nanf[(tid + k * kThreads) / 32] = 1;
    __syncthreads();

    // acc[rt][nf][q] = (dW^T / 2)[K row kt0 + 32 (kg RF + rt) + 8 (q / 4) + 4 h + q % 4][output o]
#pragma unroll
    for (int rt = 0; rt < RF; ++rt) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int R = kt0 + 32 * (kg * RF + rt) + 8 * (q / 4) + 4 * h + q % 4;
            const int f = R / a.cp;
            const int c = R - f * a.cp;
            const int fq = min(max(f - F0, 0), NFEAT - 1);
            if (c != 0 && nanf[fq]) {
#pragma unroll
                for (int nf = 0; nf < NFW; ++nf) acc[rt][nf][q] = __builtin_nanf("");
            }
        }
    }
    float* P = a.P + (int64_t)blockIdx.y * a.out32 * a.kr;
#pragma unroll
    for (int rt = 0; rt < RF; ++rt) {
#pragma unroll
        for (int nf = 0; nf < NFW; ++nf) {
            const int o = ot0 + (oh * NFW + nf) * 32 + r;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int R = kt0 + 32 * (kg * RF + rt) + 8 * m + 4 * h;
                if (o < a.out32 && R < a.kr)
                    *reinterpret_cast<floatx4*>(P + (int64_t)o * a.kr + R) =
                        floatx4{acc[rt][nf][4 * m], acc[rt][nf][4 * m + 1], acc[rt][nf][4 * m + 2],
                                acc[rt][nf][4 * m + 3]};
            }
        }
    }
}

// dcoef[o][f][c - 1] / dbw[o][f] = 2 sum_s P[s][o][f cp + c], splits in order.
template <typename T>
__global__ __launch_bounds__(256) void dw_reduce_kernel(const float* __restrict__ P,
                                                        T* __restrict__ dcoef, T* __restrict__ dbw,
                                                        int split, int out, int out32, int in,
                                                        int nb, int cp, int kr) {
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t n = (int64_t)out * in * (nb + 1);
    if (u >= n) return;
    const int c = (int)(u % (nb + 1));
    const int64_t of = u / (nb + 1);  // o * in + f
    const int f = (int)(of % in);
    const int o = (int)(of / in);
    float s = 0.0f;
    for (int k = 0; k < split; ++k)
        s += P[((int64_t)k * out32 + o) * kr + (int64_t)f * cp + c];
    s *= 2.0f;
    if (c == 0)
        B<T>::st(dbw + of, s);
    else
        B<T>::st(dcoef + of * nb + c - 1, s);
}

// ---------------------------------------------------------------- launches

template <typename T, int SM, int RF, int NW = 8>
hipError_t launch_dx_sm(const BwdGeom& g, const DxArgs<T>& d, hipStream_t s) {
    constexpr int BM = NW * 32 * RF;
    const dim3 grid((unsigned)((d.batch + BM - 1) / BM), (unsigned)g.nchunk,
                    (unsigned)g.dx_ksplit);
    hipLaunchKernelGGL((dx_kernel<T, SM, RF, NW>), grid, dim3(64 * NW), 0, s, d);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_dx(const BwdGeom& g, const DxArgs<T>& d, hipStream_t s) {
    const int sm = min(g.groups, g.gmax);  // groups of the largest chunk
    // two row tiles per wave while their dy registers stay within 64
    if (g.dx_rf == 2) {
        if (sm <= 1) return launch_dx_sm<T, 1, 2>(g, d, s);
        if (sm <= 2) return launch_dx_sm<T, 2, 2>(g, d, s);
        if (sm <= 4) return launch_dx_sm<T, 4, 2>(g, d, s);
        if (sm <= 8) return launch_dx_sm<T, 8, 2>(g, d, s);
        return hipErrorInvalidValue;
    }
    if (sm <= 16) return launch_dx_sm<T, 16, 1>(g, d, s);
    if constexpr (sizeof(T) == 4) {
        if (sm <= 32) return launch_dx_sm<T, 32, 1>(g, d, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_dw(const BwdGeom& g, const DwArgs<T>& d, hipStream_t s) {
    const dim3 grid((unsigned)g.ktiles, (unsigned)g.split, (unsigned)g.otiles);
    if (g.oh == 1 && g.nfw == 1)
        hipLaunchKernelGGL((dw_kernel<T, 1, 1>), grid, dim3(kThreads), 0, s, d);
    else if (g.oh == 2 && g.nfw == 1)
        hipLaunchKernelGGL((dw_kernel<T, 2, 1>), grid, dim3(kThreads), 0, s, d);
    else if (g.oh == 2 && g.nfw == 2)
        hipLaunchKernelGGL((dw_kernel<T, 2, 2>), grid, dim3(kThreads), 0, s, d);
    else if (g.oh == 2 && g.nfw == 4)
        hipLaunchKernelGGL((dw_kernel<T, 2, 4>), grid, dim3(kThreads), 0, s, d);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// ------------------------------------------------------- dx of narrow layers
//
// Layers of at most 16 outputs at large batches: dx on the vector ALUs.  Of a
// (row, feature)'s columns only the SiLU column and the four basis columns
// whose support holds x have a nonzero derivative, so
//   dx[b, i] = silu'(x) t_0 + (1/h) sum_{k<4} N'(u of column c0 + k) t_{c0+k},
//   t_c = sum_o dy[b, o] W[o, (i, c)],
// with a feature's columns [SiLU weight, coef[o, i, 0 .. nb - 1]] and c0 the
// window's first column, placed as in the forward's narrow-layer kernel
// (c0 in [1, nb - 1]; a column the clamp takes in has |v| >= 2, where the
// closed form of N' is exactly 0).  narrow_dx_table_kernel writes the weights
// as a table [feature][column][output] (zeros past out, nb and in) into the
// workspace, in 32-bit words: rows of nrs fp32 weights, or in bf16 of nrs / 2
// words that each hold two consecutive outputs' bf16 weights unchanged;
// narrow_dx_kernel stages 8 features of it at a time in LDS (two stages, one
// barrier per chunk).  Each lane owns one batch row with its dy in registers;
// the four waves of a 64-row workgroup take two features of every chunk each.
// dx has no sum over features, so the chunks can be split over blockIdx.y
// (cpg chunks per workgroup) to give the CUs more waves, as far as they all
// fit at once (a second, partial round of workgroups costs more than the
// waves gain: 784 -> 16 at batch 65536).
// In bf16 each t_c is a chain of two-term dot products (v_dot2_f32_bf16) of
// dy and weight pairs: both are bf16 inputs, so the products are exact and
// only the fp32 sums round, as with fp32 FMAs; it halves the VALU
// instructions and LDS bytes of the sums.  dx goes through LDS and out as one
// row's 8 consecutive features per thread.
constexpr int kNdxRows = 64;
constexpr int kNdxFeat = 8;

template <typename T>
__global__ __launch_bounds__(256) void narrow_dx_table_kernel(const T* __restrict__ coef,
                                                              const T* __restrict__ bw,
                                                              uint32_t* __restrict__ tab, int in,
                                                              int nfeat, int out, int nb, int ncw,
                                                              int nrs) {
    constexpr int PW = sizeof(T) == 2 ? 2 : 1;  // outputs per word
    const int rw = nrs / PW;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= (int64_t)nfeat * ncw * rw) return;
    const int p = (int)(u % rw);
    const int64_t r = u / rw;
    const int c = (int)(r % ncw);
    const int f = (int)(r / ncw);
    uint32_t v = 0;
#pragma unroll
    for (int e = 0; e < PW; ++e) {
        const int o = PW * p + e;
        T w = T(0);
        if (f < in && o < out) {
            if (c == 0) w = bw[(int64_t)o * in + f];
            else if (c <= nb) w = coef[((int64_t)o * in + f) * nb + (c - 1)];
        }
        if constexpr (PW == 2)
            v |= (uint32_t)w << (16 * e);
        else
            v = __float_as_uint(w);
    }
    tab[u] = v;
}

template <typename T>
struct NdxArgs {
    const T* xt;       // x transposed: [in][bpad]
    int64_t bpad;
    const T* dy;       // [batch][out]
    const uint32_t* tab;  // [nfeat][ncw][row words] (narrow_dx_table_kernel)
    T* dx;             // [batch][in]
    int64_t batch;
    int in, out, nb, ncw;
    int cpg;  // feature chunks per workgroup (blockIdx.y)
    float inv_h, inv_lo, xlim, a_int, a_frac;
};

// NO: outputs per lane (even, >= out); RS: outputs per table row; RW: its
// 32-bit words (even).
template <typename T, int NO>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
void narrow_dx_kernel(NdxArgs<T> a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int RS = (NO + 3) / 4 * 4;
    constexpr int RW = BF ? RS / 2 : RS;
    extern __shared__ floatx4 nds4[];
    float* stg0 = reinterpret_cast<float*>(nds4);  // table words (bf16: pairs)
    __shared__ float dxs[2][kNdxRows][kNdxFeat + 1];
    const int stage_floats = kNdxFeat * a.ncw * RW;  // a multiple of 4, at most 2048
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t row0 = (int64_t)blockIdx.x * kNdxRows;
    // rows past the batch read the last row (their dx is not stored)
    const int64_t rowc = row0 + lane < a.batch ? row0 + lane : a.batch - 1;
    float dyv[NO];
#pragma unroll
    for (int o = 0; o < NO; ++o) dyv[o] = o < a.out ? B<T>::ld(a.dy + rowc * a.out + o) : 0.0f;
    // bf16: dy of outputs 2 q, 2 q + 1 as one operand (exact: dy is bf16)
    bf16x2_t dyp[NO / 2];
#pragma unroll
    for (int q = 0; q < NO / 2; ++q) dyp[q] = bf16x2_t{(__bf16)dyv[2 * q], (__bf16)dyv[2 * q + 1]};
    const int c_begin = blockIdx.y * a.cpg;
    const int nchunks = min((a.in + kNdxFeat - 1) / kNdxFeat, c_begin + a.cpg);

    // the chunk's table rows are contiguous: at most two 16-byte units per thread
    const int n4 = stage_floats / 4;
    floatx4 wv[2];
    auto load_w = [&](int c) {
        const floatx4* src = reinterpret_cast<const floatx4*>(a.tab + (int64_t)c * stage_floats);
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int i = tid + 256 * m;
            wv[m] = i < n4 ? src[i] : floatx4{0.0f, 0.0f, 0.0f, 0.0f};
        }
    };
    auto store_w = [&](int st) {
        floatx4* d = reinterpret_cast<floatx4*>(stg0 + st * stage_floats);
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int i = tid + 256 * m;
            if (i < n4) d[i] = wv[m];
        }
    };
    float xc[2], xn[2];
    auto load_x = [&](int c, float (&xv)[2]) {
        const int f0 = c * kNdxFeat + 2 * wave;
#pragma unroll
        for (int j = 0; j < 2; ++j)
            xv[j] = f0 + j < a.in ? B<T>::ld(a.xt + (int64_t)(f0 + j) * a.bpad + rowc) : 0.0f;
    };
    // sum over the outputs of dy times one table row
    auto tdot = [&](const float* r) -> float {
        float t = 0.0f;
        if constexpr (BF) {
            // (the words are read as bf16 pairs directly: with this compiler,
            // __builtin_bit_cast of element 1 of a two-float vector produced
            // element 0's bits)
            const bf16x2_t* rb = reinterpret_cast<const bf16x2_t*>(r);
#pragma unroll
            for (int q = 0; q < NO / 2; ++q)
                t = __builtin_amdgcn_fdot2_f32_bf16(dyp[q], rb[q], t, false);
            return t;
        }
#pragma unroll
        for (int q = 0; q < NO / 4; ++q) {
            const floatx4 w = reinterpret_cast<const floatx4*>(r)[q];
            t = __builtin_fmaf(dyv[4 * q], w[0], t);
            t = __builtin_fmaf(dyv[4 * q + 1], w[1], t);
            t = __builtin_fmaf(dyv[4 * q + 2], w[2], t);
            t = __builtin_fmaf(dyv[4 * q + 3], w[3], t);
        }
        if constexpr (NO % 4 != 0) {
            const floatx2 w = reinterpret_cast<const floatx2*>(r)[NO / 2 - 1];
            t = __builtin_fmaf(dyv[NO - 2], w[0], t);
            t = __builtin_fmaf(dyv[NO - 1], w[1], t);
        }
        return t;
    };
    const float nbf = (float)a.nb;
    // pairs of dx elements stored together: even rows of dx and an aligned base
    const bool pair_st = (a.in & 1) == 0 &&
                         reinterpret_cast<uintptr_t>(a.dx) % (2 * sizeof(T)) == 0;

    load_w(c_begin);
    load_x(c_begin, xc);
    store_w(c_begin & 1);
    __syncthreads();
    for (int c = c_begin; c < nchunks; ++c) {
        const bool more = c + 1 < nchunks;
        if (more) {
            load_w(c + 1);
            load_x(c + 1, xn);
        }
        const float* stg = stg0 + (c & 1) * stage_floats;
        // (bf16: the chunk's two features unrolled, so one's LDS reads overlap the
        // other's dot products: 256 -> 10 at 65536 rows 79 -> 76 us per dx call)
#pragma unroll (BF ? 2 : 1)
        for (int j = 0; j < 2; ++j) {
            const float xv = xc[j];
            const float sv = __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f) +
                             coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
            const float f1 = __builtin_amdgcn_fmed3f(__builtin_floorf(sv), 2.0f, nbf);
            const int c0 = min(max((int)f1 - 1, 1), a.nb - 1);
            const float d = sv - (f1 - 1.0f);  // v of column c0
            const float* tb = stg + (2 * wave + j) * a.ncw * RW;
            const float* tw = tb + c0 * RW;
            float sb = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) sb = __builtin_fmaf(dbasis(d - (float)k), tdot(tw + k * RW), sb);
            dxs[c & 1][lane][2 * wave + j] = __builtin_fmaf(tdot(tb), silu_deriv(xv), a.inv_h * sb);
        }
        if (more) store_w((c + 1) & 1);
        __syncthreads();
        // dx of chunk c: thread t stores features 2 (t % 4) and 2 (t % 4) + 1
        // of row row0 + t / 4 (four threads write a row's 8 features), as one
        // two-element store where the pair is whole and aligned
        {
            const int rl = tid >> 2;
            const int fl = 2 * (tid & 3);
            const int64_t row = row0 + rl;
            const int f = c * kNdxFeat + fl;
            if (row < a.batch && f < a.in) {
                T* dst = a.dx + row * a.in + f;
                const float v0 = dxs[c & 1][rl][fl], v1 = dxs[c & 1][rl][fl + 1];
                if (pair_st && f + 1 < a.in) {
                    B<T>::st2(dst, v0, v1);
                } else {
                    B<T>::st(dst, v0);
                    if (f + 1 < a.in) B<T>::st(dst + 1, v1);
                }
            }
        }
        if (more) {
            xc[0] = xn[0];
            xc[1] = xn[1];
        }
    }
}

template <typename T, int NO>
hipError_t launch_ndx_no(const BwdGeom& g, const NdxArgs<T>& d0, hipStream_t s) {
    // (bf16 table words hold two outputs)
    const size_t lds = (size_t)2 * kNdxFeat * g.ncw * g.nrs * (sizeof(T) == 2 ? 2 : 4);
    const int64_t blocks = (d0.batch + kNdxRows - 1) / kNdxRows;
    // Feature groups: as many as keep every workgroup resident at once on the
    // 256 CUs: at most eight per CU (eight waves per SIMD, as these kernels
    // take at most 64 VGPRs) and as many as the CU's 160 KB of LDS holds.
    const int64_t lds_wg = (int64_t)lds + 2 * kNdxRows * (kNdxFeat + 1) * (int64_t)sizeof(float);
    const int64_t per_cu = std::min<int64_t>(8, (160 * 1024) / lds_wg);
    const int64_t nch = (d0.in + kNdxFeat - 1) / kNdxFeat;
    const int64_t fg = std::max<int64_t>(1, std::min<int64_t>(nch, 256 * per_cu / blocks));
    NdxArgs<T> d = d0;
    d.cpg = (int)((nch + fg - 1) / fg);
    const unsigned groups = (unsigned)((nch + d.cpg - 1) / d.cpg);
    hipLaunchKernelGGL((narrow_dx_kernel<T, NO>), dim3((unsigned)blocks, groups), dim3(256), lds, s,
                       d);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_narrow_dx(const BwdGeom& g, const NdxArgs<T>& d, hipStream_t s) {
    const int no = (d.out + 1) & ~1;
    if (g.nrs != (no + 3) / 4 * 4) return hipErrorInvalidValue;
    switch (no) {
        case 2: return launch_ndx_no<T, 2>(g, d, s);
        case 4: return launch_ndx_no<T, 4>(g, d, s);
        case 6: return launch_ndx_no<T, 6>(g, d, s);
        case 8: return launch_ndx_no<T, 8>(g, d, s);
        case 10: return launch_ndx_no<T, 10>(g, d, s);
        case 12: return launch_ndx_no<T, 12>(g, d, s);
        case 14: return launch_ndx_no<T, 14>(g, d, s);
        case 16: return launch_ndx_no<T, 16>(g, d, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t backward_t(const BwdGeom& g, const BwdArgs& a, hipStream_t s) {
    char* ws = static_cast<char*>(a.ws);
    const T* x = static_cast<const T*>(a.x);
    hipError_t e = hipSuccess;
    T* xt = reinterpret_cast<T*>(ws + g.off_xt);
    if (a.batch > 0) {
        // x transposed for both kernels (natural row order), dy for dW.  bf16
        // x in 64 x 64 tiles with 16-byte accesses (65536 x 784: 50 us against
        // 95 in 32 x 32 tiles of element accesses); fp32 x in 32 x 32 tiles,
        // whose rows are already 128 bytes (103 us against 130 in 64 x 64
        // tiles, whose LDS columns conflict)
        if constexpr (sizeof(T) == 2) {
            const int drows = (a.in + 31) / 32 * 32;
            const bool vec = reinterpret_cast<uintptr_t>(x) % 16 == 0 && a.in % 8 == 0;
            hipLaunchKernelGGL(transpose64_kernel<T>,
                               dim3((unsigned)((g.bpad + 63) / 64), (unsigned)((drows + 63) / 64)),
                               dim3(256), 0, s, x, xt, a.batch, a.in, g.bpad, drows, vec);
        } else {
            hipLaunchKernelGGL((transpose_kernel<T, false>),
                               dim3((unsigned)(g.bpad / 32), (unsigned)((a.in + 31) / 32)),
                               dim3(256), 0, s, x, xt, a.batch, a.in, g.bpad);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.dx != nullptr && a.batch > 0 && g.nx) {
        uint32_t* tab = reinterpret_cast<uint32_t*>(ws + g.off_wt);
        const int64_t n = (int64_t)g.nfeat * g.ncw * g.nrs / (sizeof(T) == 2 ? 2 : 1);
        hipLaunchKernelGGL(narrow_dx_table_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256),
                           0, s, static_cast<const T*>(a.coef), static_cast<const T*>(a.bw), tab,
                           a.in, g.nfeat, a.out, g.nb, g.ncw, g.nrs);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        NdxArgs<T> d;
        d.xt = xt;
        d.bpad = g.bpad;
        d.dy = static_cast<const T*>(a.dy);
        d.tab = tab;
        d.dx = static_cast<T*>(a.dx);
        d.batch = a.batch;
        d.in = a.in;
        d.out = a.out;
        d.nb = g.nb;
        d.ncw = g.ncw;
        d.cpg = 1;  // (set at launch)
        d.inv_h = a.inv_h;
        d.inv_lo = a.inv_lo;
        d.xlim = a.xlim;
        d.a_int = a.a_int;
        d.a_frac = a.a_frac;
        if ((e = launch_narrow_dx<T>(g, d, s)) != hipSuccess) return e;
    } else if (a.dx != nullptr && a.batch > 0) {
        T* wtp = reinterpret_cast<T*>(ws + g.off_wt);
        const int64_t units = (int64_t)g.ntiles * g.groups * 64;
        hipLaunchKernelGGL(pack_dx_kernel<T>, dim3((unsigned)((units + 255) / 256)), dim3(256), 0,
                           s, static_cast<const T*>(a.coef), static_cast<const T*>(a.bw), wtp,
                           a.in, a.out, g.nb, g.cp, g.groups, units);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        DxArgs<T> d;
        d.xt = xt;
        d.bpad = g.bpad;
        d.dy = static_cast<const T*>(a.dy);
        d.wtp = reinterpret_cast<const u32x4*>(wtp);
        d.dx = static_cast<T*>(a.dx);
        d.dxp = g.nchunk > 1 ? reinterpret_cast<float*>(ws + g.off_dxp) : nullptr;
        d.batch = a.batch;
        d.in = a.in;
        d.out = a.out;
        d.nb = g.nb;
        d.cp = g.cp;
        d.ntiles = g.ntiles;
        d.groups = g.groups;
        d.gmax = g.gmax;
        d.tiles_per_split = g.dx_tiles_per_split;
        d.inv_h = a.inv_h;
        d.inv_lo = a.inv_lo;
        d.xlim = a.xlim;
        d.a_int = a.a_int;
        d.a_frac = a.a_frac;
        if ((e = launch_dx<T>(g, d, s)) != hipSuccess) return e;
        if (g.nchunk > 1) {
            const int64_t n = a.batch * a.in;
            hipLaunchKernelGGL(dx_reduce_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256),
                               0, s, d.dxp, d.dx, n, g.nchunk);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    if (a.dcoef != nullptr) {
        float* P = reinterpret_cast<float*>(ws + g.off_p);
        int split = 0;
        if (a.batch > 0) {
            T* dyt = reinterpret_cast<T*>(ws + g.off_dyt);
            if constexpr (sizeof(T) == 2) {
                const bool vec = reinterpret_cast<uintptr_t>(a.dy) % 16 == 0 && a.out % 8 == 0;
                hipLaunchKernelGGL(transpose64_kernel<T>,
                                   dim3((unsigned)((g.bpad + 63) / 64),
                                        (unsigned)((g.out32 + 63) / 64)),
                                   dim3(256), 0, s, static_cast<const T*>(a.dy), dyt, a.batch,
                                   a.out, g.bpad, g.out32, vec);
            } else {
                hipLaunchKernelGGL((transpose_kernel<T, true>),
                                   dim3((unsigned)(g.bpad / 32), (unsigned)(g.out32 / 32)),
                                   dim3(256), 0, s, static_cast<const T*>(a.dy), dyt, a.batch,
                                   a.out, g.bpad);
            }
            if ((e = hipGetLastError()) != hipSuccess) return e;
            DwArgs<T> d;
            d.xt = xt;
            d.dyt = dyt;
            d.P = P;
            d.batch = a.batch;
            d.bpad = g.bpad;
            d.in = a.in;
            d.out32 = g.out32;
            d.nb = g.nb;
            d.cp = g.cp;
            d.kr = g.kr;
            d.rows_per_split = g.rows_per_split;
            d.inv_h = a.inv_h;
            d.inv_lo = a.inv_lo;
            d.xlim = a.xlim;
            d.a_int = a.a_int;
            d.a_frac = a.a_frac;
            if ((e = launch_dw<T>(g, d, s)) != hipSuccess) return e;
            split = g.split;
        }
        const int64_t n = (int64_t)a.out * a.in * (g.nb + 1);
        hipLaunchKernelGGL(dw_reduce_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                           P, static_cast<T*>(a.dcoef), static_cast<T*>(a.dbw), split, a.out,
                           g.out32, a.in, g.nb, g.cp, g.kr);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return e;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

bool bwd_geom(int nb, bool bf16, int64_t batch, int in, int out, BwdGeom* g) {
    g->nb = nb;
    g->cp = nb + 1 <= 16 ? 16 : 32 * ((nb + 1 + 31) / 32);
    const int64_t ntiles = g->cp == 16 ? ((int64_t)in + 1) / 2 : (int64_t)in * (g->cp / 32);
    if (ntiles * 32 > 0x7fffffffLL / 4) return false;
    g->ntiles = (int)ntiles;
    g->kr = (int)(32 * ntiles);
    g->out32 = (out + 31) / 32 * 32;
    const int go = bf16 ? 16 : 8;
    g->groups = (out + go - 1) / go;
    g->gmax = 256 / go;
    g->nchunk = (g->groups + g->gmax - 1) / g->gmax;
    if (g->out32 <= 32) { g->oh = 1; g->nfw = 1; }
    else if (g->out32 <= 64) { g->oh = 2; g->nfw = 1; }
    else if (g->out32 <= 128) { g->oh = 2; g->nfw = 2; }
    else { g->oh = 2; g->nfw = 4; }
    g->kt = 256;
    g->ktiles = (g->kr + g->kt - 1) / g->kt;
    const int ot = g->oh * g->nfw * 32;
    g->otiles = (g->out32 + ot - 1) / ot;
    if (g->otiles > 65535) return false;
    // dx: two 32-row tiles per wave while their dy registers stay within 64
    // (up to 8 k-step groups: 128 outputs bf16, 64 fp32), and the K tiles split over
    // workgroups (whole features each) until the grid fills the chip
    g->dx_rf = (g->groups < g->gmax ? g->groups : g->gmax) <= 8 ? 2 : 1;
    {
        const int tpf = g->cp == 16 ? 1 : g->cp / 32;
        g->dx_bm = 32 * g->dx_rf * 8;  // rows per workgroup (eight waves)
        const int64_t rblocks = (batch + g->dx_bm - 1) / g->dx_bm;
        int64_t ks = rblocks * g->nchunk >= 256 ? 1 : (256 + rblocks * g->nchunk - 1) /
                                                     (rblocks * g->nchunk > 0 ? rblocks * g->nchunk : 1);
        const int64_t nfe = g->ntiles / tpf;  // features' tile groups
        if (ks > nfe) ks = nfe > 0 ? nfe : 1;
        if (ks < 1) ks = 1;
        int64_t tps = (g->ntiles + ks - 1) / ks;
        tps = (tps + tpf - 1) / tpf * tpf;
        g->dx_tiles_per_split = (int)tps;
        g->dx_ksplit = (int)((g->ntiles + tps - 1) / tps);
        if (g->dx_ksplit > 65535 || rblocks > 0x7fffffffLL) return false;
    }
    g->bpad = (batch + 31) / 32 * 32;
    const int64_t nck = g->bpad / 32;
    // Batch splits of the weight gradient: towards 256 workgroups, in bf16
    // towards 512 while the splits' fp32 partial sums stay within 16 MB (the
    // 256 -> 10 layer at batch 65536: 30 splits, 121 -> 105 us; the wide
    // layers keep theirs; fp32 256 -> 10 with 30 splits: 3% slower)
    int64_t split = (bf16 ? 512 : 256) / ((int64_t)g->ktiles * g->otiles);
    if (split < 1) split = 1;
    while (split > 1 && split * g->ktiles * g->otiles > 256 &&
           split * g->out32 * (int64_t)g->kr * 4 > ((int64_t)16 << 20))
        --split;
    if (split > nck) split = nck > 0 ? nck : 1;
    const int64_t rps_chunks = nck > 0 ? (nck + split - 1) / split : 1;
    if (rps_chunks * 32 > 0x7fffffffLL) return false;
    g->rows_per_split = (int)(rps_chunks * 32);
    g->split = nck > 0 ? (int)((nck + rps_chunks - 1) / rps_chunks) : 0;
    if (g->split > 65535 || (batch + 255) / 256 > 0x7fffffffLL) return false;
    // dx of narrow layers (at most 16 outputs, from 16384 rows) on the vector
    // ALUs, with its weight table (fp32 weights, or bf16 weights in pairs) in
    // the place of the packed weights
    g->ncw = (nb + 4) & ~1;
    g->nrs = (((out + 1) & ~1) + 3) / 4 * 4;
    g->nfeat = (in + 7) / 8 * 8;
    g->nx = out <= 16 && g->ncw * g->nrs <= 256 && batch >= 16384;
    const size_t es = bf16 ? 2 : 4;
    size_t off = 0;
    g->off_wt = off;
    size_t wt_bytes = (size_t)g->ntiles * g->groups * 1024;
    if (g->nx) wt_bytes = std::max(wt_bytes, (size_t)g->nfeat * g->ncw * g->nrs * es);
    off = align256(off + wt_bytes);
    g->off_dyt = off;
    off = align256(off + (size_t)g->out32 * (size_t)g->bpad * es);
    g->off_xt = off;
    off = align256(off + (size_t)((in + 31) / 32 * 32) * (size_t)g->bpad * es);
    g->off_p = off;
    off = align256(off + (size_t)(g->split > 0 ? g->split : 1) * g->out32 * (size_t)g->kr * 4);
    g->off_dxp = off;
    if (g->nchunk > 1) off = align256(off + (size_t)g->nchunk * (size_t)batch * in * 4);
    g->bytes = off;
    return true;
}

hipError_t launch_backward(bool bf16, const BwdGeom& g, const BwdArgs& a, hipStream_t s) {
    return bf16 ? backward_t<uint16_t>(g, a, s) : backward_t<float>(g, a, s);
}

}  // namespace kan
