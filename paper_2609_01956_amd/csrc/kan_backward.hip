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
    static constexpr int E = 4;   // elements per 16-byte unit
};
template <> struct B<uint16_t> {
    static __device__ __forceinline__ float ld(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void st(uint16_t* p, float v) { *p = f32_to_bf16(v); }
    static constexpr int E = 8;
};

// Local K row of A-operand row i of a 32-row dx tile: rows with (i / 4) % 2 == h
// land in lane half h of the accumulators, as local rows 16 h .. 16 h + 15.
__host__ __device__ constexpr int dx_local_row(int i) {
    return 16 * ((i / 4) % 2) + 4 * (i / 8) + i % 4;
}

// ------------------------------------------------------------ dy transpose

// dyt[o][pos(b)] = dy[b][o], zero-padded to out32 rows and bpad columns.  fp32
// keeps each 32-row chunk of the batch as its even rows then its odd rows
// (position 16 (b % 2) + b / 2 in the chunk): a 32x32x2 k-step takes rows 2 j
// and 2 j + 1 in its two lane halves, so a lane's rows of a chunk are then
// consecutive.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ dy,
                                                        T* __restrict__ dyt, int64_t batch,
                                                        int out, int64_t bpad) {
    __shared__ T tile[32][33];
    const int64_t b0 = (int64_t)blockIdx.x * 32;
    const int o0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 8 rows of 32
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int bl = ty + 8 * k;
        const int64_t b = b0 + bl;
        const int o = o0 + tx;
        tile[bl][tx] = (b < batch && o < out) ? dy[b * out + o] : T(0);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int ol = ty + 8 * k;
        const int bl = tx;
        const int pos = sizeof(T) == 4 ? 16 * (bl & 1) + (bl >> 1) : bl;
        dyt[(int64_t)(o0 + ol) * bpad + b0 + pos] = tile[bl][ol];
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
    const T* x;
    const T* dy;
    const u32x4* wtp;  // packed weights, 16-byte units
    T* dx;
    float* dxp;        // per-chunk partials when the outputs take several chunks
    int64_t batch;
    int in, out, nb, cp, ntiles, groups, gmax;
    float inv_h, a_int, a_frac;
};

// One workgroup: 256 batch rows (eight waves of 32) against every K tile, for
// output chunk blockIdx.y (up to gmax k-step groups, 256 outputs).  SM is
// the compile-time bound on the groups of a chunk.
template <typename T, int SM>
__global__ __launch_bounds__(kThreads) void dx_kernel(DxArgs<T> a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int UPT = (SM * 64 + kThreads - 1) / kThreads;  // 16-byte units per thread per tile
    __shared__ u32x4 lds[2][SM * 64];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, r = lane & 31, h = lane >> 5;
    const int64_t row = (int64_t)blockIdx.x * 256 + wave * 32 + r;
    const int64_t rowc = row < a.batch ? row : a.batch - 1;
    const int ch = blockIdx.y;
    const int g0 = ch * a.gmax;
    const int S = min(a.gmax, a.groups - g0);

    // B operand: the lane's batch row of dy for every k-step group of the chunk
    u32x4 dyr[SM];
    const T* dyrow = a.dy + rowc * a.out;
#pragma unroll
    for (int s = 0; s < SM; ++s) {
        float v[B<T>::E];
#pragma unroll
        for (int e = 0; e < B<T>::E; ++e) {
            const int o = BF ? (g0 + s) * 16 + 8 * h + e : (g0 + s) * 8 + 2 * e + h;
            v[e] = (s < S && o < a.out) ? B<T>::ld(dyrow + o) : 0.0f;
        }
        if constexpr (BF)
            dyr[s] = u32x4{pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]), pack2_bf16(v[4], v[5]),
                           pack2_bf16(v[6], v[7])};
        else
            dyr[s] = u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                           __float_as_uint(v[3])};
    }

    u32x4 stg[UPT];
    auto load_tile = [&](int t) {
        const u32x4* src = a.wtp + ((int64_t)t * a.groups + g0) * 64;
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + k * kThreads;
            if (u < S * 64) stg[k] = src[u];
        }
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + k * kThreads;
            if (u < S * 64) lds[buf][u] = stg[k];
        }
    };

    load_tile(0);
    store_tile(0);
    __syncthreads();

    const int tpf = a.cp / 32;  // tiles per feature (cp >= 32)
    float dxacc = 0.0f;
    for (int t = 0; t < a.ntiles; ++t) {
        if (t + 1 < a.ntiles) load_tile(t + 1);
        const int R0 = 32 * t + 16 * h;
        const int f = R0 / a.cp;
        const int c0 = R0 - f * a.cp;
        const float xv = f < a.in ? B<T>::ld(a.x + rowc * a.in + f) : 0.0f;

        floatx16 acc;
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[q] = 0.0f;
        const u32x4* st = lds[t & 1];
#pragma unroll
        for (int s = 0; s < SM; ++s) {
            if (s < S) {
                const u32x4 w = st[s * 64 + lane];
                if constexpr (BF) {
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, w), __builtin_bit_cast(bf16x8, dyr[s]), acc, 0,
                        0, 0);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            __uint_as_float(w[j]), __uint_as_float(dyr[s][j]), acc, 0, 0, 0);
                }
            }
        }

        // acc[q] = Gm[row][feature f, column c0 + q].  v of column c0 in one
        // rounding at the magnitude of the group's own coordinates (the
        // column offset is folded into the fma's exact integer addend), then
        // v - q exactly where the derivative is nonzero.
        const float s0 = __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f - (float)c0) + a.a_frac;
        float sb = 0.0f;
#pragma unroll
        for (int q = 1; q < 16; ++q) sb = __builtin_fmaf(acc[q], dbasis(s0 - (float)q), sb);
        const float d0 = c0 == 0 ? silu_deriv(xv) : a.inv_h * dbasis(s0);
        const float sum = __builtin_fmaf(acc[0], d0, a.inv_h * sb);
        auto put = [&](float v) {
            if (row < a.batch && f < a.in) {
                if (a.dxp != nullptr)
                    a.dxp[((int64_t)ch * a.batch + row) * a.in + f] = v;
                else
                    B<T>::st(a.dx + row * a.in + f, v);
            }
        };
        if (a.cp == 16) {
            put(sum);
        } else {
            dxacc += sum;
            if ((t + 1) % tpf == 0) {  // the feature's last tile: add the two lane halves
                const float tot = dxacc + __shfl_xor(dxacc, 32);
                if (h == 0) put(tot);
                dxacc = 0.0f;
            }
        }

        if (t + 1 < a.ntiles) store_tile((t + 1) & 1);
        __syncthreads();
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
    const T* x;
    const T* dyt;   // [out32][bpad]
    float* P;       // [split][out32][kr] partial sums of dW^T / 2
    int64_t batch, bpad;
    int in, out32, nb, cp, kr, rows_per_split;
    float inv_h, a_int, a_frac;
};

// Workgroup: K rows [kt0, kt0 + KT) x outputs [ot0, ot0 + OT) over the batch
// rows of split blockIdx.y.  Wave (kg, oh) holds two 32-row K tiles (RF = 2)
// by NFW 32-output fragments, so every B fragment read from LDS feeds two
// MFMAs and every generated A element NFW.  Per chunk of 32 batch rows the
// workgroup stages the transposed dy of its outputs (plain copies of
// contiguous runs) and x / silu(x) / 2 of its features (fp32, transposed to
// batch-fastest) in LDS, double-buffered; each lane generates its A rows'
// values N_c(x) / 2 (or silu / 2) at its batch rows.
template <typename T, int OH, int NFW>
__global__ __launch_bounds__(kThreads) void dw_kernel(DwArgs<T> a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int RF = 2;
    constexpr int KG = 8 / OH;
    constexpr int KT = KG * RF * 32;
    constexpr int OT = OH * NFW * 32;
    constexpr int NFEAT = KT / 16 + 2;          // features a workgroup's K rows touch, at most
    constexpr int UR = BF ? 4 : 8;              // 16-byte units of a chunk's dy run per output
    constexpr int ROWU = UR + 1;                // LDS row stride in units (one unit of padding)
    constexpr int DU = (OT * UR + kThreads - 1) / kThreads;    // dy units per thread
    constexpr int XU = (32 * NFEAT + kThreads - 1) / kThreads;  // x values per thread
    __shared__ u32x4 dys[2][OT * ROWU];
    __shared__ __attribute__((aligned(16))) float xs[2][NFEAT][32];
    __shared__ __attribute__((aligned(16))) float ss[2][NFEAT][32];
    // features with a NaN input in this workgroup's rows: their basis
    // gradients are NaN (N_j(NaN) is NaN; the clamp in half_basis would
    // otherwise swallow it)
    __shared__ int nanf[NFEAT];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, r = lane & 31, h = lane >> 5;
    const int kg = wave / OH, oh = wave % OH;
    for (int i = tid; i < NFEAT; i += kThreads) nanf[i] = 0;
    __syncthreads();
    const int kt0 = blockIdx.x * KT;
    const int ot0 = blockIdx.z * OT;
    const int F0 = kt0 / a.cp;
    const int F1 = min((kt0 + KT - 1) / a.cp, (a.kr - 1) / a.cp);
    const int nfeat = F1 - F0 + 1;
    const int64_t b_begin = (int64_t)blockIdx.y * a.rows_per_split;
    const int64_t b_end = min(b_begin + a.rows_per_split, a.bpad);
    const int nchunks = (int)((b_end - b_begin) / 32);

    // the lane's A rows: K row R = kt0 + 32 (kg RF + rt) + r
    int fl[RF];
    float cj[RF];
    bool sil[RF];
#pragma unroll
    for (int rt = 0; rt < RF; ++rt) {
        const int R = kt0 + 32 * (kg * RF + rt) + r;
        const int f = R / a.cp;
        const int c = R - f * a.cp;
        fl[rt] = min(max(f - F0, 0), NFEAT - 1);
        cj[rt] = a.a_int + 1.0f - (float)c;
        sil[rt] = c == 0;
    }

    u32x4 dreg[DU];
    float xreg[XU];
    auto load_chunk = [&](int64_t b0) {
#pragma unroll
        for (int k = 0; k < DU; ++k) {
            const int u = tid + k * kThreads;
            const int o = u / UR, w = u % UR;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (u < OT * UR && ot0 + o < a.out32)
                v = *reinterpret_cast<const u32x4*>(
                    reinterpret_cast<const char*>(a.dyt + (int64_t)(ot0 + o) * a.bpad + b0) +
                    16 * w);
            dreg[k] = v;
        }
#pragma unroll
        for (int k = 0; k < XU; ++k) {
            const int idx = tid + k * kThreads;
            float v = 0.0f;
            if (idx < 32 * nfeat) {
                const int bl = idx / nfeat, f = F0 + idx % nfeat;
                const int64_t b = b0 + bl;
                if (b < a.batch && f < a.in) v = B<T>::ld(a.x + b * a.in + f);
            }
            xreg[k] = v;
        }
    };
    auto store_chunk = [&](int buf) {
#pragma unroll
        for (int k = 0; k < DU; ++k) {
            const int u = tid + k * kThreads;
            if (u < OT * UR) dys[buf][(u / UR) * ROWU + u % UR] = dreg[k];
        }
#pragma unroll
        for (int k = 0; k < XU; ++k) {
            const int idx = tid + k * kThreads;
            if (idx < 32 * nfeat) {
                const int bl = idx / nfeat, f = idx % nfeat;
                const int pos = BF ? bl : 16 * (bl & 1) + (bl >> 1);
                xs[buf][f][pos] = xreg[k];
                ss[buf][f][pos] = half_silu_b(xreg[k]);
                if (xreg[k] != xreg[k]) nanf[f] = 1;
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

    if (nchunks > 0) {
        load_chunk(b_begin);
        store_chunk(0);
    }
    __syncthreads();
    for (int ck = 0; ck < nchunks; ++ck) {
        const int buf = ck & 1;
        if (ck + 1 < nchunks) load_chunk(b_begin + 32 * (int64_t)(ck + 1));
        const char* dl = reinterpret_cast<const char*>(dys[buf]);
        if constexpr (BF) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {  // k-steps of 16 batch rows
                bf16x8 A[RF];
#pragma unroll
                for (int rt = 0; rt < RF; ++rt) {
                    const floatx4* xp = reinterpret_cast<const floatx4*>(&xs[buf][fl[rt]][16 * s + 8 * h]);
                    const floatx4* sp = reinterpret_cast<const floatx4*>(&ss[buf][fl[rt]][16 * s + 8 * h]);
                    float v[8];
#pragma unroll
                    for (int m = 0; m < 2; ++m) {
                        const floatx4 xv = xp[m], sv = sp[m];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float bv = half_basis(
                                __builtin_fmaf(xv[e], a.inv_h, cj[rt]) + a.a_frac);
                            v[4 * m + e] = sil[rt] ? sv[e] : bv;
                        }
                    }
                    A[rt] = __builtin_bit_cast(
                        bf16x8, u32x4{pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]),
                                      pack2_bf16(v[4], v[5]), pack2_bf16(v[6], v[7])});
                }
#pragma unroll
                for (int nf = 0; nf < NFW; ++nf) {
                    const int o = (oh * NFW + nf) * 32 + r;
                    const bf16x8 Bv = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u32x4*>(dl + (o * ROWU) * 16 + 32 * s + 16 * h));
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
                    const floatx4 xv = *reinterpret_cast<const floatx4*>(&xs[buf][fl[rt]][16 * h + 4 * jg]);
                    const floatx4 sv = *reinterpret_cast<const floatx4*>(&ss[buf][fl[rt]][16 * h + 4 * jg]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float bv = half_basis(__builtin_fmaf(xv[e], a.inv_h, cj[rt]) + a.a_frac);
                        A[rt][e] = sil[rt] ? sv[e] : bv;
                    }
                }
#pragma unroll
                for (int nf = 0; nf < NFW; ++nf) {
                    const int o = (oh * NFW + nf) * 32 + r;
                    const floatx4 Bv = *reinterpret_cast<const floatx4*>(
                        dl + (o * ROWU) * 16 + 64 * h + 16 * jg);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int rt = 0; rt < RF; ++rt)
                            acc[rt][nf] = __builtin_amdgcn_mfma_f32_32x32x2f32(A[rt][e], Bv[e],
                                                                              acc[rt][nf], 0, 0, 0);
                }
            }
        }
        if (ck + 1 < nchunks) store_chunk(buf ^ 1);
        __syncthreads();
    }

    // acc[rt][nf][q] = (dW^T / 2)[K row kt0 + 32 (kg RF + rt) + 8 (q / 4) + 4 h + q % 4][output o]
    // (the lane's A row of tile rt is K row kt0 + 32 (kg RF + rt) + r, but the
    // accumulator rows are the output rows above: their features are looked
    // up for the NaN flags)
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

template <typename T, int SM>
hipError_t launch_dx_sm(const BwdGeom& g, const DxArgs<T>& d, hipStream_t s) {
    const dim3 grid((unsigned)((d.batch + 255) / 256), (unsigned)g.nchunk);
    hipLaunchKernelGGL((dx_kernel<T, SM>), grid, dim3(kThreads), 0, s, d);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_dx(const BwdGeom& g, const DxArgs<T>& d, hipStream_t s) {
    const int sm = min(g.groups, g.gmax);  // groups of the largest chunk
    if (sm <= 1) return launch_dx_sm<T, 1>(g, d, s);
    if (sm <= 2) return launch_dx_sm<T, 2>(g, d, s);
    if (sm <= 4) return launch_dx_sm<T, 4>(g, d, s);
    if (sm <= 8) return launch_dx_sm<T, 8>(g, d, s);
    if (sm <= 16) return launch_dx_sm<T, 16>(g, d, s);
    if constexpr (sizeof(T) == 4) {
        if (sm <= 32) return launch_dx_sm<T, 32>(g, d, s);
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

template <typename T>
hipError_t backward_t(const BwdGeom& g, const BwdArgs& a, hipStream_t s) {
    char* ws = static_cast<char*>(a.ws);
    const T* x = static_cast<const T*>(a.x);
    hipError_t e = hipSuccess;
    if (a.dx != nullptr && a.batch > 0) {
        T* wtp = reinterpret_cast<T*>(ws + g.off_wt);
        const int64_t units = (int64_t)g.ntiles * g.groups * 64;
        hipLaunchKernelGGL(pack_dx_kernel<T>, dim3((unsigned)((units + 255) / 256)), dim3(256), 0,
                           s, static_cast<const T*>(a.coef), static_cast<const T*>(a.bw), wtp,
                           a.in, a.out, g.nb, g.cp, g.groups, units);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        DxArgs<T> d;
        d.x = x;
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
        d.inv_h = a.inv_h;
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
            hipLaunchKernelGGL(transpose_kernel<T>, dim3((unsigned)(g.bpad / 32),
                                                         (unsigned)(g.out32 / 32)),
                               dim3(256), 0, s, static_cast<const T*>(a.dy), dyt, a.batch, a.out,
                               g.bpad);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            DwArgs<T> d;
            d.x = x;
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
    g->kt = (8 / g->oh) * 2 * 32;
    g->ktiles = (g->kr + g->kt - 1) / g->kt;
    const int ot = g->oh * g->nfw * 32;
    g->otiles = (g->out32 + ot - 1) / ot;
    if (g->otiles > 65535) return false;
    g->bpad = (batch + 31) / 32 * 32;
    const int64_t nck = g->bpad / 32;
    int64_t split = 256 / ((int64_t)g->ktiles * g->otiles);
    if (split < 1) split = 1;
    if (split > nck) split = nck > 0 ? nck : 1;
    const int64_t rps_chunks = nck > 0 ? (nck + split - 1) / split : 1;
    if (rps_chunks * 32 > 0x7fffffffLL) return false;
    g->rows_per_split = (int)(rps_chunks * 32);
    g->split = nck > 0 ? (int)((nck + rps_chunks - 1) / rps_chunks) : 0;
    if (g->split > 65535 || (batch + 255) / 256 > 0x7fffffffLL) return false;
    const size_t es = bf16 ? 2 : 4;
    size_t off = 0;
    g->off_wt = off;
    off = align256(off + (size_t)g->ntiles * g->groups * 1024);
    g->off_dyt = off;
    off = align256(off + (size_t)g->out32 * (size_t)g->bpad * es);
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
