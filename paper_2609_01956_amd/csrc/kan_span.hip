// kan_span.hip -- span-sparse KAN layer forward (eq. kan_forward restricted
// to the nonzero terms):
//
//   y[b, o] = sum_i ( silu(x[b, i]) Wb[o, i] + sum_{c in window(x[b, i])} N_{c-1}(x[b, i]) C[o, i, c-1] )
//
// The clamped basis is exactly 0 outside its support (eq. bounded), so of a
// feature's G + k basis columns only the k + 1 whose support holds x can be
// nonzero: with s the coordinate of the feature's column 0 (the SiLU
// column; column c holds basis c - 1 at v = s - c), they are the columns
// c_lo .. c_lo + k, c_lo = floor(s - (k + 1) / 2) + 1.  Each is still the
// closed clamped form at its own coordinate; the terms left out are exact
// zeros of the dense contraction, so the result is the dense one up to the
// fp32 summation order.  For large grids the dense contraction multiplies
// mostly zeros (G = 200: 4 of 203 bases); here the work per (row, feature)
// is (k + 2) rows of weights instead of G + k + 1.
//
// The window differs per row, so the contraction is a gather: each
// workgroup stages one feature's weights [column][its output tile] (fp32) in
// LDS, double-buffered, and every thread accumulates its rows' outputs on
// the vector ALUs from the (k + 2) weight rows its rows select.  Features
// are split over workgroups when the row blocks do not fill the chip; the
// partial sums are then added in a fixed order by a reduce kernel.
#include "kan_internal.h"

namespace kan {

namespace {

constexpr int kThreads = 256;
constexpr int64_t kSpanLdsBytes = 65536;  // both stages of a feature's weight tile
constexpr int64_t kSpanTargetWgs = 512;

template <typename T> struct S;
template <> struct S<float> {
    static __device__ __forceinline__ float ld(const float* p) { return *p; }
    static __device__ __forceinline__ float val(float v) { return v; }
    static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
};
template <> struct S<uint16_t> {
    static __device__ __forceinline__ float ld(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ float val(uint16_t v) { return bf16_to_f32(v); }
    static __device__ __forceinline__ void st(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// Transposed fp32 weights: wt[f][c][o] for o < outp (zero past `out`),
// c = 0 the SiLU weight, c = 1 .. nb the spline coefficients.  One workgroup
// moves a 64 x 64 tile (outputs x columns) of one feature through LDS, so the
// reads run along a coefficient row and the writes along the outputs.
template <typename T>
__global__ __launch_bounds__(256) void span_pack_kernel(const T* __restrict__ coef,
                                                        const T* __restrict__ bw,
                                                        float* __restrict__ wt, int in, int out,
                                                        int nb, int outp) {
    __shared__ float tile[64][65];
    const int f = blockIdx.x, o0 = blockIdx.y * 64, c0 = blockIdx.z * 64;
    const int ncol = nb + 1;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int idx = threadIdx.x + 256 * i;
        const int ol = idx / 64, cl = idx % 64;
        const int o = o0 + ol, c = c0 + cl;
        float v = 0.0f;
        if (o < out && c < ncol) {
            const int64_t row = (int64_t)o * in + f;
            v = c == 0 ? S<T>::ld(bw + row) : S<T>::ld(coef + row * nb + c - 1);
        }
        tile[ol][cl] = v;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int idx = threadIdx.x + 256 * i;
        const int cl = idx / 64, ol = idx % 64;
        const int o = o0 + ol, c = c0 + cl;
        if (o < outp && c < ncol) wt[((int64_t)f * ncol + c) * outp + o] = tile[ol][cl];
    }
}

// OPT outputs per thread, NG output groups (OT = OPT NG outputs per
// workgroup), NR rows per thread: thread (row lane rl, group og) holds rows
// rl + (256 / NG) r, r < NR, so a workgroup covers 256 NR / NG rows.  GD: a
// degree other than 3 (run-time form).
template <typename T, int OPT, int NG, int NR, bool GD>
__global__ __launch_bounds__(kThreads) void span_kernel(SpanArgs a) {
    constexpr int OT = OPT * NG;
    constexpr int RL = kThreads / NG;  // row lanes
    constexpr int RW = RL * NR;        // rows per workgroup
    extern __shared__ floatx4 wl4[];    // [2][ncol][cs] floats
    float* wl = reinterpret_cast<float*>(wl4);
    const int ncol = a.nb + 1;
    const int stage_f = ncol * a.cs;   // LDS floats per stage
    const int stage_u = ncol * OT / 4; // 16-byte units of the tile per stage
    const int csu = a.cs / 4;          // column stride in 16-byte units

    const int tid = threadIdx.x;
    const int og = tid % NG, rl = tid / NG;
    const int64_t rb0 = (int64_t)blockIdx.x * RW;
    const int f0 = blockIdx.y * a.fpf;
    const int f1 = min(f0 + a.fpf, a.in);
    const int ot0 = blockIdx.z * OT;
    const T* x = static_cast<const T*>(a.x);
    float* P = a.fs > 1 ? reinterpret_cast<float*>(static_cast<char*>(a.ws) + a.off_p) : nullptr;

    int64_t rowc[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int64_t row = rb0 + rl + RL * r;
        rowc[r] = row < a.batch ? row : a.batch - 1;
    }
    float acc[NR][OPT];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int o = 0; o < OPT; ++o) acc[r][o] = 0.0f;

    // staging of feature f's weight tile: unit u = (c, o / 4) of the tile
    auto stage_src = [&](int f, int u) -> const floatx4* {
        const int c = u / (OT / 4), oq = u % (OT / 4);
        return reinterpret_cast<const floatx4*>(a.wt + ((int64_t)f * ncol + c) * a.outp + ot0) + oq;
    };
    constexpr int MAXU = kSpanLdsBytes / 2 / 16 / kThreads;  // 16-byte units per thread per stage
    floatx4 reg[MAXU];
    const int upt = (stage_u + kThreads - 1) / kThreads;
    auto issue = [&](int f) {
        const int fc = min(f, f1 - 1);
#pragma unroll
        for (int k = 0; k < MAXU; ++k)
            if (k < upt) reg[k] = *stage_src(fc, min(tid + k * kThreads, stage_u - 1));
    };
    auto put = [&](int buf) {
#pragma unroll
        for (int k = 0; k < MAXU; ++k) {
            const int u = tid + k * kThreads;
            if (k < upt && u < stage_u)
                wl4[buf * (stage_f / 4) + (u / (OT / 4)) * csu + u % (OT / 4)] = reg[k];
        }
    };

    const float c0 = a.a_int + 1.0f;  // column 0 of a feature: s = x / h + c0 (+ lo term)
    const int kw = GD ? a.kdeg + 1 : 4;
    // x of the next feature's rows, loaded a feature ahead
    T xn[NR];
    auto issue_x = [&](int f) {
        const int fc = min(f, f1 - 1);
#pragma unroll
        for (int r = 0; r < NR; ++r) xn[r] = x[rowc[r] * a.in + fc];
    };
    issue(f0);
    issue_x(f0);
    put(0);
    __syncthreads();
    for (int f = f0; f < f1; ++f) {
        const int buf = (f - f0) & 1;
        float xf[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) xf[r] = S<T>::val(xn[r]);
        if (f + 1 < f1) {
            issue(f + 1);
            issue_x(f + 1);
        }
        const float* w = wl + buf * stage_f + og * OPT;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const float xv = xf[r];
            const float lot = coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
            const float s = __builtin_amdgcn_fmed3f(__builtin_fmaf(xv, a.inv_h, c0) + lot, -16.0f,
                                                   (float)(ncol + 16));
            const int clo = (int)__builtin_floorf(s - a.hw) + 1;
            // SiLU column
            {
                const float sl = silu(xv);
                const floatx4* wp = reinterpret_cast<const floatx4*>(w);
#pragma unroll
                for (int q = 0; q < OPT / 4; ++q) {
                    const floatx4 wv = wp[q];
                    acc[r][4 * q] = __builtin_fmaf(sl, wv[0], acc[r][4 * q]);
                    acc[r][4 * q + 1] = __builtin_fmaf(sl, wv[1], acc[r][4 * q + 1]);
                    acc[r][4 * q + 2] = __builtin_fmaf(sl, wv[2], acc[r][4 * q + 2]);
                    acc[r][4 * q + 3] = __builtin_fmaf(sl, wv[3], acc[r][4 * q + 3]);
                }
            }
            for (int m = 0; m < kw; ++m) {
                const int c = clo + m;
                if (c < 1 || c > a.nb) continue;
                // v of column c in one rounding at its own magnitude
                const float v = __builtin_fmaf(xv, a.inv_h, c0 - (float)c) + lot;
                float bv;
                if constexpr (GD) bv = 2.0f * half_basis_deg(v, a.kdeg, a.hw, a.hc);
                else bv = 2.0f * half_basis(v);
                const floatx4* wp = reinterpret_cast<const floatx4*>(w + c * a.cs);
#pragma unroll
                for (int q = 0; q < OPT / 4; ++q) {
                    const floatx4 wv = wp[q];
                    acc[r][4 * q] = __builtin_fmaf(bv, wv[0], acc[r][4 * q]);
                    acc[r][4 * q + 1] = __builtin_fmaf(bv, wv[1], acc[r][4 * q + 1]);
                    acc[r][4 * q + 2] = __builtin_fmaf(bv, wv[2], acc[r][4 * q + 2]);
                    acc[r][4 * q + 3] = __builtin_fmaf(bv, wv[3], acc[r][4 * q + 3]);
                }
            }
            // a NaN input: whatever window its clamped coordinate selects,
            // the SiLU term carries the NaN into every output of the row
        }
        if (f + 1 < f1) put(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int64_t row = rb0 + rl + RL * r;
        if (row >= a.batch) continue;
#pragma unroll
        for (int o = 0; o < OPT; ++o) {
            const int col = ot0 + og * OPT + o;
            if (col >= a.out) continue;
            if (P != nullptr)
                P[((int64_t)blockIdx.y * a.batch + row) * a.out + col] = acc[r][o];
            else
                S<T>::st(static_cast<T*>(a.y) + row * a.out + col, acc[r][o]);
        }
    }
}

template <typename T>
__global__ __launch_bounds__(256) void span_reduce_kernel(const float* __restrict__ P,
                                                          T* __restrict__ y, int64_t n, int fs) {
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= n) return;
    float s = 0.0f;
    for (int k = 0; k < fs; ++k) s += P[(int64_t)k * n + u];
    S<T>::st(y + u, s);
}

template <typename T, int OPT, int NG, int NR>
hipError_t launch_span_shape(const SpanGeom& g, const SpanArgs& a, hipStream_t s) {
    const dim3 grid((unsigned)g.rblocks, (unsigned)g.fs, (unsigned)g.otiles);
    const size_t lds = 2 * (size_t)(a.nb + 1) * a.cs * 4;
    if (a.kdeg == 3)
        hipLaunchKernelGGL((span_kernel<T, OPT, NG, NR, false>), grid, dim3(kThreads), lds, s, a);
    else
        hipLaunchKernelGGL((span_kernel<T, OPT, NG, NR, true>), grid, dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

template <typename T>
hipError_t span_t(const SpanGeom& g, SpanArgs a, const void* coef, const void* bw,
                  hipStream_t s) {
    char* ws = static_cast<char*>(a.ws);
    float* wt = reinterpret_cast<float*>(ws + g.off_w);
    const dim3 pgrid((unsigned)a.in, (unsigned)((g.outp + 63) / 64),
                     (unsigned)((a.nb + 1 + 63) / 64));
    hipLaunchKernelGGL(span_pack_kernel<T>, pgrid, dim3(256), 0, s, static_cast<const T*>(coef),
                       static_cast<const T*>(bw), wt, a.in, a.out, a.nb, g.outp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    a.wt = wt;
    a.outp = g.outp;
    a.fpf = g.fpf;
    a.fs = g.fs;
    a.off_p = g.off_p;
    a.cs = g.cs;
    if (g.opt == 16 && g.ng == 1 && g.nr == 2) e = launch_span_shape<T, 16, 1, 2>(g, a, s);
    else if (g.opt == 32 && g.ng == 1 && g.nr == 2) e = launch_span_shape<T, 32, 1, 2>(g, a, s);
    else e = hipErrorInvalidValue;
    if (e != hipSuccess || g.fs == 1) return e;
    const int64_t ny = a.batch * a.out;
    hipLaunchKernelGGL(span_reduce_kernel<T>, dim3((unsigned)((ny + 255) / 256)), dim3(256), 0, s,
                       reinterpret_cast<const float*>(ws + g.off_p), static_cast<T*>(a.y), ny,
                       g.fs);
    return hipGetLastError();
}

size_t align256s(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

bool span_geom(int nb, int64_t batch, int in, int out, SpanGeom* g) {
    // 512 rows per workgroup (two per thread), 16 outputs per thread for
    // narrow layers, else 32; both stages of one feature's weight tile within
    // 64 KiB of LDS (two workgroups per compute unit)
    g->ng = 1;
    g->nr = 2;
    g->opt = out <= 16 ? 16 : 32;
    if ((int64_t)(nb + 1) * g->opt * 4 * 2 > kSpanLdsBytes) g->opt = 16;
    if ((int64_t)(nb + 1) * g->opt * 4 * 2 > kSpanLdsBytes) return false;
    // a column stride of a multiple of 16 floats would put every row's window
    // column on the same LDS banks: pad it by one 16-byte unit where it fits
    g->cs = g->opt * g->ng;
    if ((int64_t)(nb + 1) * (g->cs + 4) * 4 * 2 <= kSpanLdsBytes) g->cs += 4;
    g->otiles = (out + g->opt * g->ng - 1) / (g->opt * g->ng);
    g->outp = g->otiles * g->opt * g->ng;
    const int64_t rw = (int64_t)kThreads / g->ng * g->nr;
    g->rblocks = (batch + rw - 1) / rw;
    // at least two workgroups per compute unit where the features allow it
    const int64_t tiles = g->rblocks * g->otiles > 0 ? g->rblocks * g->otiles : 1;
    int64_t fs = (kSpanTargetWgs + tiles - 1) / tiles;
    if (fs > in) fs = in;
    if (fs < 1) fs = 1;
    g->fpf = (int)((in + fs - 1) / fs);
    g->fs = (in + g->fpf - 1) / g->fpf;
    // (the grid's x extent in work-items must fit 32 bits)
    if (g->rblocks * kThreads > 0xffffffffLL || g->otiles > 65535 || g->fs > 65535) return false;
    size_t off = 0;
    g->off_w = off;
    off = align256s(off + (size_t)in * (nb + 1) * g->outp * 4);
    g->off_p = off;
    if (g->fs > 1) off = align256s(off + (size_t)g->fs * (size_t)batch * out * 4);
    g->bytes = off;
    return true;
}

hipError_t launch_span(bool bf16, const SpanGeom& g, const SpanArgs& a, const void* coef,
                       const void* bw, hipStream_t s) {
    if (a.batch == 0) return hipSuccess;
    return bf16 ? span_t<uint16_t>(g, a, coef, bw, s) : span_t<float>(g, a, coef, bw, s);
}

}  // namespace kan
