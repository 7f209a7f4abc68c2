// kan_basis.hip -- basis-only kernel: phi[e, j] = N_j(x[e]) for every input
// element and every basis j (eq. truncated with the clamp of eq. bounded; for
// degrees other than 3, eq. general_truncated with the clamp to [0, k + 1]).
//
// The kernel is bound by HBM writes (nb outputs per input read).  Each
// 256-thread workgroup owns xb consecutive inputs, i.e. one contiguous
// xb * nb run of the output:
//   phase 1  tpx threads per input evaluate its nb values in registers (the
//            coordinate, then for the cubic 6 VALU ops for N / 2 and one
//            scale, no span lookup, no data-dependent branches) and write them
//            to LDS in output order;
//   phase 2  the workgroup streams the run from LDS to HBM with 16-byte
//            non-temporal stores, so every store instruction of a wave covers
//            1 KiB of consecutive output.
// NaN inputs give NaN outputs: the final scale (2 for the cubic's N / 2, else
// 1) is replaced by the NaN itself.
#include "kan_internal.h"

namespace kan {

namespace {

constexpr int kThreads = 256;

template <typename T>
__device__ __forceinline__ void store_vec(T* dst, const float* src);

template <>
__device__ __forceinline__ void store_vec<float>(float* dst, const float* src) {
    const floatx4 v = *reinterpret_cast<const floatx4*>(src);
    __builtin_nontemporal_store(v, reinterpret_cast<floatx4*>(dst));
}

template <>
__device__ __forceinline__ void store_vec<uint16_t>(uint16_t* dst, const float* src) {
    const floatx4 lo = *reinterpret_cast<const floatx4*>(src);
    const floatx4 hi = *reinterpret_cast<const floatx4*>(src + 4);
    u16x8 v;
    v[0] = f32_to_bf16(lo[0]); v[1] = f32_to_bf16(lo[1]);
    v[2] = f32_to_bf16(lo[2]); v[3] = f32_to_bf16(lo[3]);
    v[4] = f32_to_bf16(hi[0]); v[5] = f32_to_bf16(hi[1]);
    v[6] = f32_to_bf16(hi[2]); v[7] = f32_to_bf16(hi[3]);
    __builtin_nontemporal_store(v, reinterpret_cast<u16x8*>(dst));
}

// A basis at v = u - (K + 1) / 2, up to the factor kScale<K>: the cubic's
// two-term form N / 2 (kan_device.h) for K = 3, the reflected general form
// otherwise.
template <int K>
__device__ __forceinline__ float basis_value(float v) {
    if constexpr (K == 3) return half_basis(v);
    else return basis_deg<K>(v);
}
template <int K> constexpr float kScale = K == 3 ? 2.0f : 1.0f;

// Phase 2 of the basis kernels: stream the contiguous run of `total` staged
// values to `out`.
template <typename T>
__device__ __forceinline__ void stream_out(const float* stage, T* out, int total, int vec) {
    int done = 0;
    if (vec && (reinterpret_cast<uintptr_t>(out) % 16) == 0) {
        constexpr int V = 16 / sizeof(T);
        const int nvec = total / V;
        for (int q = threadIdx.x; q < nvec; q += kThreads)
            store_vec<T>(out + q * V, stage + q * V);
        done = nvec * V;
    }
    for (int q = done + threadIdx.x; q < total; q += kThreads)
        Storage<T>::store(out + q, stage[q]);
}

template <typename T, int K>
__global__ __launch_bounds__(kThreads) void basis_kernel(const T* __restrict__ x, int64_t n,
                                                         T* __restrict__ phi, GridConst g,
                                                         int tpx, int jc, int vec) {
    extern __shared__ float stage[];
    const int nb = g.nb;
    const int xb = kThreads / tpx;
    const int64_t e0 = (int64_t)blockIdx.x * xb;
    const int64_t left = n - e0;
    const int cnt = left < xb ? (int)left : xb;

    // Phase 1: values [jb, je) of input el, written to stage[el * nb + j].
    const int el = threadIdx.x / tpx;
    const int jb = (threadIdx.x % tpx) * jc;
    const int je = min(jb + jc, nb);
    if (el < cnt) {
        const float xv = Storage<T>::load(x + e0 + el);
        const float scale = (xv != xv) ? xv : kScale<K>;  // a NaN input gives NaN values
        float cj = g.a_int - (float)jb;
        float* dst = stage + el * nb;
        if (tpx == 1 && g.a_frac == 0.0f && g.inv_lo == 0.0f) {
            // (uniform trip count; on grids whose 1 / h and lo / h are exact
            // the coordinate is the fma alone)
#pragma unroll 4
            for (int j = 0; j < nb; ++j) {
                dst[j] = basis_value<K>(__builtin_fmaf(xv, g.inv_h, cj)) * scale;
                cj -= 1.0f;
            }
        } else {
            const float lo = coord_lo(xv, g.xlim, g.inv_lo, g.a_frac);
#pragma unroll 4
            for (int j = jb; j < je; ++j) {
                dst[j] = basis_value<K>(__builtin_fmaf(xv, g.inv_h, cj) + lo) * scale;
                cj -= 1.0f;
            }
        }
    }
    __syncthreads();
    stream_out<T>(stage, phi + e0 * nb, cnt * nb, vec);
}

// ------------------------------------------------------------ Cox-de Boor
//
// The same basis by the recursion of eq. cdb0 / eq. cdbk over every knot
// interval, as a B-spline layer without span lookup evaluates it (the
// evaluation the paper measures its truncated-power form against).  With
// uniform knots t_j = lo + (j - K) h the recursion's weights are
// (x - t_j) / (t_{j+p} - t_j) = u_j / p and (t_{j+p+1} - x) / (t_{j+p+1} -
// t_{j+1}) = (p + 1 - u_j) / p, u_j = (x - t_j) / h, so for p = 1 .. K
//   N_{j,p} = (u_j N_{j,p-1} + (p + 1 - u_j) N_{j+1,p-1}) / p,
// starting from N_{j,0} = [0 <= u_j < 1] for the W = G + 2K intervals (the
// half-open indicator of eq. cdb0), set from floor(u_0) so that exactly one
// interval holds x.  Each weight's u_j is one fma at its own magnitude (plus
// the 1/h residual term).  A NaN input gives NaN values
// (its indicators are all 0, so the NaN is added back explicitly).
//
// basis_cdb_kernel: one thread per input, the W values of a level in
// registers (MW >= W at compile time).
template <typename T, int K, int MW>
__global__ __launch_bounds__(kThreads) void basis_cdb_kernel(const T* __restrict__ x, int64_t n,
                                                             T* __restrict__ phi, GridConst g,
                                                             int vec) {
    extern __shared__ float stage[];
    const int nb = g.nb;
    const int W = nb + K;
    const int64_t e0 = (int64_t)blockIdx.x * kThreads;
    const int64_t left = n - e0;
    const int cnt = left < kThreads ? (int)left : kThreads;
    const int el = threadIdx.x;
    if (el < cnt) {
        const float xv = Storage<T>::load(x + e0 + el);
        // (an input clamped to +-xlim, past every knot, gives the same zeros
        // and keeps the weights u_j finite for infinite inputs)
        const float xc = __builtin_amdgcn_fmed3f(xv, -g.xlim, g.xlim);
        const float lo = coord_lo(xc, g.xlim, g.inv_lo, g.a_frac);
        const float c0 = g.a_int + g.hw;  // u_j = x / h - lo / h + K - j
        // the interval holding x, from one coordinate (so that exactly one
        // indicator is set, however the u_j below round)
        const float span = __builtin_floorf(__builtin_fmaf(xc, g.inv_h, c0) + lo);
        float u[MW], w[MW];
#pragma unroll
        for (int j = 0; j < MW; ++j) {
            u[j] = __builtin_fmaf(xc, g.inv_h, c0 - (float)j) + lo;
            w[j] = (j < W && span == (float)j) ? 1.0f : 0.0f;
        }
#pragma unroll
        for (int p = 1; p <= K; ++p) {
            const float ip = 1.0f / (float)p;
#pragma unroll
            for (int j = 0; j + p < MW; ++j)
                w[j] = (u[j] * w[j] + ((float)(p + 1) - u[j]) * w[j + 1]) * ip;
        }
        const float nanv = xv != xv ? xv : 0.0f;
        float* dst = stage + el * nb;
#pragma unroll
        for (int j = 0; j + K < MW; ++j)
            if (j < nb) dst[j] = w[j] + nanv;
    }
    __syncthreads();
    stream_out<T>(stage, phi + e0 * nb, cnt * nb, vec);
}

// basis_cdb_lds_kernel: wider grids, each thread's level in an LDS row of
// wp >= W floats (tpb threads per workgroup); the rows' first nb values are
// the output.
template <typename T, int K>
__global__ __launch_bounds__(64) void basis_cdb_lds_kernel(const T* __restrict__ x, int64_t n,
                                                           T* __restrict__ phi, GridConst g,
                                                           int wp, int tpb) {
    extern __shared__ float work[];
    const int nb = g.nb;
    const int W = nb + K;
    const int64_t e0 = (int64_t)blockIdx.x * tpb;
    const int64_t left = n - e0;
    const int cnt = left < tpb ? (int)left : tpb;
    const int el = threadIdx.x;
    if (el < cnt) {
        const float xv = Storage<T>::load(x + e0 + el);
        const float xc = __builtin_amdgcn_fmed3f(xv, -g.xlim, g.xlim);
        const float lo = coord_lo(xc, g.xlim, g.inv_lo, g.a_frac);
        const float c0 = g.a_int + g.hw;
        const float span = __builtin_floorf(__builtin_fmaf(xc, g.inv_h, c0) + lo);
        float* w = work + el * wp;
        for (int j = 0; j < W; ++j) w[j] = span == (float)j ? 1.0f : 0.0f;
        for (int p = 1; p <= K; ++p) {
            const float ip = 1.0f / (float)p;
            float next = w[0];
            for (int j = 0; j + p < W; ++j) {
                const float u = __builtin_fmaf(xc, g.inv_h, c0 - (float)j) + lo;
                const float cur = next;
                next = w[j + 1];
                w[j] = (u * cur + ((float)(p + 1) - u) * next) * ip;
            }
        }
        if (xv != xv)
            for (int j = 0; j < nb; ++j) w[j] = xv;
    }
    __syncthreads();
    T* out = phi + e0 * nb;
    for (int q = threadIdx.x; q < cnt * nb; q += blockDim.x)
        Storage<T>::store(out + q, work[(q / nb) * wp + q % nb]);
}

}  // namespace

BasisLaunch plan_basis(int64_t n, int nb, const void* phi) {
    BasisLaunch L;
    // Smallest power-of-two split of each input's nb values over threads that
    // keeps the workgroup's LDS run at or below 32 KiB (at most 64 KiB for the
    // largest grids).  A run whose start is not 16-byte aligned (possible only
    // when xb * nb * sizeof(T) is not a multiple of 16) falls back to scalar
    // stores for that workgroup.
    int tpx = 1;
    while (tpx < 64 && (size_t)(kThreads / tpx) * nb * 4 > 32768) tpx *= 2;
    L.tpx = tpx;
    L.xb = kThreads / tpx;
    L.jc = (nb + tpx - 1) / tpx;
    L.lds = (size_t)L.xb * nb * 4;
    L.blocks = (n + L.xb - 1) / L.xb;
    L.vec = (reinterpret_cast<uintptr_t>(phi) % 16) == 0;
    return L;
}

template <typename T, int K>
static hipError_t launch_k(const T* x, int64_t n, T* phi, const GridConst& g,
                           const BasisLaunch& L, hipStream_t s) {
    hipLaunchKernelGGL((basis_kernel<T, K>), dim3((unsigned)L.blocks), dim3(kThreads), L.lds, s,
                       x, n, phi, g, L.tpx, L.jc, L.vec ? 1 : 0);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch(const T* x, int64_t n, T* phi, const GridConst& g, const BasisLaunch& L,
                         hipStream_t s) {
    switch (g.k) {
        case 1: return launch_k<T, 1>(x, n, phi, g, L, s);
        case 2: return launch_k<T, 2>(x, n, phi, g, L, s);
        case 3: return launch_k<T, 3>(x, n, phi, g, L, s);
        case 4: return launch_k<T, 4>(x, n, phi, g, L, s);
        case 5: return launch_k<T, 5>(x, n, phi, g, L, s);
        case 6: return launch_k<T, 6>(x, n, phi, g, L, s);
        case 7: return launch_k<T, 7>(x, n, phi, g, L, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_basis_f32(const float* x, int64_t n, float* phi, const GridConst& g,
                            const BasisLaunch& L, hipStream_t s) {
    return launch<float>(x, n, phi, g, L, s);
}

hipError_t launch_basis_bf16(const uint16_t* x, int64_t n, uint16_t* phi, const GridConst& g,
                             const BasisLaunch& L, hipStream_t s) {
    return launch<uint16_t>(x, n, phi, g, L, s);
}

}  // namespace kan

namespace kan {

namespace {

template <typename T, int K>
hipError_t launch_cdb_k(const T* x, int64_t n, T* phi, const GridConst& g, hipStream_t s) {
    const int W = g.nb + K;
    const int vec = (reinterpret_cast<uintptr_t>(phi) % 16) == 0 ? 1 : 0;
    const unsigned blocks = (unsigned)((n + kThreads - 1) / kThreads);
    const size_t lds = (size_t)kThreads * g.nb * 4;
    if (W <= 16) {
        hipLaunchKernelGGL((basis_cdb_kernel<T, K, 16>), dim3(blocks), dim3(kThreads), lds, s, x,
                           n, phi, g, vec);
    } else if (W <= 32) {
        hipLaunchKernelGGL((basis_cdb_kernel<T, K, 32>), dim3(blocks), dim3(kThreads), lds, s, x,
                           n, phi, g, vec);
    } else {
        // rows of an odd number of floats (no bank conflicts between the
        // threads' rows), as many threads as fit 64 KiB of LDS
        const int wp = W | 1;
        int tpb = 64;
        while (tpb > 1 && (size_t)tpb * wp * 4 > 65536) tpb /= 2;
        const int64_t nblk = (n + tpb - 1) / tpb;
        if (nblk > 0x7fffffffLL) return hipErrorInvalidValue;
        hipLaunchKernelGGL((basis_cdb_lds_kernel<T, K>), dim3((unsigned)nblk), dim3(tpb),
                           (size_t)tpb * wp * 4, s, x, n, phi, g, wp, tpb);
    }
    return hipGetLastError();
}

template <typename T>
hipError_t launch_cdb(const T* x, int64_t n, T* phi, const GridConst& g, hipStream_t s) {
    switch (g.k) {
        case 1: return launch_cdb_k<T, 1>(x, n, phi, g, s);
        case 2: return launch_cdb_k<T, 2>(x, n, phi, g, s);
        case 3: return launch_cdb_k<T, 3>(x, n, phi, g, s);
        case 4: return launch_cdb_k<T, 4>(x, n, phi, g, s);
        case 5: return launch_cdb_k<T, 5>(x, n, phi, g, s);
        case 6: return launch_cdb_k<T, 6>(x, n, phi, g, s);
        case 7: return launch_cdb_k<T, 7>(x, n, phi, g, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_basis_cdb_f32(const float* x, int64_t n, float* phi, const GridConst& g,
                                hipStream_t s) {
    return launch_cdb<float>(x, n, phi, g, s);
}

hipError_t launch_basis_cdb_bf16(const uint16_t* x, int64_t n, uint16_t* phi, const GridConst& g,
                                 hipStream_t s) {
    return launch_cdb<uint16_t>(x, n, phi, g, s);
}

}  // namespace kan
