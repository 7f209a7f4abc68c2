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

    // Phase 2: stream the contiguous run [e0 * nb, (e0 + cnt) * nb) out.
    const int total = cnt * nb;
    T* out = phi + e0 * nb;
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
