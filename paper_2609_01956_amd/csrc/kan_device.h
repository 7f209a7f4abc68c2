// kan_device.h -- device-side helpers shared by the gfx950 kernels.
//
// Basis evaluation.  With the grid convention t_j = lo + (j - 3) h, the
// normalised coordinate of basis j is u_j = (x - t_j) / h = x/h - lo/h + 3 - j.
// The kernels form v_j = u_j - 2 with one fused multiply-add,
//     v_j = fma(x, inv_h, a_int - j) + a_frac,
// where a_int + a_frac = 1 - lo/h is split on the host into an integer part
// (so a_int - j is exact) and a small remainder (zero on grids whose lo/h is an
// integer, e.g. [-1, 1] with even G).  Near the support |v_j| <= 2, so the
// single rounding of the fma is at most 2^-23 in u.
//
// The truncated-power form (eq. truncated) with the bounded coordinate
// ubar = clamp(u, 0, 4) (eq. bounded) is evaluated at the reflected coordinate
// w = min(ubar, 4 - ubar) = 2 - min(|v|, 2).  The stencil {1, -4, 6, -4, 1} is
// symmetric, so N(ubar) = N(4 - ubar) = N(w), and for w <= 2 the terms
// (w - m)_+^3 with m >= 2 vanish:
//     6 N = w^3 - 4 b^3,   b = (w - 1)_+ = max(1 - min(|v|, 2), 0).
// With the 1/6 and the 4 folded into two scale factors (both below 1):
//     N / 2 = P^3 - Q^3,
//     P = (2/3)^(1/3) w / 2 = clamp01((2/3)^(1/3) (1 - |v| / 2)),
//     Q = (1/3)^(1/3) b     = clamp01((1/3)^(1/3) (1 - |v|)),
// where the clamp to [0, 1] only ever acts at 0.  Each value is two clamped
// fused multiply-adds (the clamp and |v| fold into the instruction), three
// multiplies and one fused multiply-add.  Evaluating at w instead of ubar
// avoids the cancellation of terms of size up to 64 near ubar = 4; the fp32
// error stays below 4e-7.  Off the support P = Q = 0 and the value is exactly
// 0 (also for +-Inf inputs).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace kan {

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Fourth word of a raw buffer resource (stride 0) on CDNA GPUs: 32-bit data
// format, no swizzling; reads past the resource's byte count return 0.
constexpr int kBufferWord3 = 0x00020000;
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// Grid constants shared by all kernels (computed on the host in double).
// For degree k the coordinate of basis j relative to the centre of its
// support is v_j = u_j - (k + 1) / 2 = x / h - lo / h + (k - 1) / 2 - j, formed as
//     v_j = fma(x, inv_h, a_int - j) + (x' inv_lo + a_frac),
// with inv_h + inv_lo = 1 / h (inv_lo the fp32 rounding residual of 1 / h,
// 0 when 1 / h is exact) and a_int + a_frac = (k - 1) / 2 - lo / h, and x'
// the input clamped to [-xlim, xlim] (a range past every support: the
// correction stays finite for infinite inputs, whose basis is 0 anyway).
struct GridConst {
    int nb;        // G + k basis functions per input
    int k;         // spline degree, 1 .. 7
    float inv_h;   // G / (hi - lo), rounded to fp32
    float inv_lo;  // G / (hi - lo) - inv_h, rounded to fp32
    float a_int;   // nearest integer to (k - 1) / 2 - lo / h
    float a_frac;  // ((k - 1) / 2 - lo / h) - a_int, rounded to fp32
    float xlim;    // max(|lo|, |hi|) + (k + 2) h
    float hw;      // (k + 1) / 2, the half width of a support
    float hc[4];   // (-1)^m C(k + 1, m) / (2 k!), m = 0 .. 3
};

// x' inv_lo + a_frac (see GridConst).
__device__ __forceinline__ float coord_lo(float x, float xlim, float inv_lo, float a_frac) {
    return __builtin_fmaf(__builtin_amdgcn_fmed3f(x, -xlim, xlim), inv_lo, a_frac);
}

// N_k(u) / 2 at v = u - (k + 1) / 2 for a degree k known at run time
// (eq. general_truncated with the clamp of eq. bounded, at the reflected
// coordinate w = hw - min(|v|, hw), where only the terms m < w survive:
// N / 2 = sum_m hc[m] (w - m)_+^k).
__device__ __forceinline__ float half_basis_deg(float v, int k, float hw, const float (&hc)[4]) {
    const float w = hw - __builtin_fminf(__builtin_fabsf(v), hw);
    float s = 0.0f;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const float z = __builtin_fmaxf(w - (float)m, 0.0f);
        float p = z;
        for (int i = 1; i < k; ++i) p *= z;
        s = __builtin_fmaf(hc[m], p, s);
    }
    return s;
}

// N_K(u) at v = u - (K + 1) / 2 for a compile-time degree K, the same form.
template <int K>
__device__ __forceinline__ float basis_deg(float v) {
    constexpr float hw = 0.5f * (K + 1);
    constexpr int M = (K + 1) / 2;  // terms m < hw
    const float w = hw - __builtin_fminf(__builtin_fabsf(v), hw);
    float kf = 1.0f;
    for (int i = 2; i <= K; ++i) kf *= (float)i;
    float s = 0.0f, binom = 1.0f;
#pragma unroll
    for (int m = 0; m < M + (K % 2 == 0 ? 1 : 0) && m < 4; ++m) {
        const float z = __builtin_fmaxf(w - (float)m, 0.0f);
        float p = z;
#pragma unroll
        for (int i = 1; i < K; ++i) p *= z;
        s = __builtin_fmaf((m & 1 ? -binom : binom) / kf, p, s);
        binom = binom * (float)(K + 1 - m) / (float)(m + 1);
    }
    return s;
}

constexpr float kCbrtTwoThirds = 0.87358046473629571f;  // (2/3)^(1/3)
constexpr float kCbrtOneThird = 0.69336127435063470f;   // (1/3)^(1/3)

// N(u) / 2 from v = u - 2 (see the header comment).
__device__ __forceinline__ float half_basis(float v) {
    const float av = __builtin_fabsf(v);
    const float P = __builtin_amdgcn_fmed3f(
        __builtin_fmaf(av, -0.5f * kCbrtTwoThirds, kCbrtTwoThirds), 0.0f, 1.0f);
    const float Q = __builtin_amdgcn_fmed3f(
        __builtin_fmaf(av, -kCbrtOneThird, kCbrtOneThird), 0.0f, 1.0f);
    return __builtin_fmaf(P * P, P, -(Q * Q * Q));
}

// v_j = u_j - (k + 1) / 2 for basis j, given cj = a_int - j.
__device__ __forceinline__ float coord(float x, const GridConst& g, float cj) {
    return __builtin_fmaf(x, g.inv_h, cj) + coord_lo(x, g.xlim, g.inv_lo, g.a_frac);
}

// silu(x) = x / (1 + exp(-x)).
__device__ __forceinline__ float silu(float x) {
    return x / (1.0f + __expf(-x));
}

// bfloat16 storage <-> fp32.  Widening is exact; narrowing rounds to nearest
// even (v_cvt_pk_bf16_f32 on gfx950) and keeps NaN a NaN.
__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
    return __uint_as_float(((uint32_t)u) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    __bf16 b = (__bf16)f;
    return __builtin_bit_cast(uint16_t, b);
}

template <typename T> struct Storage;
template <> struct Storage<float> {
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Storage<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// Compile-time loop: f(std::integral_constant<int, I>) for I = 0 .. N - 1.
template <int I, int N>
struct StaticFor {
    template <typename F>
    __device__ __forceinline__ static void run(F&& f) {
        f(std::integral_constant<int, I>{});
        StaticFor<I + 1, N>::run(f);
    }
};
template <int N>
struct StaticFor<N, N> {
    template <typename F>
    __device__ __forceinline__ static void run(F&&) {}
};

}  // namespace kan
