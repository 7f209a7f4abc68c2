// kan_layer.hip -- fused KAN-layer forward on MFMA (eq. kan_forward):
//
//   y[b, o] = sum_i sum_{j<=nb} A[b, (i, j)] * W[o, (i, j)]
//   A[b, (i, j)] = N_j(x[b, i]) for j < nb,   silu(x[b, i]) for j = nb
//   W[o, (i, j)] = coef[o, i, j]   for j < nb,   base_w[o, i]  for j = nb
//
// i.e. a dense [batch, in * (nb + 1)] x [in * (nb + 1), out] contraction whose
// left operand is never stored: every lane generates its own A elements in
// registers, directly in the MFMA operand layout, from one x value per K-step.
//
// Work decomposition
//   * A workgroup is 4 waves (wm x wn).  Each wave owns 32 rows of the batch and
//     nt 32-column tiles of y, accumulated in fp32 MFMA registers.
//   * The K dimension is walked feature-major: step (p, c) covers features
//     2p and 2p + 1 and columns [c * cw, c * cw + cw) of each feature's
//     nbp = roundup(nb + 1, kgroup) columns.  Lanes 0..31 of a wave feed the
//     first feature and lanes 32..63 the second: that is exactly the k split of
//     v_mfma_f32_32x32x2_f32 (one k per lane half) and of
//     v_mfma_f32_32x32x16_bf16 (eight consecutive k per lane half), so one x
//     load per lane serves a whole step.
//   * The matching W slice [bn, 2, cw] is staged in LDS, shared by the waves,
//     with columns beyond nb + 1 (and features or outputs beyond the problem)
//     zero-filled, so padding contributes exactly 0.
//
// fp32 path: A is fp32, MFMA 32x32x2 f32.  bf16 path: x and W are bf16 in
// memory; A is generated in fp32 and rounded to bf16 (RNE) in registers; MFMA
// 32x32x16 bf16 with fp32 accumulation; y is rounded to bf16 on store.
#include "kan_internal.h"

#include <cstdlib>
#include <cstring>

namespace kan {

namespace {

constexpr int kThreads = 256;

template <typename T> struct Mma;

template <> struct Mma<float> {
    static constexpr int kGroup = 1;   // k per lane half per MFMA
    static constexpr int kCwMax = kLayerCwMaxF32;  // columns per feature per K-step
    static constexpr int kPad = 4;     // LDS row padding (elements)
    typedef float AVec;
    static __device__ __forceinline__ floatx16 mma(AVec a, AVec b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ void put(float* p, float v) { *p = v; }
};

template <> struct Mma<uint16_t> {
    static constexpr int kGroup = 8;
    static constexpr int kCwMax = kLayerCwMaxBf16;
    static constexpr int kPad = 8;
    typedef bf16x8 AVec;
    static __device__ __forceinline__ floatx16 mma(AVec a, AVec b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void put(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// A element for column j of a feature whose input is xv (silu value sv).
__device__ __forceinline__ float a_value(float xv, float sv, int j, const GridConst& g) {
    if (j < g.nb) return tp6(coord(xv, g, g.a_int - (float)j)) * (1.0f / 6.0f);
    return j == g.nb ? sv : 0.0f;
}

template <typename T, int NT>
struct Operand;

template <int NT>
struct Operand<float, NT> {
    static __device__ __forceinline__ float a(float xv, float sv, int j0, const GridConst& g) {
        return a_value(xv, sv, j0, g);
    }
    static __device__ __forceinline__ float b(const float* Bs) { return *Bs; }
};

template <int NT>
struct Operand<uint16_t, NT> {
    static __device__ __forceinline__ bf16x8 a(float xv, float sv, int j0, const GridConst& g) {
        bf16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (__bf16)a_value(xv, sv, j0 + e, g);
        return v;
    }
    static __device__ __forceinline__ bf16x8 b(const uint16_t* Bs) {
        const u16x8 u = *reinterpret_cast<const u16x8*>(Bs);
        return __builtin_bit_cast(bf16x8, u);
    }
};

template <typename T, int NT, int WM, int WN>
__global__ __launch_bounds__(kThreads) void layer_kernel(LayerArgs a) {
    typedef Mma<T> M;
    constexpr int KG = M::kGroup;
    constexpr int BM = 32 * WM;
    constexpr int BN = 32 * NT * WN;
    constexpr int RSMAX = 2 * M::kCwMax + M::kPad;
    __shared__ __attribute__((aligned(16))) T Bs[BN * RSMAX];

    const T* __restrict__ x = static_cast<const T*>(a.x);
    const T* __restrict__ coef = static_cast<const T*>(a.coef);
    const T* __restrict__ wb = static_cast<const T*>(a.wb);
    T* __restrict__ y = static_cast<T*>(a.y);
    const GridConst g = a.g;
    const int nb = g.nb;
    const int cw = a.cw;
    const int rs = 2 * cw + M::kPad;

    const int tid = threadIdx.x;
    const int wave = tid / 64;
    const int lane = tid % 64;
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int r = lane % 32;
    const int h = lane / 32;

    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int64_t row = m0 + wm * 32 + r;
    const bool row_ok = row < a.batch;

    floatx16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[t][q] = 0.0f;

    const int npairs = (a.in + 1) / 2;
    const int tile_elems = BN * 2 * cw;
    for (int p = 0; p < npairs; ++p) {
        const int f0 = 2 * p;
        // x of this lane's feature; features past `in` read as 0 (their W is 0).
        const int f = f0 + h;
        float xv = 0.0f;
        if (row_ok && f < a.in) xv = M::load(x + row * a.in + f);
        const float sv = silu(xv);

        for (int c = 0; c < a.nchunks; ++c) {
            const int jbase = c * cw;
            // Stage W[n0 .. n0 + BN, (f0, f0 + 1), jbase .. jbase + cw) in LDS.
            for (int idx = tid; idx < tile_elems; idx += kThreads) {
                const int jj = idx & (cw - 1);
                const int hh = (idx / cw) & 1;
                const int nl = idx / (2 * cw);
                const int ng = n0 + nl;
                const int fg = f0 + hh;
                const int j = jbase + jj;
                float v = 0.0f;
                if (ng < a.out && fg < a.in) {
                    if (j < nb)
                        v = M::load(coef + ((int64_t)ng * a.in + fg) * nb + j);
                    else if (j == nb)
                        v = M::load(wb + (int64_t)ng * a.in + fg);
                }
                M::put(&Bs[nl * rs + hh * cw + jj], v);
            }
            __syncthreads();

            const int ncols = min(cw, a.nbp - jbase);
            const int nm = ncols / KG;
            for (int s = 0; s < nm; ++s) {
                const typename M::AVec av = Operand<T, NT>::a(xv, sv, jbase + s * KG, g);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int nl = wn * NT * 32 + t * 32 + r;
                    const typename M::AVec bv = Operand<T, NT>::b(&Bs[nl * rs + h * cw + s * KG]);
                    acc[t] = M::mma(av, bv, acc[t]);
                }
            }
            __syncthreads();
        }
    }

    // Epilogue: 32x32 accumulator layout, element q of lane l holds
    // row 8 * (q / 4) + 4 * (l / 32) + (q % 4), column l % 32.
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int col = n0 + wn * NT * 32 + t * 32 + r;
        if (col >= a.out) continue;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int64_t rr = m0 + wm * 32 + 8 * (q / 4) + 4 * h + (q % 4);
            if (rr < a.batch) Storage<T>::store(y + rr * a.out + col, acc[t][q]);
        }
    }
}

template <typename T, int NT, int WM, int WN>
hipError_t launch_tile(const LayerArgs& a, hipStream_t s) {
    constexpr int BM = 32 * WM;
    constexpr int BN = 32 * NT * WN;
    const dim3 grid((unsigned)((a.batch + BM - 1) / BM), (unsigned)((a.out + BN - 1) / BN));
    hipLaunchKernelGGL((layer_kernel<T, NT, WM, WN>), grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

// Workgroup tiles are at most 256 columns wide (nt * wn <= 8).
template <typename T, int NT>
hipError_t launch_nt(const LayerArgs& a, const LayerTile& t, hipStream_t s) {
    if (t.wm == 4 && t.wn == 1) return launch_tile<T, NT, 4, 1>(a, s);
    if constexpr (NT <= 4) {
        if (t.wm == 2 && t.wn == 2) return launch_tile<T, NT, 2, 2>(a, s);
    }
    if constexpr (NT <= 2) {
        if (t.wm == 1 && t.wn == 4) return launch_tile<T, NT, 1, 4>(a, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_any(const LayerArgs& a, const LayerTile& t, hipStream_t s) {
    switch (t.nt) {
        case 1: return launch_nt<T, 1>(a, t, s);
        case 2: return launch_nt<T, 2>(a, t, s);
        case 4: return launch_nt<T, 4>(a, t, s);
        case 8: return launch_nt<T, 8>(a, t, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

LayerTile plan_layer_tile(int64_t batch, int out) {
    // One 4-wave workgroup per (128 rows x up to 256 columns) by default; when
    // that leaves fewer than two workgroups per CU (256 CUs), trade rows for
    // columns inside the workgroup (2 x 2, then 1 x 4 waves).
    LayerTile t;
    int nt = 1;
    while (nt < 8 && 32 * nt < out) nt *= 2;
    t.nt = nt;
    t.wm = 4;
    t.wn = 1;
    auto blocks = [&](const LayerTile& c) {
        const int64_t bm = 32 * c.wm, bn = 32 * c.nt * c.wn;
        return ((batch + bm - 1) / bm) * ((out + bn - 1) / bn);
    };
    const int64_t want = 512;
    if (blocks(t) < want && t.nt >= 2) {
        LayerTile c{t.nt / 2, 2, 2};
        t = c;
        if (blocks(t) < want && t.nt >= 2) {
            LayerTile d{t.nt / 2, 1, 4};
            t = d;
        }
    }
    return t;
}

// KAN_LAYER_TILE="nt,wm,wn" forces a tile configuration (testing and tuning).
bool parse_layer_tile_override(LayerTile* t) {
    const char* s = std::getenv("KAN_LAYER_TILE");
    if (!s || !*s) return false;
    int nt = 0, wm = 0, wn = 0;
    if (std::sscanf(s, "%d,%d,%d", &nt, &wm, &wn) != 3) return false;
    const bool nt_ok = nt == 1 || nt == 2 || nt == 4 || nt == 8;
    const bool w_ok = (wm == 4 && wn == 1) || (wm == 2 && wn == 2) || (wm == 1 && wn == 4);
    if (!nt_ok || !w_ok || nt * wn > 8) return false;
    t->nt = nt;
    t->wm = wm;
    t->wn = wn;
    return true;
}

hipError_t launch_layer_f32(const LayerArgs& a, const LayerTile& t, hipStream_t s) {
    return launch_any<float>(a, t, s);
}

hipError_t launch_layer_bf16(const LayerArgs& a, const LayerTile& t, hipStream_t s) {
    return launch_any<uint16_t>(a, t, s);
}

}  // namespace kan
