// kan_narrow.hip -- fused KAN-layer forward (eq. kan_forward) of narrow fp32
// layers (cubic, at most 16 outputs) on the vector ALUs.
//
// With a handful of outputs the matrix cores have little to do: a 32-column
// fp32 MFMA tile is mostly padding, and its A operand needs every one of a
// feature's G + 3 basis columns.  Here each lane owns one batch row.  Per
// input feature it evaluates only the four basis functions whose support
// holds x (the clamped form of eq. bounded is exactly zero elsewhere) and the
// SiLU value, and adds them times the feature's weights into its outputs,
// held in registers:
//
//   y[b, o] = 2 sum_i ( silu(x)/2 W[o, (i, 0)] + sum_{k<4} N_{c0+k-1}(x)/2 W[o, (i, c0 + k)] )
//
// with the columns of a feature ordered [SiLU weight, coef[.., 0 .. nb - 1]]
// as in the packed buffer and c0 the first column of x's window.  The four
// waves of a workgroup take the same 64 rows and a quarter of the features
// each (two consecutive features of every chunk of 8), and add their partial
// sums through LDS at the end, in wave order.
//
// The weights of a chunk of 8 features go from the packed buffer (the MFMA
// layout, kan_internal.h) through registers into LDS as a table
// [feature][column][output]: one row of RS floats per column, the columns
// zero-padded up to the last window column (nb + 2).  Each lane reads the
// rows of its window; the SiLU row has the same address in every lane.  Two
// LDS stages: chunk c + 1 is loaded while chunk c is evaluated, stored
// after it, and one barrier per chunk separates the two.
#include "kan_layer_kernel.h"

#include "kan.h"

namespace kan {

namespace {

// Features per staged chunk, two per wave (256 -> 10 at batch 65536: 58 us,
// against 63 with 16 features per chunk, 66 with 4 and 76 with 32).
constexpr int kNarrowFeat = 8;
constexpr int kFW = kNarrowFeat / 4;  // features per wave and chunk

// Columns of a feature's LDS rows: the SiLU column, nb coefficients and the
// zero columns up to nb + 2 (the last window column), rounded up to even.
inline int narrow_cols(int nb) { return (nb + 4) & ~1; }

// NO: outputs computed per lane (even, >= out); RS: LDS row stride in floats.
template <int NO>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
void narrow_kernel(LayerArgs a, int cw) {
    constexpr int RS = (NO + 3) / 4 * 4;
    constexpr int NV = 2 * RS;  // floats of one staging unit (two columns)
    extern __shared__ floatx4 lds4[];
    float* lds = reinterpret_cast<float*>(lds4);
    const int stage_floats = kNarrowFeat * cw * RS;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t row0 = (int64_t)blockIdx.x * kNarrowRows;
    // rows past the batch read the last row (their results are not stored)
    const int64_t row = row0 + lane < a.batch ? row0 + lane : a.batch - 1;
    const float* __restrict__ xr = static_cast<const float*>(a.x) + row * (int64_t)a.in;
    const float* __restrict__ wp = static_cast<const float*>(a.wp);
    const int nchunks = (a.in + kNarrowFeat - 1) / kNarrowFeat;
    const int fpk = 2 * a.npairs;  // features the packed buffer holds (zero past in)

    // Staging: thread t < 8 * cw / 2 moves unit (feature fl, column pair cp)
    // of every chunk: in the packed buffer outputs 0 .. RS - 1 of block
    // (pair, cp), half fl % 2, are 2 RS consecutive floats (columns 2 cp and
    // 2 cp + 1 interleaved); in LDS they become rows 2 cp and 2 cp + 1 of the
    // feature.  Column pairs past the packed blocks (cp >= nsb) are zeros.
    const int cpn = cw / 2;
    const bool stager = tid < kNarrowFeat * cpn;
    const int sfl = tid / cpn, scp = tid - (tid / cpn) * cpn;
    const bool s_cols = scp < a.nsb;
    // float offset of the unit in chunk 0; a chunk is 4 pairs further on
    const int64_t s_off = ((((int64_t)(sfl >> 1) * a.nsb + scp) * 2 + (sfl & 1)) * 32) * 2;
    const int64_t chunk_floats = (int64_t)(kNarrowFeat / 2) * a.nsb * 128;
    const int s_row = (sfl * cw + 2 * scp) * RS;

    float wv[NV];
    auto load_w = [&](int c) {
        const bool ok = stager && s_cols && c * kNarrowFeat + sfl < fpk;
        const floatx4* src = reinterpret_cast<const floatx4*>(wp + c * chunk_floats + s_off);
#pragma unroll
        for (int q = 0; q < NV / 4; ++q) {
            const floatx4 v = ok ? src[q] : floatx4{0.0f, 0.0f, 0.0f, 0.0f};
            wv[4 * q] = v[0];
            wv[4 * q + 1] = v[1];
            wv[4 * q + 2] = v[2];
            wv[4 * q + 3] = v[3];
        }
    };
    auto store_w = [&](int st) {
        if (!stager) return;
        floatx4* d0 = reinterpret_cast<floatx4*>(lds + st * stage_floats + s_row);
        floatx4* d1 = reinterpret_cast<floatx4*>(lds + st * stage_floats + s_row + RS);
#pragma unroll
        for (int q = 0; q < RS / 4; ++q) {
            d0[q] = floatx4{wv[8 * q], wv[8 * q + 2], wv[8 * q + 4], wv[8 * q + 6]};
            d1[q] = floatx4{wv[8 * q + 1], wv[8 * q + 3], wv[8 * q + 5], wv[8 * q + 7]};
        }
    };
    // x of the wave's features of chunk c (0 past in: their weights are 0)
    float xc[kFW], xn[kFW];
    auto load_x = [&](int c, float (&xv)[kFW]) {
        const int f0 = c * kNarrowFeat + kFW * wave;
#pragma unroll
        for (int j = 0; j < kFW; ++j) xv[j] = f0 + j < a.in ? xr[f0 + j] : 0.0f;
    };

    float acc[NO];
#pragma unroll
    for (int o = 0; o < NO; ++o) acc[o] = 0.0f;
    const float nbf = (float)a.nb;

    auto fma_row = [&](float v, const float* r) {
#pragma unroll
        for (int q = 0; q < NO / 4; ++q) {
            const floatx4 w = reinterpret_cast<const floatx4*>(r)[q];
            acc[4 * q] = __builtin_fmaf(v, w[0], acc[4 * q]);
            acc[4 * q + 1] = __builtin_fmaf(v, w[1], acc[4 * q + 1]);
            acc[4 * q + 2] = __builtin_fmaf(v, w[2], acc[4 * q + 2]);
            acc[4 * q + 3] = __builtin_fmaf(v, w[3], acc[4 * q + 3]);
        }
        if constexpr (NO % 4 != 0) {
            const floatx2 w = reinterpret_cast<const floatx2*>(r)[NO / 2 - 1];
            acc[NO - 2] = __builtin_fmaf(v, w[0], acc[NO - 2]);
            acc[NO - 1] = __builtin_fmaf(v, w[1], acc[NO - 1]);
        }
    };

    load_w(0);
    load_x(0, xc);
    store_w(0);
    __syncthreads();
    for (int c = 0; c < nchunks; ++c) {
        const bool more = c + 1 < nchunks;
        if (more) {
            load_w(c + 1);
            load_x(c + 1, xn);
        }
        const float* stg = lds + (c & 1) * stage_floats;
        // (one feature at a time: unrolled, the LDS rows of every feature
        // are loaded up front and the registers run out)
#pragma unroll 1
        for (int j = 0; j < kFW; ++j) {
            const float xv = xc[j];
            // v of column c is sv - c (column c is basis c - 1); the window
            // c0 .. c0 + 3 holds every basis with |v| < 2, c0 in [1, nb - 1]
            const float sv = __builtin_fmaf(xv, a.inv_h, a.a_int + 1.0f) +
                             coord_lo(xv, a.xlim, a.inv_lo, a.a_frac);
            const float f1 = __builtin_amdgcn_fmed3f(__builtin_floorf(sv), 2.0f, nbf);
            const int c0 = min(max((int)f1 - 1, 1), a.nb - 1);
            const float d = sv - (f1 - 1.0f);  // v of column c0
            const float* tb = stg + (kFW * wave + j) * cw * RS;
            fma_row(layer_detail::half_silu(xv), tb);
            const float* tw = tb + c0 * RS;
#pragma unroll
            for (int k = 0; k < 4; ++k) fma_row(half_basis(d - (float)k), tw + k * RS);
        }
        if (more) store_w((c + 1) & 1);
        __syncthreads();
        if (more) {
#pragma unroll
            for (int j = 0; j < kFW; ++j) xc[j] = xn[j];
        }
    }

    // The four waves' partial sums of each (row, output), added in wave
    // order; y = 2 sum (the operands carry N / 2 and silu / 2).
    float* red = lds;  // [wave][o][lane] (the stages are no longer read)
#pragma unroll
    for (int o = 0; o < NO; ++o) red[(wave * NO + o) * 64 + lane] = acc[o];
    __syncthreads();
    const int64_t nrows = a.batch - row0 < kNarrowRows ? a.batch - row0 : kNarrowRows;
    float* __restrict__ y = static_cast<float*>(a.y) + row0 * a.out;
    for (int i = tid; i < nrows * a.out; i += 256) {
        const int r = i / a.out;
        const int o = i - r * a.out;
        const float s = ((red[o * 64 + r] + red[(NO + o) * 64 + r]) + red[(2 * NO + o) * 64 + r]) +
                        red[(3 * NO + o) * 64 + r];
        y[i] = 2.0f * s;
    }
}

template <int NO>
hipError_t launch_no(const LayerArgs& a, int cw, hipStream_t s) {
    constexpr int RS = (NO + 3) / 4 * 4;
    const size_t stages = (size_t)2 * kNarrowFeat * cw * RS * sizeof(float);
    const size_t red = (size_t)4 * NO * 64 * sizeof(float);
    const size_t lds = stages > red ? stages : red;
    const unsigned blocks = (unsigned)((a.batch + kNarrowRows - 1) / kNarrowRows);
    hipLaunchKernelGGL(narrow_kernel<NO>, dim3(blocks), dim3(256), lds, s, a, cw);
    return hipGetLastError();
}

}  // namespace

bool narrow_ok(const LayerGeom& g) {
    // fp32 cubic layers of at most 16 outputs with at most 64 columns per
    // feature (G <= 58): two LDS stages of at most 64 KB, one staging unit
    // per thread
    return g.kj == 2 && g.kdeg == 3 && g.out >= 1 && g.out <= kNarrowMaxOut &&
           narrow_cols(g.nb) <= 64;
}

hipError_t launch_narrow(const LayerGeom& g, const LayerArgs& a, hipStream_t s) {
    if (!narrow_ok(g) || a.batch < 1) return hipErrorInvalidValue;
    const int cw = narrow_cols(g.nb);
    switch ((a.out + 1) & ~1) {
        case 2: return launch_no<2>(a, cw, s);
        case 4: return launch_no<4>(a, cw, s);
        case 6: return launch_no<6>(a, cw, s);
        case 8: return launch_no<8>(a, cw, s);
        case 10: return launch_no<10>(a, cw, s);
        case 12: return launch_no<12>(a, cw, s);
        case 14: return launch_no<14>(a, cw, s);
        case 16: return launch_no<16>(a, cw, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace kan
