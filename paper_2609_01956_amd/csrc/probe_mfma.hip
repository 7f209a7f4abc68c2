// probe_mfma.hip -- measurement support, not part of the KAN ABI: the rate of
// back-to-back v_mfma_f32_32x32x16_bf16 on this device with constant or with
// random operands, and the shader clock while it runs; and the rate of plain
// (non-packed) fp32 VALU fmas per SIMD with 1, 2 or 4 waves on it.
//
// Each wave keeps 8 independent 32x32 fp32 accumulators and issues 16 MFMAs
// per loop trip (two A fragments, sixteen B fragments, all in registers), so
// the loop is nothing but matrix-core work.  Wave 0 of workgroup 0 reads the
// shader-clock counter (s_memtime) and the 100 MHz reference counter
// (s_memrealtime) at its start and end; their ratio is the average shader
// clock over the run.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kOperandWords = 64 * 16 + 64 * 2;  // u32x4 words read per workgroup

template <bool RANDOM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
void mfma_loop(const u32x4* __restrict__ operands, float* __restrict__ out,
               unsigned long long* __restrict__ clk, int trips) {
    const int lane = threadIdx.x & 63;
    const bool timer = blockIdx.x == 0 && threadIdx.x == 0;
    if (timer) {
        clk[0] = __builtin_amdgcn_s_memtime();
        clk[1] = __builtin_amdgcn_s_memrealtime();
    }
    floatx16 acc[8];
    for (int i = 0; i < 8; ++i)
        for (int q = 0; q < 16; ++q) acc[i][q] = 0.0f;
    bf16x8 A[2], B[16];
    for (int k = 0; k < 16; ++k)
        B[k] = __builtin_bit_cast(bf16x8, RANDOM ? operands[lane * 16 + k]
                                                 : u32x4{1u, 2u, 3u, (unsigned)k});
    for (int k = 0; k < 2; ++k)
        A[k] = __builtin_bit_cast(bf16x8, RANDOM ? operands[64 * 16 + lane * 2 + k]
                                                 : u32x4{0x3dcc3dccu, 0x3e4c3e4cu,
                                                         0x3e993e99u, 0x3ecc3eccu});
    for (int t = 0; t < trips; ++t) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[0], B[i], acc[i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[1], B[8 + i], acc[i], 0, 0, 0);
    }
    float r = 0.0f;
    for (int i = 0; i < 8; ++i)
        for (int q = 0; q < 16; ++q) r += acc[i][q];
    out[(size_t)blockIdx.x * 256 + threadIdx.x] = r;
    if (timer) {
        clk[2] = __builtin_amdgcn_s_memtime();
        clk[3] = __builtin_amdgcn_s_memrealtime();
    }
}

// W waves per SIMD (one workgroup of 4 W waves per CU), each running 8
// independent fp32 fma chains, 128 fmas per loop trip.  Every wave of
// workgroup 0 records its own start and end shader-clock counters, so the
// span over them is the time the SIMDs took for all their waves.
__global__ __launch_bounds__(1024) void valu_loop(float* __restrict__ out,
                                                  unsigned long long* __restrict__ clk,
                                                  int trips, float seed) {
    const int lane = threadIdx.x & 63;
    float v[8];
    for (int k = 0; k < 8; ++k) v[k] = seed * (float)(lane + k);
    const float c1 = 0.999f + seed, c2 = 0.001f * seed;
    const unsigned long long t0 = __builtin_amdgcn_s_memtime();
    for (int t = 0; t < trips; ++t) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = __builtin_fmaf(v[k], c1, c2);
    }
    const unsigned long long t1 = __builtin_amdgcn_s_memtime();
    float r = 0.0f;
    for (int k = 0; k < 8; ++k) r += v[k];
    out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = r;
    if (blockIdx.x == 0 && lane == 0) {
        clk[2 * (threadIdx.x >> 6)] = t0;
        clk[2 * (threadIdx.x >> 6) + 1] = t1;
    }
}

}  // namespace

// out: device, blocks * 256 * waves_per_simd floats; clk: device, 8 *
// waves_per_simd counters (start, end of each wave of workgroup 0).  Each wave
// issues 128 * trips fp32 fmas.  waves_per_simd is 1, 2 or 4.  Returns a
// hipError_t code.
extern "C" int kan_probe_valu_f32(void* out, void* clk, int blocks, int waves_per_simd, int trips,
                                  void* stream) {
    if (blocks <= 0 || trips <= 0 || !out || !clk ||
        (waves_per_simd != 1 && waves_per_simd != 2 && waves_per_simd != 4))
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(valu_loop, dim3(blocks), dim3(256 * waves_per_simd), 0,
                       static_cast<hipStream_t>(stream), static_cast<float*>(out),
                       static_cast<unsigned long long*>(clk), trips, 1e-3f);
    return (int)hipGetLastError();
}

// operands: device, at least kan_probe_operand_words() 16-byte words of
// finite bf16 values (read only with random != 0); out: device, blocks * 256
// floats; clk: device, 4 counters.  Each workgroup issues 4 waves x 16 x trips
// MFMAs of 32768 flops.  Returns a hipError_t code.
extern "C" int kan_probe_operand_words(void) { return kOperandWords; }

extern "C" int kan_probe_mfma_bf16(const void* operands, void* out, void* clk, int blocks,
                                   int trips, int random, void* stream) {
    if (blocks <= 0 || trips <= 0 || !out || !clk || (random && !operands))
        return (int)hipErrorInvalidValue;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (random)
        hipLaunchKernelGGL(mfma_loop<true>, dim3(blocks), dim3(256), 0, s,
                           static_cast<const u32x4*>(operands), static_cast<float*>(out),
                           static_cast<unsigned long long*>(clk), trips);
    else
        hipLaunchKernelGGL(mfma_loop<false>, dim3(blocks), dim3(256), 0, s,
                           static_cast<const u32x4*>(operands), static_cast<float*>(out),
                           static_cast<unsigned long long*>(clk), trips);
    return (int)hipGetLastError();
}
