// probe_mfma.hip -- measurement support, not part of the KAN ABI: the rate of
// back-to-back v_mfma_f32_32x32x16_bf16 on this device with constant or with
// random operands, and the shader clock while it runs.
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

}  // namespace

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
