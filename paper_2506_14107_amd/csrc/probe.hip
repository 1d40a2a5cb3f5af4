// Measurement probe: the bf16 MFMA rate the chip sustains, the ceiling the packed GEMMs are
// compared with beside the nominal peak.
#include "dv_internal.h"

namespace dv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline float hash_unit(unsigned v) {   // a value in [-1, 1) from an integer hash
    v ^= v >> 16; v *= 0x7feb352du; v ^= v >> 15; v *= 0x846ca68bu; v ^= v >> 16;
    return (float)(v >> 8) * (2.0f / 16777216.0f) - 1.0f;
}

// Sustained bf16 MFMA rate of the chip: four independent accumulator chains per wavefront of
// v_mfma_f32_32x32x16_bf16 (enough to cover the instruction's dependent-issue latency), each
// chain with its own random operands so that consecutive instructions see different inputs (as
// in a GEMM; constant operands draw less power and run at a higher clock), operands in
// registers, no memory traffic in the loop; one value per lane is stored so the chains are
// live.  32768 FLOP per instruction.
__global__ __launch_bounds__(256) void mfma_loop_k(int iters, float* sink) {
    const unsigned t = blockIdx.x * 256u + threadIdx.x;
    bf16x8 x[4], y[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            x[k][e] = (__bf16)hash_unit(t * 64u + k * 16u + e);
            y[k][e] = (__bf16)hash_unit(t * 64u + k * 16u + 8u + e);
        }
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int i = 0; i < iters; ++i) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[0], y[0], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[1], y[1], c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[2], y[2], c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[3], y[3], c3, 0, 0, 0);
    }
    float v = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) v += c0[e] + c1[e] + c2[e] + c3[e];
    sink[(size_t)blockIdx.x * 256 + threadIdx.x] = v;
}

}  // namespace

double launch_mfma_loop(int blocks, int iters, float* sink, hipStream_t s) {
    hipLaunchKernelGGL(mfma_loop_k, dim3(blocks), dim3(256), 0, s, iters, sink);
    return (double)blocks * 4 * 4 * (double)iters * 32768.0;
}

}  // namespace dv
