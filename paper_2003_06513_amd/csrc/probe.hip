// Measurement probes (not part of the method): the vector-ALU fp32 FMA rate
// the library's kernels can issue, for the roofline of the conv kernels, and
// the fp32 matrix-core rate, for the roofline of the dense kernels.  Each lane runs
// 8 independent chains of v_fmac_f32 (the library is compiled with packed fp32
// disabled); the result is stored so nothing is elided.
#include "common.h"
#include "launch.h"

namespace psc {
namespace {

__global__ __launch_bounds__(256) void k_probe_fma(int iters, float b, float c, float* __restrict__ out) {
    float a[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = float(threadIdx.x + j);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("v_fmac_f32_e32 %0, %1, %2" : "+v"(a[j]) : "v"(b), "v"(c));
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += a[j];
    out[int64_t(blockIdx.x) * 256 + threadIdx.x] = s;
}

// The fp32 matrix-core rate (v_mfma_f32_16x16x4_f32, the instruction of the
// dense kernels): each wave runs 4 independent accumulator chains.  With A
// all a and B all b every MFMA adds 4ab to each of a chain's 16x16 results.
__global__ __launch_bounds__(256) void k_probe_mfma(int iters, float a, float b, float* __restrict__ out) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    f4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) s += (acc[j].x + acc[j].y) + (acc[j].z + acc[j].w);
    out[int64_t(blockIdx.x) * 256 + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_probe_mfma(int blocks, int iters, float* out, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_mfma, dim3(unsigned(blocks)), dim3(256), 0, stream, iters, 1.0f, 0.25f, out);
    return hipGetLastError();
}

hipError_t launch_probe_fma(int blocks, int iters, float* out, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_fma, dim3(unsigned(blocks)), dim3(256), 0, stream, iters, 1.0000001f, 1e-7f, out);
    return hipGetLastError();
}

}  // namespace psc
