// Measurement probe (not part of the method): the vector-ALU fp32 FMA rate
// the library's kernels can issue, for the roofline of the conv kernels.  Each lane runs
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

}  // namespace

hipError_t launch_probe_fma(int blocks, int iters, float* out, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_fma, dim3(unsigned(blocks)), dim3(256), 0, stream, iters, 1.0000001f, 1e-7f, out);
    return hipGetLastError();
}

}  // namespace psc
