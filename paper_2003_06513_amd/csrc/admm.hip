// Kernels of the data-free ADMM pattern pruning of one layer (Sec. 4.3,
// Eq. 4-7; Algorithm 1).  One iteration on the GPU is
//
//   Z = W X + b                    psc_dense3x3_fwd (the pre-trained target
//                                  X' = relu(W0 X + b0) the same way)
//   G, loss                        k_admm_residual: G = 2c (relu(Z) - X')[Z > 0]
//   dW, db                         the dense weight gradient (wgrad.hip)
//   W, b, V = W + D                k_admm_primal: the SGD step of Eq. 4
//   pattern ids, keep mask         psc_project + psc_select on V (Eq. 6)
//   A, D                           k_admm_dual: A = V on the kept pattern
//                                  positions, 0 elsewhere; D = V - A (Eq. 7)
//
// All in fp32 (the training precision); the loss is summed in fp64.
#include "common.h"
#include "launch.h"

// Each rounding is the one the code writes (the steps are checked against
// the oracle's fp64 arithmetic with per-step bounds).
#pragma clang fp contract(off)

namespace psc {
namespace {

constexpr int kResBlocks = 1024;   // partial sums of the loss (fixed: deterministic order)

__global__ __launch_bounds__(256) void k_admm_residual(const float* __restrict__ z, const float* __restrict__ t,
                                                       int64_t numel, float two_c, float* __restrict__ g,
                                                       double* __restrict__ partial) {
    __shared__ double part[4];
    double acc = 0.0;
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < numel; i += int64_t(gridDim.x) * 256) {
        const float zv = z[i];
        const float e = (zv > 0.f ? zv : 0.f) - t[i];
        g[i] = zv > 0.f ? two_c * e : 0.f;
        acc += double(e) * double(e);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = (part[0] + part[1]) + (part[2] + part[3]);
}

__global__ __launch_bounds__(256) void k_sum_partials(const double* __restrict__ partial, int nb, double c,
                                                      double* __restrict__ out) {
    __shared__ double part[256];
    double acc = 0.0;
    for (int i = threadIdx.x; i < nb; i += 256) acc += partial[i];
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = c * part[0];
}

// The SGD step of Eq. 4 on W (gradient dW + rho (W - A + D)) and on b, and
// V = W + D for the projection.
__global__ __launch_bounds__(256) void k_admm_primal(float* __restrict__ w, const float* __restrict__ dw,
                                                     const float* __restrict__ a, const float* __restrict__ d,
                                                     int64_t nw, float* __restrict__ b, const float* __restrict__ db,
                                                     int cout, float lr, float rho, float* __restrict__ v) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < nw; i += int64_t(gridDim.x) * 256) {
        const float wi = w[i], di = d[i];
        const float pen = rho * ((wi - a[i]) + di);
        const float wn = wi - lr * (dw[i] + pen);
        w[i] = wn;
        v[i] = wn + di;
    }
    if (b && blockIdx.x == 0)
        for (int o = threadIdx.x; o < cout; o += 256) b[o] = b[o] - lr * db[o];
}

// Eq. 6 given the projection's choices (pattern ids, keep mask of V) and
// Eq. 7: A = V at the kept pattern positions, 0 elsewhere; D = V - A.
__global__ __launch_bounds__(256) void k_admm_dual(const float* __restrict__ v, const uint8_t* __restrict__ pat,
                                                   const uint8_t* __restrict__ keep, int64_t nk, PatTable tab,
                                                   float* __restrict__ a, float* __restrict__ d) {
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < nk * 9; e += int64_t(gridDim.x) * 256) {
        const int64_t k = e / 9;
        const int q = int(e - k * 9);
        const int p = pat[k];
        const bool on = keep[k] && p < tab.m && ((tab.mask[p] >> q) & 1u);
        const float vi = v[e];
        const float ai = on ? vi : 0.f;
        a[e] = ai;
        d[e] = vi - ai;
    }
}

int grid_of(int64_t n, int cap) {
    const int64_t g = (n + 255) / 256;
    return int(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

size_t admm_residual_workspace_bytes() { return size_t(kResBlocks) * sizeof(double); }

hipError_t launch_admm_residual(const float* z, const float* t, int64_t numel, float scale, float* g,
                                double* loss, void* ws, hipStream_t stream) {
    double* partial = static_cast<double*>(ws);
    const int nb = numel > 0 ? grid_of((numel + 7) / 8, kResBlocks) : 1;
    hipLaunchKernelGGL(k_admm_residual, dim3(unsigned(nb)), dim3(256), 0, stream, z, t, numel, 2.0f * scale, g,
                       partial);
    hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(256), 0, stream, partial, nb, double(scale), loss);
    return hipGetLastError();
}

hipError_t launch_admm_primal(float* w, const float* dw, const float* a, const float* d, int64_t nw, float* b,
                              const float* db, int cout, float lr, float rho, float* v, hipStream_t stream) {
    hipLaunchKernelGGL(k_admm_primal, dim3(unsigned(grid_of(nw, 4096))), dim3(256), 0, stream, w, dw, a, d, nw, b,
                       db, cout, lr, rho, v);
    return hipGetLastError();
}

hipError_t launch_admm_dual(const PatTable& tab, const float* v, const uint8_t* pat, const uint8_t* keep, int64_t nk,
                            float* a, float* d, hipStream_t stream) {
    hipLaunchKernelGGL(k_admm_dual, dim3(unsigned(grid_of(nk * 9, 4096))), dim3(256), 0, stream, v, pat, keep, nk,
                       tab, a, d);
    return hipGetLastError();
}

}  // namespace psc
