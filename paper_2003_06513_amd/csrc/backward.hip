// Backward of the pattern-sparse layer for the user's retraining (Sec. 3.3:
// retraining is ordinary training except that the pruned weights' gradients
// are zero).  For y = W x (Eq. 1, stride 1, zero padding 1):
//
//  * dx = W^T dy is the same pattern-sparse convolution run on dy with the
//    transposed layer: filter ci, input channel f, each kernel rotated by
//    180 degrees.  A rotated 4-of-9 mask is another 4-of-9 mask (bit q ->
//    bit 8-q), so the transposed layer is an ordinary layer of the library of
//    rotated masks; k_transpose_prep writes its dense weights, pattern ids
//    and keep mask, psc_pack packs it, and the tuned forward kernels run it.
//  * dv, the gradient of the 4 stored values of each kept kernel (the masked
//    gradient: nothing for pruned weights), and db are reductions over the
//    batch and the image (wgrad.hip).
#include "common.h"
#include "launch.h"

namespace psc {
namespace {

template <typename B>
__global__ __launch_bounds__(256) void k_transpose_prep(const B* __restrict__ w, const uint8_t* __restrict__ pat,
                                                        const uint8_t* __restrict__ keep, int cout, int cin,
                                                        B* __restrict__ wt, uint8_t* __restrict__ pat_t,
                                                        uint8_t* __restrict__ keep_t) {
    const int64_t n = int64_t(cout) * cin;
    for (int64_t k = int64_t(blockIdx.x) * 256 + threadIdx.x; k < n; k += int64_t(gridDim.x) * 256) {
        const int f = int(k / cin), ci = int(k - int64_t(f) * cin);
        const int64_t kt = int64_t(ci) * cout + f;
#pragma unroll
        for (int q = 0; q < 9; ++q) wt[kt * 9 + q] = w[k * 9 + (8 - q)];   // bit copies, rotated
        pat_t[kt] = pat[k];
        keep_t[kt] = keep[k];
    }
}

int grid_cap(int64_t n, int cap) {
    const int64_t g = (n + 255) / 256;
    return int(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_transpose_prep(int dtype, int cout, int cin, const void* w, const uint8_t* pat,
                                 const uint8_t* keep, void* wt, uint8_t* pat_t, uint8_t* keep_t,
                                 hipStream_t stream) {
    const int64_t n = int64_t(cout) * cin;
    const dim3 grid(unsigned(grid_cap(n, 8192)));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_transpose_prep<uint16_t>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(w),
                           pat, keep, cout, cin, static_cast<uint16_t*>(wt), pat_t, keep_t);
    else
        hipLaunchKernelGGL(k_transpose_prep<uint32_t>, grid, dim3(256), 0, stream, static_cast<const uint32_t*>(w),
                           pat, keep, cout, cin, static_cast<uint32_t*>(wt), pat_t, keep_t);
    return hipGetLastError();
}

}  // namespace psc
