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
//    batch and the image: k_bwd_weight gives one wave to each kept kernel,
//    k_bias_grad one block to each filter.
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

// One wave per kept kernel k (storage order): dv[4k + t] = sum over images,
// rows and columns of dy[n, f, i, j] * x[n, ci, i + r_t - 1, j + s_t - 1].
// A wave covers RPI = max(1, 64 / W) output rows of up to 64 columns per
// step (W > 64: 64-column tiles); the 4 partial sums of each lane are added
// across the wave at the end.  fp32 accumulation.
template <int DT>
__global__ __launch_bounds__(256) void k_bwd_weight(const typename Elt<DT>::T* __restrict__ x,
                                                    const typename Elt<DT>::T* __restrict__ dy, int n, int cin,
                                                    int H, int W, int cout, PatTable tab,
                                                    const int32_t* __restrict__ perm,
                                                    const int32_t* __restrict__ fptr,
                                                    const int32_t* __restrict__ cin_idx,
                                                    const uint8_t* __restrict__ pat_id, int64_t keep,
                                                    float* __restrict__ dv) {
    using E = Elt<DT>;
    const int lane = threadIdx.x & 63;
    const int64_t k = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (k >= keep) return;                                   // whole waves leave together
    // the filter holding kernel k: the last i with fptr[i] <= k
    int lo = 0, hi = cout - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (fptr[mid] <= k) lo = mid;
        else hi = mid - 1;
    }
    const int f = perm[lo];
    const int ci = cin_idx[k], p = pat_id[k];
    if (unsigned(ci) >= unsigned(cin) || p >= tab.m) return;   // malformed storage
    int dr[4], dc[4], t = 0;
    const unsigned mk = tab.mask[p];
    for (int q = 0; q < 9; ++q)
        if ((mk >> q) & 1u) {
            if (t < 4) {
                dr[t] = q / 3 - 1;
                dc[t] = q % 3 - 1;
            }
            ++t;
        }
    const int rpi = W >= 64 ? 1 : 64 / W;                    // output rows per step
    const int cw = W >= 64 ? 64 : W;                         // columns per row slot
    const int lr = lane / cw, lc = lane - lr * cw;
    const int plane = H * W;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (lr < rpi) {
        for (int nn = 0; nn < n; ++nn) {
            const typename E::T* xc = x + (int64_t(nn) * cin + ci) * plane;
            const typename E::T* yc = dy + (int64_t(nn) * cout + f) * plane;
            for (int i0 = 0; i0 < H; i0 += rpi) {
                const int i = i0 + lr;
                if (i >= H) continue;
                for (int j = lc; j < W; j += cw) {
                    const float g = E::load(yc, i * W + j);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int ii = i + dr[u], jj = j + dc[u];
                        const float xv = (ii >= 0 && ii < H && jj >= 0 && jj < W) ? E::load(xc, ii * W + jj) : 0.f;
                        acc[u] = fmaf(g, xv, acc[u]);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        float v = acc[u];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
        acc[u] = v;
    }
    if (lane == 0) {
        float4 o{acc[0], acc[1], acc[2], acc[3]};
        *reinterpret_cast<float4*>(dv + k * 4) = o;
    }
}

// db[f] = sum over images and pixels of dy[n, f]; one block per filter.
template <int DT>
__global__ __launch_bounds__(256) void k_bias_grad(const typename Elt<DT>::T* __restrict__ dy, int n, int cout,
                                                   int plane, float* __restrict__ db) {
    using E = Elt<DT>;
    __shared__ float part[4];
    const int f = blockIdx.x;
    float acc = 0.f;
    for (int nn = 0; nn < n; ++nn) {
        const typename E::T* yc = dy + (int64_t(nn) * cout + f) * plane;
        for (int q = threadIdx.x; q < plane; q += 256) acc += E::load(yc, q);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) db[f] = (part[0] + part[1]) + (part[2] + part[3]);
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

hipError_t launch_bwd_weight(const PatTable& tab, const PackedView& pk, int dtype, int n, int cin, int h, int w,
                             int cout, int64_t keep, const void* x, const void* dy, float* dv, float* db,
                             hipStream_t stream) {
    if (keep > 0) {
        const dim3 grid(unsigned((keep + 3) / 4));
        if (dtype == DT_F16)
            hipLaunchKernelGGL(k_bwd_weight<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x),
                               static_cast<const uint16_t*>(dy), n, cin, h, w, cout, tab, pk.filter_perm,
                               pk.filter_ptr, pk.cin_idx, pk.pat_id, keep, dv);
        else
            hipLaunchKernelGGL(k_bwd_weight<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x),
                               static_cast<const float*>(dy), n, cin, h, w, cout, tab, pk.filter_perm,
                               pk.filter_ptr, pk.cin_idx, pk.pat_id, keep, dv);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (db) {
        if (dtype == DT_F16)
            hipLaunchKernelGGL(k_bias_grad<DT_F16>, dim3(unsigned(cout)), dim3(256), 0, stream,
                               static_cast<const uint16_t*>(dy), n, cout, h * w, db);
        else
            hipLaunchKernelGGL(k_bias_grad<DT_F32>, dim3(unsigned(cout)), dim3(256), 0, stream,
                               static_cast<const float*>(dy), n, cout, h * w, db);
    }
    return hipGetLastError();
}

}  // namespace psc
