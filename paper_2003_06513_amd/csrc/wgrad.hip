// Weight gradients of the 3x3 layer (stride 1, zero padding 1): for a kernel
// (f, ci) and each of its taps t at position (r_t, s_t),
//
//   dW_t = sum over images and output pixels (i, j) of
//          dy[n, f, i, j] * x[n, ci, i + r_t - 1, j + s_t - 1].
//
// Used for the masked gradient of the retraining function (Sec. 3.3: the 4
// stored values of each kept kernel, nothing for pruned weights) and for the
// dense gradient of the ADMM primal step (Sec. 4.3 Eq. 4: all 9 positions
// of every (f, ci)).
//
// Layout of the work: one wave per kernel and share of the image.  As in the
// forward kernels, a lane owns one column and R rows of an output band (a
// wave holds S bands of full rows separated by a zero lane, or a column tile
// with one halo lane on each side); per band it loads its R rows of dy and
// the R+2 rows of x around them once, takes the left/right neighbour columns
// of x from the adjacent lanes by DPP, and accumulates every tap's products
// in a register of its own.  The bands of a share are walked in turn, and
// the per-lane sums are added across the wave once at the end.  With several
// shares per kernel the share sums go to a workspace and a second kernel
// adds them in share order, so results do not depend on scheduling.
#include "common.h"
#include "launch.h"

namespace psc {
namespace {

struct WGeo {
    int n, cin, cout, H, W;
    int S;          // bands (segments) per wave
    int seg_len;    // lanes per segment
    int Wt;         // output columns per segment
    int cols_mode;  // 0: full-row segments with zero separators, 1: haloed column tiles
    int RB, CT;     // row bands and column tiles per image
    int units;      // n * RB * CT
    int slots;      // waves' worth of units: ceil(units / S)
    int KS;         // shares of the slots per kernel
    int64_t nk;     // kernels
    int dense;      // 1: kernel k is (k / cin, k % cin) with all 9 taps
    int m;
    uint16_t mask[kMaxPatterns];
};

constexpr int kDppShr = 0x138;   // wave_shr:1 -- lane i reads lane i-1
constexpr int kDppShl = 0x130;   // wave_shl:1 -- lane i reads lane i+1

__device__ __forceinline__ float dpp_shift(float v, int ctrl_is_shr) {
    const int iv = __builtin_bit_cast(int, v);
    const int r = ctrl_is_shr ? __builtin_amdgcn_update_dpp(0, iv, kDppShr, 0xf, 0xf, true)
                              : __builtin_amdgcn_update_dpp(0, iv, kDppShl, 0xf, 0xf, true);
    return __builtin_bit_cast(float, r);
}

// acc += sum_r dy[r] * xs[r + DR] for one tap (DR: row offset 0..2).
template <int R, int DR>
__device__ __forceinline__ void tap_rows(float& acc, const float (&dyr)[R], const float (&xs)[R + 2]) {
#pragma unroll
    for (int r = 0; r < R; ++r) acc = fmaf(dyr[r], xs[r + DR], acc);
}

template <int R>
__device__ __forceinline__ void tap_dyn(int q, float& acc, const float (&dyr)[R], const float (&xl)[R + 2],
                                        const float (&xc)[R + 2], const float (&xr)[R + 2]) {
    switch (q) {
        case 0: tap_rows<R, 0>(acc, dyr, xl); break;
        case 1: tap_rows<R, 0>(acc, dyr, xc); break;
        case 2: tap_rows<R, 0>(acc, dyr, xr); break;
        case 3: tap_rows<R, 1>(acc, dyr, xl); break;
        case 4: tap_rows<R, 1>(acc, dyr, xc); break;
        case 5: tap_rows<R, 1>(acc, dyr, xr); break;
        case 6: tap_rows<R, 2>(acc, dyr, xl); break;
        case 7: tap_rows<R, 2>(acc, dyr, xc); break;
        default: tap_rows<R, 2>(acc, dyr, xr); break;
    }
}

// NT = 4 (the kept positions of a pattern, dispatched per tap) or 9 (dense).
template <int DT, int R, int NT>
__global__ __launch_bounds__(256) void k_wgrad(const typename Elt<DT>::T* __restrict__ x,
                                               const typename Elt<DT>::T* __restrict__ dy,
                                               const int32_t* __restrict__ perm, const int32_t* __restrict__ fptr,
                                               const int32_t* __restrict__ cin_idx,
                                               const uint8_t* __restrict__ pat_id, WGeo g, float* __restrict__ out) {
    using E = Elt<DT>;
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t k = wid / g.KS;
    const int s = int(wid - k * g.KS);
    if (k >= g.nk) return;                                   // whole waves leave together
    int f, ci;
    int q[NT];
    if (g.dense) {
        f = int(k / g.cin);
        ci = int(k - int64_t(f) * g.cin);
#pragma unroll
        for (int t = 0; t < NT; ++t) q[t] = t;
    } else {
        // the filter holding kernel k: the last i with fptr[i] <= k
        int lo = 0, hi = g.cout - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (fptr[mid] <= k) lo = mid;
            else hi = mid - 1;
        }
        f = perm[lo];
        ci = cin_idx[k];
        const int p = pat_id[k];
        const unsigned mk = p < g.m ? g.mask[p] : 0u;
        int t = 0;
#pragma unroll
        for (int u = 0; u < NT; ++u) q[u] = 4;
        for (int u = 0; u < 9; ++u)
            if ((mk >> u) & 1u) {
                if (t < NT) q[t] = u;
                ++t;
            }
        if (unsigned(ci) >= unsigned(g.cin) || p >= g.m || t != NT) ci = -1;   // malformed storage: no terms
    }
    const int seg = lane / g.seg_len, cidx = lane - seg * g.seg_len;
    const int plane = g.H * g.W;
    float acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = 0.f;
    const int sl0 = int(int64_t(g.slots) * s / g.KS), sl1 = int(int64_t(g.slots) * (s + 1) / g.KS);
    for (int sl = sl0; sl < sl1; ++sl) {
        const int u = sl * g.S + seg;
        int ld_col = -1, out_col = -1, nimg = 0, h0 = 0;
        if (seg < g.S && u < g.units && ci >= 0) {
            nimg = u / (g.RB * g.CT);
            const int rb = (u / g.CT) % g.RB, ct = u % g.CT;
            h0 = rb * R;
            if (!g.cols_mode) {
                if (cidx < g.W) ld_col = out_col = cidx;
            } else {
                const int col = ct * g.Wt + cidx - 1;
                if (col >= 0 && col < g.W) ld_col = col;
                if (cidx >= 1 && cidx <= g.Wt && col < g.W) out_col = col;
            }
        }
        float dyr[R], xc[R + 2], xl[R + 2], xr[R + 2];
        const typename E::T* yp = dy + (int64_t(nimg) * g.cout + f) * plane;
        const typename E::T* xp = x + (int64_t(nimg) * g.cin + (ci < 0 ? 0 : ci)) * plane;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = h0 + r;
            dyr[r] = (out_col >= 0 && row < g.H) ? E::load(yp, row * g.W + out_col) : 0.f;
        }
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            const int row = h0 - 1 + r;
            xc[r] = (ld_col >= 0 && row >= 0 && row < g.H) ? E::load(xp, row * g.W + ld_col) : 0.f;
        }
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            xl[r] = dpp_shift(xc[r], 1);
            xr[r] = dpp_shift(xc[r], 0);
        }
        if constexpr (NT == 9) {
            tap_rows<R, 0>(acc[0], dyr, xl);
            tap_rows<R, 0>(acc[1], dyr, xc);
            tap_rows<R, 0>(acc[2], dyr, xr);
            tap_rows<R, 1>(acc[3], dyr, xl);
            tap_rows<R, 1>(acc[4], dyr, xc);
            tap_rows<R, 1>(acc[5], dyr, xr);
            tap_rows<R, 2>(acc[6], dyr, xl);
            tap_rows<R, 2>(acc[7], dyr, xc);
            tap_rows<R, 2>(acc[8], dyr, xr);
        } else {
#pragma unroll
            for (int t = 0; t < NT; ++t) tap_dyn<R>(q[t], acc[t], dyr, xl, xc, xr);
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float v = acc[t];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
        acc[t] = v;
    }
    if (lane == 0) {
        float* o = out + (int64_t(s) * g.nk + k) * NT;
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] = acc[t];
    }
}

// out[e] = sum over shares s (in order) of part[s][e].
__global__ __launch_bounds__(256) void k_wgrad_reduce(const float* __restrict__ part, int KS, int64_t n,
                                                      float* __restrict__ out) {
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256) {
        float v = part[e];
        for (int s = 1; s < KS; ++s) v += part[int64_t(s) * n + e];
        out[e] = v;
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

constexpr int kTargetWaves = 32768;
constexpr int kMaxShares = 64;

WGeo plan(int n, int cin, int cout, int h, int w, int64_t nk, bool dense, const PatTable* tab) {
    WGeo g{};
    g.n = n;
    g.cin = cin;
    g.cout = cout;
    g.H = h;
    g.W = w;
    g.nk = nk;
    g.dense = dense ? 1 : 0;
    g.m = tab ? tab->m : 0;
    for (int p = 0; p < kMaxPatterns; ++p) g.mask[p] = (tab && p < tab->m) ? tab->mask[p] : 0;
    if (w <= 63) {
        g.cols_mode = 0;
        g.seg_len = w + 1;
        g.S = 65 / (w + 1);
        g.Wt = w;
        g.CT = 1;
    } else {
        g.cols_mode = 1;
        g.Wt = 62;
        g.seg_len = 64;
        g.S = 1;
        g.CT = (w + 61) / 62;
    }
    const int R = h >= 8 ? 8 : 4;
    g.RB = (h + R - 1) / R;
    g.units = n * g.RB * g.CT;
    g.slots = (g.units + g.S - 1) / g.S;
    int64_t ks = nk > 0 ? (kTargetWaves + nk - 1) / nk : 1;
    if (ks > g.slots) ks = g.slots;
    if (ks > kMaxShares) ks = kMaxShares;
    g.KS = int(ks < 1 ? 1 : ks);
    return g;
}

template <int DT, int NT>
hipError_t run(const WGeo& g, const void* x, const void* dy, const int32_t* perm, const int32_t* fptr,
               const int32_t* cin_idx, const uint8_t* pat_id, float* out, void* ws, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    if (g.nk == 0) return hipSuccess;
    float* dst = g.KS > 1 ? static_cast<float*>(ws) : out;
    const dim3 grid(unsigned((g.nk * g.KS + 3) / 4));
    if (g.H >= 8)
        hipLaunchKernelGGL((k_wgrad<DT, 8, NT>), grid, dim3(256), 0, stream, static_cast<const T*>(x),
                           static_cast<const T*>(dy), perm, fptr, cin_idx, pat_id, g, dst);
    else
        hipLaunchKernelGGL((k_wgrad<DT, 4, NT>), grid, dim3(256), 0, stream, static_cast<const T*>(x),
                           static_cast<const T*>(dy), perm, fptr, cin_idx, pat_id, g, dst);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || g.KS == 1) return e;
    const int64_t n = g.nk * NT;
    const int64_t gb = (n + 255) / 256;
    hipLaunchKernelGGL(k_wgrad_reduce, dim3(unsigned(gb > 8192 ? 8192 : gb)), dim3(256), 0, stream, dst, g.KS, n,
                       out);
    return hipGetLastError();
}

template <int DT>
hipError_t bias_grad(const void* dy, int n, int cout, int plane, float* db, hipStream_t stream) {
    hipLaunchKernelGGL(k_bias_grad<DT>, dim3(unsigned(cout)), dim3(256), 0, stream,
                       static_cast<const typename Elt<DT>::T*>(dy), n, cout, plane, db);
    return hipGetLastError();
}

}  // namespace

size_t wgrad_workspace_bytes(int n, int cin, int cout, int h, int w, int64_t nk, bool dense) {
    const WGeo g = plan(n, cin, cout, h, w, nk, dense, nullptr);
    return g.KS > 1 ? size_t(g.KS) * size_t(nk) * (dense ? 9 : 4) * sizeof(float) : 0;
}

hipError_t launch_bwd_weight(const PatTable& tab, const PackedView& pk, int dtype, int n, int cin, int h, int w,
                             int cout, int64_t keep, const void* x, const void* dy, float* dv, float* db, void* ws,
                             hipStream_t stream) {
    const WGeo g = plan(n, cin, cout, h, w, keep, false, &tab);
    hipError_t e = dtype == DT_F16
                       ? run<DT_F16, 4>(g, x, dy, pk.filter_perm, pk.filter_ptr, pk.cin_idx, pk.pat_id, dv, ws, stream)
                       : run<DT_F32, 4>(g, x, dy, pk.filter_perm, pk.filter_ptr, pk.cin_idx, pk.pat_id, dv, ws, stream);
    if (e != hipSuccess || !db) return e;
    return dtype == DT_F16 ? bias_grad<DT_F16>(dy, n, cout, h * w, db, stream)
                           : bias_grad<DT_F32>(dy, n, cout, h * w, db, stream);
}

hipError_t launch_dense_wgrad(const float* x, const float* g_, int n, int cin, int h, int w, int cout, float* dw,
                              float* db, void* ws, hipStream_t stream) {
    const WGeo g = plan(n, cin, cout, h, w, int64_t(cout) * cin, true, nullptr);
    hipError_t e = run<DT_F32, 9>(g, x, g_, nullptr, nullptr, nullptr, nullptr, dw, ws, stream);
    if (e != hipSuccess || !db) return e;
    return bias_grad<DT_F32>(g_, n, cout, h * w, db, stream);
}

}  // namespace psc
