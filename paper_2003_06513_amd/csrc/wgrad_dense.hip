// The dense weight gradient of a 3x3 layer (stride 1, zero padding 1) on the
// matrix cores, for the primal step of the data-free ADMM loop (Sec. 4.3,
// Eq. 4) and, gathered at the kept taps, for the masked gradient of batch-1
// layers (Sec. 3.3):
//   dW[f][c][q] = sum over images and pixels p of g[n, f, p] x[n, c, p + off(q)]
// is a GEMM with M = filters, N = (tap, input channel) and K = pixels,
// computed by fp32 MFMA 16x16x4 (fp16 x and g are widened exactly as they
// load, so both accumulate in fp32).  A block owns 64 filters x 16 channels x 9
// taps; each of its 4 waves owns 16 filters x 16 channels x 9 taps, i.e. one
// MFMA tile per tap.  K runs over 4x16 pixel tiles of the images: a tile's
// gradient values (transposed to [pixel][filter]) and its 16 input channels
// with a 1-pixel halo are staged through LDS, and per K step of 4 pixels a
// lane reads 1 gradient value and 9 shifted inputs for the 9 MFMAs.  The
// next tile's values load into registers while the current one computes;
// each step's LDS operands load while the previous step's MFMAs issue.
// The pixel tiles are split over KS blocks whose partial sums go to KS
// workspace slots, added afterwards in slot order (deterministic).
//
// Operand layout of v_mfma_f32_16x16x4_f32: lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; the result element D[i][j] sits in lane
// j + 16 (i / 4), register i % 4.  Here A[i][k] = g(filter i, pixel k) and
// B[k][j] = x(channel j, pixel k shifted by the tap).
#include "common.h"
#include "launch.h"

namespace psc {
namespace {

constexpr int kWF = 64;                 // filters per block
constexpr int kWC = 16;                 // channels per block
constexpr int kWTR = 4, kWTC = 16;      // pixel tile
constexpr int kWP = kWTR * kWTC;        // pixels per tile: 16 K steps of 4
constexpr int kWGS = 80;                // LDS stride (floats) of a pixel's gradient row [f]
constexpr int kWXR = kWTR + 2, kWXC = kWTC + 2;
constexpr int kWXE = kWXR * kWXC;       // 108 inputs per channel tile
constexpr int kWXS = 109;               // LDS stride (floats) of a channel's input tile
constexpr int kWGJ = kWF * kWP / 256;   // 16 gradient values per thread and tile
constexpr int kWXJ = (kWC * kWXE + 255) / 256;   // 7 inputs per thread and tile
constexpr int kWMaxKS = 64;             // workspace slots at most
constexpr int kWTargetBlocks = 512;

typedef float wf4 __attribute__((ext_vector_type(4)));

template <int DT>
__global__ __launch_bounds__(256) void k_wgrad_mfma(const typename Elt<DT>::T* __restrict__ x,
                                                    const typename Elt<DT>::T* __restrict__ g, int n, int cin, int H,
                                                    int W, int cout, int tiles_w, int tiles_img, int64_t tiles, int KS,
                                                    float* __restrict__ out) {
    using T = typename Elt<DT>::T;
    constexpr uint32_t ESZ = uint32_t(sizeof(T));
    __shared__ float gs[kWP * kWGS];
    __shared__ float xs[kWC * kWXS];
    const int f0 = blockIdx.x * kWF, c0 = blockIdx.y * kWC, ks = blockIdx.z;
    const int64_t t0 = tiles * ks / KS, t1 = tiles * (ks + 1) / KS;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int li = lane & 15, kq = lane >> 4;
    const int plane = H * W;
    // buffer descriptors: 32-bit offsets (x and g are below 2 GiB each);
    // elements outside the image, the channels or the filters sit past the
    // range and read zero
    const auto xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(x), int16_t(0),
                                                      int(int64_t(n) * cin * plane * ESZ), 0x00020000);
    const auto gr = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(g), int16_t(0),
                                                      int(int64_t(n) * cout * plane * ESZ), 0x00020000);
    // one element, widened to fp32 (fp16 exactly)
    auto ld = [&](__amdgpu_buffer_rsrc_t rs, uint32_t vo) -> float {
        if constexpr (DT == DT_F32)
            return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, int(vo), 0, 0));
        else
            return float(__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(rs, int(vo), 0, 0)));
    };
    float rg[kWGJ], rx[kWXJ];
    auto fetch = [&](int64_t t) {
        const int img = int(t / tiles_img), tt = int(t - int64_t(img) * tiles_img);
        const int th0 = (tt / tiles_w) * kWTR, tw0 = (tt % tiles_w) * kWTC;
#pragma unroll
        for (int j = 0; j < kWGJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            const int f = e / kWP, p = e % kWP;
            const int oh = th0 + p / kWTC, ow = tw0 + p % kWTC;
            const bool in = f0 + f < cout && oh < H && ow < W;
            const uint32_t vo = in ? (uint32_t(img * cout + f0 + f) * uint32_t(plane) + uint32_t(oh * W + ow)) * ESZ
                                   : 0x80000000u;
            rg[j] = ld(gr, vo);
        }
#pragma unroll
        for (int j = 0; j < kWXJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            const int c = e / kWXE, r = (e / kWXC) % kWXR, s = e % kWXC;
            const int ih = th0 + r - 1, iw = tw0 + s - 1;
            const bool in = c < kWC && c0 + c < cin && ih >= 0 && ih < H && iw >= 0 && iw < W;
            const uint32_t vo = in ? (uint32_t(img * cin + c0 + c) * uint32_t(plane) + uint32_t(ih * W + iw)) * ESZ
                                   : 0x80000000u;
            rx[j] = ld(xr, vo);
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int j = 0; j < kWGJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            gs[(e % kWP) * kWGS + e / kWP] = rg[j];
        }
#pragma unroll
        for (int j = 0; j < kWXJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            if (e < kWC * kWXE) xs[(e / kWXE) * kWXS + e % kWXE] = rx[j];
        }
    };
    // operands of K step st: the gradient of filter 16 wave + li at pixel
    // 4 st + kq, and channel li's inputs at that pixel shifted by each tap
    auto operands = [&](int st, float (&o)[10]) {
        const int p = 4 * st + kq;
        o[0] = gs[p * kWGS + 16 * wave + li];
        const int base = li * kWXS + (p / kWTC) * kWXC + p % kWTC;
#pragma unroll
        for (int q = 0; q < 9; ++q) o[1 + q] = xs[base + (q / 3) * kWXC + q % 3];
    };
    wf4 acc[9];
#pragma unroll
    for (int q = 0; q < 9; ++q) acc[q] = wf4{0.f, 0.f, 0.f, 0.f};
    auto mfma9 = [&](const float (&o)[10]) {
#pragma unroll
        for (int q = 0; q < 9; ++q) acc[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(o[0], o[1 + q], acc[q], 0, 0, 0);
    };

    if (t0 < t1) fetch(t0);
    for (int64_t t = t0; t < t1; ++t) {
        stage();
        __syncthreads();
        if (t + 1 < t1) fetch(t + 1);   // in flight during this tile's MFMAs
        float oa[10], ob[10];
        operands(0, oa);
#pragma unroll
        for (int st = 0; st < kWP / 4; st += 2) {
            operands(st + 1, ob);
            mfma9(oa);
            if (st + 2 < kWP / 4) operands(st + 2, oa);
            mfma9(ob);
        }
        __syncthreads();
    }
    // D[i][j] of tap q: filter f0 + 16 wave + 4 kq + r, channel c0 + li
    float* dst = out + (KS > 1 ? int64_t(ks) * cout * cin * 9 : 0);
    const int c = c0 + li;
    if (c >= cin) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int f = f0 + 16 * wave + 4 * kq + r;
        if (f >= cout) continue;
#pragma unroll
        for (int q = 0; q < 9; ++q) dst[(int64_t(f) * cin + c) * 9 + q] = acc[q][r];
    }
}

// The masked weight gradient (Sec. 3.3) from a dense one: for stored kernel
// k of reordered filter i (original filter perm[i], channel cin_idx[k],
// library pattern pat_id[k]), dv[4k + j] = dw[perm[i]][cin_idx[k]][q_j], q_j
// the j-th kept position of the pattern in ascending order -- the order of
// the stored weights.  One block per reordered filter.  A malformed channel
// or pattern index gives zeros, a malformed filter index reads filter 0.
__global__ __launch_bounds__(256) void k_gather_masked(const float* __restrict__ dw, const int32_t* __restrict__ perm,
                                                       const int32_t* __restrict__ filter_ptr,
                                                       const int32_t* __restrict__ cin_idx,
                                                       const uint8_t* __restrict__ pat_id, PatTable tab, int cin,
                                                       int cout, float* __restrict__ dv) {
    const int i = blockIdx.x;
    const int f = perm[i] >= 0 && perm[i] < cout ? perm[i] : 0;
    const int k0 = filter_ptr[i], k1 = filter_ptr[i + 1];
    for (int k = k0 + int(threadIdx.x); k < k1; k += 256) {
        const int c = cin_idx[k], p = pat_id[k];
        const unsigned mask = (c >= 0 && c < cin && p < tab.m) ? tab.mask[p] : 0u;
        const float* src = dw + (int64_t(f) * cin + (c >= 0 && c < cin ? c : 0)) * 9;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        int j = 0;
        for (int q = 0; q < 9; ++q)
            if (((mask >> q) & 1u) && j < 4) v[j++] = src[q];
#pragma unroll
        for (int t = 0; t < 4; ++t) dv[int64_t(k) * 4 + t] = v[t];
    }
}

}  // namespace

// Layers of at least 16 input channels (a full MFMA tile of channels).
bool dense_wgrad_mfma_plan(int n, int cin, int cout, int h, int w, DenseWPlan* p) {
    if (cin < kWC || n <= 0 || cout <= 0 || h <= 0 || w <= 0) return false;
    DenseWPlan q{};
    q.fb = (cout + kWF - 1) / kWF;
    q.cb = (cin + kWC - 1) / kWC;
    q.tiles_w = (w + kWTC - 1) / kWTC;
    q.tiles_img = ((h + kWTR - 1) / kWTR) * q.tiles_w;
    q.tiles = int64_t(n) * q.tiles_img;
    int64_t ks = kWTargetBlocks / (int64_t(q.fb) * q.cb);
    if (ks > kWMaxKS) ks = kWMaxKS;
    if (ks > q.tiles) ks = q.tiles;
    q.KS = int(ks < 1 ? 1 : ks);
    if (p) *p = q;
    return true;
}

size_t dense_wgrad_mfma_workspace(const DenseWPlan& p, int cin, int cout) {
    return p.KS > 1 ? size_t(p.KS) * size_t(cout) * size_t(cin) * 9 * sizeof(float) : 0;
}

hipError_t launch_dense_wgrad_mfma(const DenseWPlan& p, int dtype, const void* x, const void* g, int n, int cin,
                                   int h, int w, int cout, float* dst, hipStream_t stream) {
    const dim3 grid(unsigned(p.fb), unsigned(p.cb), unsigned(p.KS));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_wgrad_mfma<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x),
                           static_cast<const uint16_t*>(g), n, cin, h, w, cout, p.tiles_w, p.tiles_img, p.tiles, p.KS,
                           dst);
    else
        hipLaunchKernelGGL(k_wgrad_mfma<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x),
                           static_cast<const float*>(g), n, cin, h, w, cout, p.tiles_w, p.tiles_img, p.tiles, p.KS,
                           dst);
    return hipGetLastError();
}

}  // namespace psc

namespace psc {
hipError_t launch_gather_masked(const PatTable& tab, const PackedView& pk, int cout, int cin, const float* dw,
                                float* dv, hipStream_t stream) {
    hipLaunchKernelGGL(k_gather_masked, dim3(unsigned(cout)), dim3(256), 0, stream, dw, pk.filter_perm, pk.filter_ptr,
                       pk.cin_idx, pk.pat_id, tab, cin, cout, dv);
    return hipGetLastError();
}
}  // namespace psc
