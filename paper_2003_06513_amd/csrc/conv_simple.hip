// Straightforward kernels: the one-output-per-lane pattern-sparse conv (a
// second implementation of Sec. 4.1 Eq. 1 for testing the tuned kernel), the
// dense vector-ALU 3x3 comparator and the 2x2 max-pool of the VGG-16 stack.
#include "common.h"
#include "launch.h"

namespace psc {

hipError_t launch_conv_stream(const PatTable& tab, const PackedView& pk, const ConvArgs& a,
                              hipStream_t stream);
bool describe_conv_stream(const PatTable& tab, const ConvArgs& a, ConvForm& out);
hipError_t launch_conv_stride2(const PatTable& tab, const PackedView& pk, const ConvArgs& a, hipStream_t stream);
bool describe_conv_stride2(const PatTable& tab, const ConvArgs& a, ConvForm& out);
hipError_t launch_conv_rows(const PatTable& tab, const PackedView& pk, const ConvArgs& a, hipStream_t stream);
bool describe_conv_rows(const PatTable& tab, const ConvArgs& a, ConvForm& out);
bool prefer_conv_rows(const PatTable& tab, const ConvArgs& a);

namespace {

// One output pixel per lane, the batch folded into the lane index (small
// planes still fill the blocks); with pool, one pooled pixel: the maximum of
// the four outputs of its 2x2 window (sigma and max commute, the bias is
// common to the window).  With stride 2 (no pool) output (oh, ow) reads the
// input around (2 oh, 2 ow).
template <int DT>
__global__ __launch_bounds__(256) void k_conv_simple(const typename Elt<DT>::T* __restrict__ x, int cin,
                                                     int H, int W, int cout, int nimg, PatTable tab,
                                                     const int32_t* __restrict__ perm,
                                                     const int32_t* __restrict__ fptr,
                                                     const int32_t* __restrict__ cin_idx,
                                                     const uint8_t* __restrict__ pat_id,
                                                     const typename Elt<DT>::T* __restrict__ values,
                                                     const typename Elt<DT>::T* __restrict__ bias,
                                                     int relu, int pool, int stride,
                                                     typename Elt<DT>::T* __restrict__ y) {
    using E = Elt<DT>;
    __shared__ uint16_t msk[kMaxPatterns];
    for (int p = threadIdx.x; p < tab.m; p += 256) msk[p] = tab.mask[p];
    __syncthreads();
    const int i = blockIdx.y;
    const int plane = H * W;
    const int OW = pool ? W / 2 : (W - 1) / stride + 1;
    const int oplane = pool ? plane / 4 : ((H - 1) / stride + 1) * OW;
    // n * oplane + pix; n * oplane < 2^31, so the unsigned index cannot wrap
    const unsigned gid = blockIdx.x * 256u + threadIdx.x;
    if (gid >= unsigned(nimg * oplane)) return;
    const int n = int(gid / unsigned(oplane)), pix = int(gid - unsigned(n) * unsigned(oplane));
    const int ph = pix / OW, pw = pix - ph * OW;
    const int f = perm[i];
    const typename E::T* xn = x + int64_t(n) * cin * plane;
    float best = 0.f;
    const int nwin = pool ? 4 : 1;
    for (int t = 0; t < nwin; ++t) {
        // output position in stride-1 coordinates (centre of the 3x3 window)
        const int oh = pool ? 2 * ph + (t >> 1) : stride * ph, ow = pool ? 2 * pw + (t & 1) : stride * pw;
        float acc = 0.f;
        for (int k = fptr[i]; k < fptr[i + 1]; ++k) {
            const int ci = cin_idx[k], p = pat_id[k];
            if (unsigned(ci) >= unsigned(cin) || p >= tab.m) continue;   // malformed storage
            const typename E::T* xc = xn + int64_t(ci) * plane;
            const unsigned mk = msk[p];
            int j = 0;
            for (int q = 0; q < 9; ++q) {
                if (!((mk >> q) & 1u)) continue;
                const float v = E::load(values, int64_t(k) * 4 + j);
                ++j;
                const int ih = oh + q / 3 - 1, iw = ow + q % 3 - 1;
                if (ih >= 0 && ih < H && iw >= 0 && iw < W) acc = fmaf(v, E::load(xc, ih * W + iw), acc);
            }
        }
        best = t == 0 ? acc : fmaxf(best, acc);
    }
    if (bias) best += E::load(bias, f);
    if (relu) best = best > 0.f ? best : 0.f;
    y[(int64_t(n) * cout + f) * oplane + pix] = E::from_f(best);
}

// Dense comparator (and the dense layer of the ADMM loop): a block computes
// a 32x16 output tile (two rows per thread, ty and ty + 16) for 8 filters of
// one image.  Input channels are staged through LDS 8 at a time with a
// 1-pixel halo; the 8 weights of a (channel, tap) sit side by side, so two
// 16-byte LDS reads (the same address in every lane) give them all: 16 FMAs
// per 2 input reads and 2 weight reads.  Only the channels present are run.
constexpr int kDTH = 32;  // tile rows
constexpr int kDTW = 16;  // tile columns
constexpr int kDF = 8;    // filters per block
constexpr int kDC = 8;    // channels per stage

template <int DT>
__global__ __launch_bounds__(256) void k_dense(const typename Elt<DT>::T* __restrict__ x, int cin, int H,
                                               int W, const typename Elt<DT>::T* __restrict__ wd,
                                               int cout, const typename Elt<DT>::T* __restrict__ bias,
                                               int relu, typename Elt<DT>::T* __restrict__ y) {
    using E = Elt<DT>;
    __shared__ float xs[kDC][kDTH + 2][kDTW + 2];
    __shared__ __align__(16) float ws[kDC][9][kDF];
    const int tiles_w = (W + kDTW - 1) / kDTW;
    const int th0 = (blockIdx.x / tiles_w) * kDTH, tw0 = (blockIdx.x % tiles_w) * kDTW;
    const int f0 = blockIdx.y * kDF, n = blockIdx.z;
    const int ty = threadIdx.x / kDTW, tx = threadIdx.x % kDTW;
    const int plane = H * W;
    const typename E::T* xn = x + int64_t(n) * cin * plane;
    float acc0[kDF], acc1[kDF];
#pragma unroll
    for (int g = 0; g < kDF; ++g) acc0[g] = acc1[g] = 0.f;
    for (int c0 = 0; c0 < cin; c0 += kDC) {
        const int cn = cin - c0 < kDC ? cin - c0 : kDC;
        for (int e = threadIdx.x; e < cn * (kDTH + 2) * (kDTW + 2); e += 256) {
            const int c = e / ((kDTH + 2) * (kDTW + 2));
            const int r = (e / (kDTW + 2)) % (kDTH + 2);
            const int s = e % (kDTW + 2);
            const int ih = th0 + r - 1, iw = tw0 + s - 1;
            float v = 0.f;
            if (ih >= 0 && ih < H && iw >= 0 && iw < W) v = E::load(xn, int64_t(c0 + c) * plane + ih * W + iw);
            xs[c][r][s] = v;
        }
        for (int e = threadIdx.x; e < cn * 9 * kDF; e += 256) {
            const int c = e / (9 * kDF), q = (e / kDF) % 9, g = e % kDF;
            float v = 0.f;
            if (f0 + g < cout) v = E::load(wd, (int64_t(f0 + g) * cin + c0 + c) * 9 + q);
            ws[c][q][g] = v;
        }
        __syncthreads();
        for (int c = 0; c < cn; ++c)
#pragma unroll
            for (int q = 0; q < 9; ++q) {
                const float x0 = xs[c][ty + q / 3][tx + q % 3];
                const float x1 = xs[c][ty + 16 + q / 3][tx + q % 3];
                const float4 wa = *reinterpret_cast<const float4*>(&ws[c][q][0]);
                const float4 wb = *reinterpret_cast<const float4*>(&ws[c][q][4]);
                const float wv[kDF] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
#pragma unroll
                for (int g = 0; g < kDF; ++g) {
                    acc0[g] = fmaf(wv[g], x0, acc0[g]);
                    acc1[g] = fmaf(wv[g], x1, acc1[g]);
                }
            }
        __syncthreads();
    }
    const int ow = tw0 + tx;
    if (ow >= W) return;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const int oh = th0 + ty + 16 * half;
        if (oh >= H) break;
#pragma unroll
        for (int g = 0; g < kDF; ++g) {
            const int f = f0 + g;
            if (f >= cout) break;
            float v = half ? acc1[g] : acc0[g];
            if (bias) v += E::load(bias, f);
            if (relu) v = v > 0.f ? v : 0.f;
            y[(int64_t(n) * cout + f) * plane + oh * W + ow] = E::from_f(v);
        }
    }
}

template <int DT>
__global__ __launch_bounds__(256) void k_maxpool(const typename Elt<DT>::T* __restrict__ x, int64_t total,
                                                 int H, int W, typename Elt<DT>::T* __restrict__ y) {
    using E = Elt<DT>;
    const int Ho = H / 2, Wo = W / 2;
    for (int64_t o = int64_t(blockIdx.x) * 256 + threadIdx.x; o < total; o += int64_t(gridDim.x) * 256) {
        const int64_t nc = o / (int64_t(Ho) * Wo);
        const int r = int(o % (int64_t(Ho) * Wo));
        const int oh = r / Wo, ow = r % Wo;
        const typename E::T* p = x + nc * H * W + int64_t(2 * oh) * W + 2 * ow;
        const float a = fmaxf(E::load(p, 0), E::load(p, 1));
        const float b = fmaxf(E::load(p, W), E::load(p, W + 1));
        y[o] = E::from_f(fmaxf(a, b));
    }
}

template <int DT>
hipError_t conv_simple(const PatTable& tab, const PackedView& pk, const ConvArgs& a, hipStream_t s) {
    using T = typename Elt<DT>::T;
    const int outs = a.pool ? (a.h / 2) * (a.w / 2) : ((a.h - 1) / a.stride + 1) * ((a.w - 1) / a.stride + 1);
    const int64_t lanes = int64_t(a.n) * outs;          // at most 2^31 - 1 (y size is checked)
    const dim3 grid(unsigned((lanes + 255) / 256), unsigned(a.cout), 1);
    hipLaunchKernelGGL(k_conv_simple<DT>, grid, dim3(256), 0, s, static_cast<const T*>(a.x), a.cin, a.h,
                       a.w, a.cout, a.n, tab, pk.filter_perm, pk.filter_ptr, pk.cin_idx, pk.pat_id,
                       static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), a.relu, a.pool,
                       a.stride, static_cast<T*>(a.y));
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv(const PatTable& tab, const PackedView& pk, const ConvArgs& a, int algo,
                       hipStream_t stream) {
    // algo 2: the one-row-per-lane kernel (the caller has checked that it
    // takes the call)
    if (algo == 2 || (algo == 0 && prefer_conv_rows(tab, a))) return launch_conv_rows(tab, pk, a, stream);
    // algo 3: the column-per-lane tuned kernels, whatever the shape
    if (algo == 3) algo = 0;
    if (algo == 0 && a.stride == 1) {
        const hipError_t e = launch_conv_stream(tab, pk, a, stream);
        if (e != hipErrorNotSupported) return e;
        // inputs beyond the 2 GiB one buffer descriptor covers and pooled
        // outputs of haloed column tiles take the one-output-per-lane kernel
    }
    if (algo == 0 && a.stride == 2) {
        const hipError_t e = launch_conv_stride2(tab, pk, a, stream);
        if (e != hipErrorNotSupported) return e;
        // odd widths and more than 63 output columns take the
        // one-output-per-lane kernel
    }
    return a.dtype == DT_F16 ? conv_simple<DT_F16>(tab, pk, a, stream)
                             : conv_simple<DT_F32>(tab, pk, a, stream);
}

bool conv_rows_takes(const PatTable& tab, const ConvArgs& a) {
    ConvForm f;
    return describe_conv_rows(tab, a, f);
}

void describe_conv(const PatTable& tab, const ConvArgs& a, int algo, ConvForm& out) {
    if ((algo == 2 || (algo == 0 && prefer_conv_rows(tab, a))) && describe_conv_rows(tab, a, out)) return;
    if (algo == 3) algo = 0;
    if (algo == 0 && a.stride == 1 && describe_conv_stream(tab, a, out)) return;
    if (algo == 0 && a.stride == 2 && describe_conv_stride2(tab, a, out)) return;
    const int outs = a.pool ? (a.h / 2) * (a.w / 2) : ((a.h - 1) / a.stride + 1) * ((a.w - 1) / a.stride + 1);
    const int64_t lanes = int64_t(a.n) * outs;
    out = ConvForm{2, 0, 1, 1, 1, 1, 1, 1, int((lanes + 255) / 256) * a.cout, 256};
}

hipError_t launch_dense(int dtype, const void* x, int n, int cin, int h, int w, const void* wd, int cout,
                        const void* bias, int relu, void* y, hipStream_t stream) {
    const dim3 grid(unsigned(((h + kDTH - 1) / kDTH) * ((w + kDTW - 1) / kDTW)),
                    unsigned((cout + kDF - 1) / kDF), unsigned(n));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_dense<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x), cin,
                           h, w, static_cast<const uint16_t*>(wd), cout,
                           static_cast<const uint16_t*>(bias), relu, static_cast<uint16_t*>(y));
    else
        hipLaunchKernelGGL(k_dense<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x), cin, h,
                           w, static_cast<const float*>(wd), cout, static_cast<const float*>(bias), relu,
                           static_cast<float*>(y));
    return hipGetLastError();
}

hipError_t launch_maxpool(int dtype, const void* x, int n, int c, int h, int w, void* y,
                          hipStream_t stream) {
    const int64_t total = int64_t(n) * c * (h / 2) * (w / 2);
    const int64_t g = (total + 255) / 256;
    const dim3 grid(unsigned(g > 65536 ? 65536 : g));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_maxpool<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x),
                           total, h, w, static_cast<uint16_t*>(y));
    else
        hipLaunchKernelGGL(k_maxpool<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x), total,
                           h, w, static_cast<float*>(y));
    return hipGetLastError();
}

}  // namespace psc
