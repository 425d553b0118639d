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

// The dense 3x3 convolution of layers with at most 8 input channels (one
// LDS stage: K = 9 cin <= 72 leaves the matrix cores idle and the layer is
// bound by writing its output), on the vector ALUs: a block computes a 16x32
// (rows x columns) output tile (two rows per thread, ty and ty + 8) for 8 filters of one
// image.  Input channels are staged through LDS 8 at a time with a
// 1-pixel halo; the 8 weights of a (channel, tap) sit side by side, so two
// 16-byte LDS reads (the same address in every lane) give them all: 16 FMAs
// per 2 input reads and 2 weight reads.  Only the channels present are run.
constexpr int kDTH = 16;  // tile rows
constexpr int kDTW = 32;  // tile columns: a row of a wave's store is 128 bytes (fp32)
constexpr int kDHalf = kDTH / 2;   // a thread's second row
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
                const float x1 = xs[c][ty + kDHalf + q / 3][tx + q % 3];
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
        const int oh = th0 + ty + kDHalf * half;
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

// The dense 3x3 convolution of layers with more than 8 input channels on the
// matrix cores: an implicit GEMM with M = filters, N = output pixels
// and K = (input channel, tap), k = 9c + q, computed by fp32 MFMA
// 16x16x4 (fp16 inputs are widened exactly, so both dtypes accumulate in
// fp32).  A block owns 64 filters and a 4x16 pixel tile of one image; each
// of its 4 waves owns 32 filters x 32 pixels (two tile rows), i.e. 2 x 2
// MFMA tiles of 16 x 16, so 16 lanes of a result register hold 16 adjacent
// pixels of one row (64-byte stores).  Input channels are staged through LDS
// 8 at a time: the 6x18 input tile with its 1-pixel halo and the weights
// transposed to [k][f].  Per K step of 4 a lane reads 2 weights and 2 inputs
// from LDS and the wave issues 4 MFMAs.  The next stage's inputs and weights
// load into registers while the current stage computes, and each step's
// LDS operands load while the previous step's MFMAs issue.
//
// Operand layout of v_mfma_f32_16x16x4_f32: lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; the result element D[i][j] sits in lane
// j + 16 (i / 4), register i % 4.
constexpr int kMTR = 4;          // output tile rows
constexpr int kMTC = 16;         // output tile columns
constexpr int kMXR = kMTR + 2;   // input tile rows and columns with the halo
constexpr int kMXC = kMTC + 2;
constexpr int kMF = 64;          // filters per block
constexpr int kMC = 8;           // channels per stage
constexpr int kMK = kMC * 9;     // K per stage
constexpr int kMWS = 65;         // LDS row stride (floats) of the weight tile

typedef float psc_mf4 __attribute__((ext_vector_type(4)));

template <int DT>
__global__ __launch_bounds__(256) void k_dense_mfma(const typename Elt<DT>::T* __restrict__ x, int cin, int H,
                                                    int W, const typename Elt<DT>::T* __restrict__ wd, int cout,
                                                    const typename Elt<DT>::T* __restrict__ bias, int relu,
                                                    typename Elt<DT>::T* __restrict__ y) {
    using E = Elt<DT>;
    __shared__ float xs[kMC * kMXR * kMXC];
    __shared__ float ws[(kMK + 4) * kMWS];
    const int tiles_w = (W + kMTC - 1) / kMTC;
    const int th0 = (blockIdx.x / tiles_w) * kMTR, tw0 = (blockIdx.x % tiles_w) * kMTC;
    const int f0 = blockIdx.y * kMF, n = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fw = (wave >> 1) * 32, pw = (wave & 1) * 32;     // the wave's first filter and pixel
    const int li = lane & 15, kq = lane >> 4;
    const int plane = H * W;
    // LDS offset of the top-left halo position of this lane's two B pixels
    int pix[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int p = pw + 16 * t + li;
        pix[t] = (p / kMTC) * kMXC + p % kMTC;
    }
    psc_mf4 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = psc_mf4{0.f, 0.f, 0.f, 0.f};

    // A stage's inputs and weights pass through registers: thread t holds
    // input tile elements t + 256 j and weight elements t + 256 j of the
    // [f][k] (k < kMK) tile, loaded while the previous stage computes.  The
    // loads go through buffer descriptors: a per-thread 32-bit offset that
    // does not depend on the stage, the stage as a scalar offset, and
    // elements outside the image, the stage or the filters at an offset past
    // the range, which reads zero.
    constexpr int ESZ = int(sizeof(typename E::T));
    constexpr int kXS = kMC * kMXR * kMXC;           // 864
    constexpr int kXJ = (kXS + 255) / 256;           // 4
    constexpr int kWJ = kMF * kMK / 256;             // 18
    static_assert(kMF * kMK % 256 == 0, "weight tile elements per thread");
    const auto xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0),
                                                      int(int64_t(gridDim.z) * cin * plane * ESZ), 0x00020000);
    const auto wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(wd), int16_t(0),
                                                      int(int64_t(cout) * cin * 9 * ESZ), 0x00020000);
    auto ld = [&](__amdgpu_buffer_rsrc_t rs, uint32_t vo, int so) -> float {
        if constexpr (DT == DT_F32)
            return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, int(vo), so, 0));
        else
            return float(__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(rs, int(vo), so, 0)));
    };
    float rx[kXJ], rw[kWJ];
    auto fetch = [&](int c0) {
        const int cn = cin - c0 < kMC ? cin - c0 : kMC;
#pragma unroll
        for (int j = 0; j < kXJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            const int c = e / (kMXR * kMXC), r = (e / kMXC) % kMXR, sx = e % kMXC;
            const int ih = th0 + r - 1, iw = tw0 + sx - 1;
            const bool in = c < cn && ih >= 0 && ih < H && iw >= 0 && iw < W;
            const uint32_t vo = in ? uint32_t(((n * cin + c) * plane + ih * W + iw) * ESZ) : 0x80000000u;
            rx[j] = ld(xr, vo, c0 * plane * ESZ);
        }
#pragma unroll
        for (int j = 0; j < kWJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            const int f = e / kMK, k = e % kMK;
            const bool in = k < cn * 9 && f0 + f < cout;
            const uint32_t vo = in ? uint32_t(((f0 + f) * cin * 9 + k) * ESZ) : 0x80000000u;
            rw[j] = ld(wr, vo, c0 * 9 * ESZ);
        }
    };
    // the operands of one K step of 4 (k = 4 st + lane / 16): 2 weights and
    // 2 inputs from LDS; past kc a zero weight and a zero input (the address
    // stays inside the tile, whatever the select compiles to)
    auto operands = [&](int st, int kc, float (&o)[4]) {
        const int k = 4 * st + kq;
        const int c = k / 9, q = k - 9 * c;
        const bool valid = k < kc;
        const int xo = valid ? c * (kMXR * kMXC) + (q / 3) * kMXC + q % 3 : 0;
        o[0] = ws[k * kMWS + fw + li];
        o[1] = ws[k * kMWS + fw + 16 + li];
        o[2] = valid ? xs[xo + pix[0]] : 0.f;
        o[3] = valid ? xs[xo + pix[1]] : 0.f;
    };
    auto mfma4 = [&](const float (&o)[4]) {
        acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(o[0], o[2], acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(o[0], o[3], acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(o[1], o[2], acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(o[1], o[3], acc[1][1], 0, 0, 0);
    };

    fetch(0);
    for (int c0 = 0; c0 < cin; c0 += kMC) {
        const int cn = cin - c0 < kMC ? cin - c0 : kMC;
#pragma unroll
        for (int j = 0; j < kXJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            if (e < kXS) xs[e] = rx[j];
        }
#pragma unroll
        for (int j = 0; j < kWJ; ++j) {
            const int e = threadIdx.x + 256 * j;
            ws[(e % kMK) * kMWS + e / kMK] = rw[j];
        }
        __syncthreads();
        if (c0 + kMC < cin) fetch(c0 + kMC);   // in flight during this stage's MFMAs
        // the operands of step st + 1 load while step st's MFMAs issue
        const int kc = cn * 9, steps = (kc + 3) / 4;
        float oa[4], ob[4];
        operands(0, kc, oa);
        int st = 0;
        for (; st + 2 <= steps; st += 2) {
            operands(st + 1, kc, ob);
            mfma4(oa);
            if (st + 2 < steps) operands(st + 2, kc, oa);
            mfma4(ob);
        }
        if (st < steps) mfma4(oa);
        __syncthreads();
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int f = f0 + fw + 16 * a + 4 * kq + r;
            if (f >= cout) continue;
            const float bv = bias ? E::load(bias, f) : 0.f;
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int p = pw + 16 * b + li;
                const int oh = th0 + p / kMTC, ow = tw0 + p % kMTC;
                if (oh >= H || ow >= W) continue;
                float v = acc[a][b][r] + bv;
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
    // the matrix-core kernel addresses x and the weights through 32-bit
    // buffer offsets
    const int esz = dtype == DT_F16 ? 2 : 4;
    const bool small = int64_t(n) * cin * h * w * esz < (int64_t(1) << 31) &&
                       int64_t(cout) * cin * 9 * esz < (int64_t(1) << 31);
    if (cin <= kDC || !small) {
        const dim3 grid(unsigned(((h + kDTH - 1) / kDTH) * ((w + kDTW - 1) / kDTW)),
                        unsigned((cout + kDF - 1) / kDF), unsigned(n));
        if (dtype == DT_F16)
            hipLaunchKernelGGL(k_dense<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x), cin,
                               h, w, static_cast<const uint16_t*>(wd), cout,
                               static_cast<const uint16_t*>(bias), relu, static_cast<uint16_t*>(y));
        else
            hipLaunchKernelGGL(k_dense<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x), cin,
                               h, w, static_cast<const float*>(wd), cout, static_cast<const float*>(bias), relu,
                               static_cast<float*>(y));
        return hipGetLastError();
    }
    const dim3 grid(unsigned(((h + kMTR - 1) / kMTR) * ((w + kMTC - 1) / kMTC)),
                    unsigned((cout + kMF - 1) / kMF), unsigned(n));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_dense_mfma<DT_F16>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(x), cin,
                           h, w, static_cast<const uint16_t*>(wd), cout, static_cast<const uint16_t*>(bias), relu,
                           static_cast<uint16_t*>(y));
    else
        hipLaunchKernelGGL(k_dense_mfma<DT_F32>, grid, dim3(256), 0, stream, static_cast<const float*>(x), cin,
                           h, w, static_cast<const float*>(wd), cout, static_cast<const float*>(bias), relu,
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
