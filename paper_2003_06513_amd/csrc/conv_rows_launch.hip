// Launch configuration of the one-row-per-lane pattern-sparse 3x3
// convolution (Sec. 4.1 Eq. 1, stride 1; conv_rows.h): images per wave,
// filter shares and the choice between it and the column-per-lane kernels.
#include "conv_rows.h"

namespace psc {
using namespace rw;

#define PSC_EXTERN_ROWS(DT, W, ST) \
    extern template hipError_t rw::launch_rows<DT, W, ST>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
PSC_EXTERN_ROWS(DT_F32, 4, 1)
PSC_EXTERN_ROWS(DT_F32, 7, 1)
PSC_EXTERN_ROWS(DT_F32, 8, 1)
PSC_EXTERN_ROWS(DT_F32, 14, 1)
PSC_EXTERN_ROWS(DT_F32, 16, 1)
PSC_EXTERN_ROWS(DT_F32, 28, 1)
PSC_EXTERN_ROWS(DT_F32, 8, 2)
PSC_EXTERN_ROWS(DT_F32, 16, 2)
PSC_EXTERN_ROWS(DT_F32, 32, 2)
PSC_EXTERN_ROWS(DT_F16, 4, 1)
PSC_EXTERN_ROWS(DT_F16, 7, 1)
PSC_EXTERN_ROWS(DT_F16, 8, 1)
PSC_EXTERN_ROWS(DT_F16, 14, 1)
PSC_EXTERN_ROWS(DT_F16, 16, 1)
PSC_EXTERN_ROWS(DT_F16, 28, 1)
PSC_EXTERN_ROWS(DT_F16, 8, 2)
PSC_EXTERN_ROWS(DT_F16, 16, 2)
PSC_EXTERN_ROWS(DT_F16, 32, 2)
#undef PSC_EXTERN_ROWS

namespace {

bool width_compiled(int dtype, int w, int stride) {
    if (stride == 2) return w == 8 || w == 16 || w == 32;
    // fp16 rows of odd width are read through a shifted 16-byte window (7 halves at most)
    if (dtype == DT_F16 && (w & 1)) return w == 7;
    return w == 4 || w == 7 || w == 8 || w == 14 || w == 16 || w == 28;
}

// Grids of fewer waves split each filter into more shares.
constexpr int64_t kSplitWavesRows = 4096;

}  // namespace

// The launch configuration, or false when the kernel does not take the call:
// a pooled output, more than 63 output rows, a width without a compiled
// variant (stride 1: 4, 7, 8, 14, 16, 28; stride 2: 8, 16, 32), x beyond the
// 2 GiB a buffer descriptor addresses here.  Host only.
bool plan_conv_rows(const PatTable& tab, const ConvArgs& a, RGeo& g) {
    if ((a.stride != 1 && a.stride != 2) || a.pool || !width_compiled(a.dtype, a.w, a.stride)) return false;
    const int oh = (a.h - 1) / a.stride + 1;
    if (oh > 63) return false;
    const int esz = a.dtype == DT_F16 ? 2 : 4;
    const int64_t x_bytes = int64_t(a.n) * a.cin * a.h * a.w * esz;
    if (x_bytes >= (int64_t(1) << 31) || a.keep * 4 * esz > 0x7fffffff) return false;
    std::memset(&g, 0, sizeof g);
    g.n = a.n;
    g.cin = a.cin;
    g.H = a.h;
    g.W = a.w;
    g.ST = a.stride;
    g.OH = oh;
    g.OW = a.w / a.stride;
    g.cout = a.cout;
    g.m = tab.m;
    g.x_bytes = int(x_bytes);
    g.keep = int(a.keep);
    g.relu = a.relu;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.shape[p] = -1;
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    g.staged = staged_geometry(a.dtype, a.w, a.h, a.stride);
    g.seg_len = g.OH + 1;
    g.S = 64 / g.seg_len;
    g.groups = (a.n + g.S - 1) / g.S;
    g.KS = 1;
    // the partial sums of the shares go through LDS: KS * OW * 64 floats
    while (g.KS < kMaxShares && int64_t(g.groups) * a.cout * g.KS < kSplitWavesRows && a.cin >= 16 * g.KS &&
           2 * g.KS * g.OW <= 128)
        g.KS *= 2;
    g.FW = g.KS >= 4 ? 1 : 4 / g.KS;
    if (g.FW > a.cout) g.FW = a.cout;
    g.groups_x = (a.cout + g.FW - 1) / g.FW;
    g.nblocks = g.groups_x * g.groups;
    return true;
}

// Whether the automatic choice (algo 0) takes this kernel: batches that fill
// at least one wave with whole images, on planes of at most 16 columns, where
// the column-per-lane kernels spend R+2 single-element loads per 4R FMAs
// (measured 1.5-4.7x faster there); 28-column rows (about 200 VGPRs, two
// waves per SIMD) only in grids of many waves, where they were measured
// slightly ahead.  Stride 2 on 8-column inputs and on fp32 16 x 16 planes
// (staged through LDS); other wider rows put the lanes of one 16-byte load
// 128 or 256 bytes apart, one cache line each, and measured slower than the
// column-per-lane stride-2 kernel.
bool prefer_conv_rows(const PatTable& tab, const ConvArgs& a) {
    RGeo g;
    if (!plan_conv_rows(tab, a, g) || a.n < g.S) return false;
    if (a.stride == 2) return a.w == 8 || g.staged;
    return a.w <= 16 || int64_t(g.groups) * a.cout >= 8192;
}

bool describe_conv_rows(const PatTable& tab, const ConvArgs& a, ConvForm& out) {
    RGeo g;
    if (!plan_conv_rows(tab, a, g)) return false;
    out = ConvForm{4, g.staged, 1, g.OW, g.S, 1, g.KS, g.FW, g.nblocks, g.FW * g.KS * 64};
    return true;
}

hipError_t launch_conv_rows(const PatTable& tab, const PackedView& pk, const ConvArgs& a, hipStream_t stream) {
    RGeo g;
    if (!plan_conv_rows(tab, a, g)) return hipErrorNotSupported;
#define PSC_ROWS_W(DT)                                                   \
    if (a.stride == 2) {                                                 \
        switch (a.w) {                                                   \
            case 8: return launch_rows<DT, 8, 2>(pk, a, g, stream);      \
            case 16: return launch_rows<DT, 16, 2>(pk, a, g, stream);    \
            case 32: return launch_rows<DT, 32, 2>(pk, a, g, stream);    \
            default: return hipErrorNotSupported;                        \
        }                                                                \
    }                                                                    \
    switch (a.w) {                                                       \
        case 4: return launch_rows<DT, 4, 1>(pk, a, g, stream);          \
        case 7: return launch_rows<DT, 7, 1>(pk, a, g, stream);          \
        case 8: return launch_rows<DT, 8, 1>(pk, a, g, stream);          \
        case 14: return launch_rows<DT, 14, 1>(pk, a, g, stream);        \
        case 16: return launch_rows<DT, 16, 1>(pk, a, g, stream);        \
        case 28: return launch_rows<DT, 28, 1>(pk, a, g, stream);        \
        default: return hipErrorNotSupported;                            \
    }
    if (a.dtype == DT_F16) {
        PSC_ROWS_W(DT_F16)
    }
    PSC_ROWS_W(DT_F32)
#undef PSC_ROWS_W
}

}  // namespace psc
