// Pattern-sparse 3x3 convolution with stride 2 (Sec. 4.1 Eq. 1 with a
// stride; the stage-entry convolutions of the ResNets the paper prunes),
// zero padding 1, for images of even width W with at most 63 output columns.
//
// As in the stride-1 kernels, one wave walks one reordered filter's
// compressed storage (Sec. 3.4) and its lanes hold output pixels: a lane
// owns output column j and R output rows of a band; a wave holds S bands of
// full output rows, each followed by one zero lane.  Output (i, j) reads
// input rows 2i-1..2i+1 and columns 2j-1..2j+1, so for each kernel a lane
// loads, for the 2R+1 input rows its R output rows need, columns 2j and
// 2j+1 in one 8-byte (fp32) or 4-byte (fp16) load, and takes column 2j-1 --
// the left lane's column 2(j-1)+1 -- by DPP.  The wave walks the filter's
// storage one pattern segment after another, each through a loop compiled
// with that centre+3 shape's taps fixed (other masks take a loop that
// dispatches each tap); the channel index and weights are wave-uniform.
// The next kernel's rows load while the current kernel's FMAs run.
#include "common.h"
#include "launch.h"

namespace psc {
namespace {

constexpr int kR2 = 4;                 // output rows per lane
constexpr int kRows2 = 2 * kR2 + 1;    // input rows per lane and kernel
constexpr int kDppShr = 0x138;         // wave_shr:1 -- lane i reads lane i-1

struct Geo2 {
    int n, cin, H, W, cout, m, OH, OW;
    int S, seg_len, RB, units, slots;
    int KS, FW, groups_x, nblocks;
    int64_t keep;
    int relu;
    uint16_t mask[kMaxPatterns];
    int8_t shape[kMaxPatterns];   // centre+3 shape index of each library pattern, -1 = other mask
};

template <int DT> struct Pair;
template <> struct Pair<DT_F32> {
    __device__ __forceinline__ static void load(const float* p, float& e, float& o) {
        const float2 v = *reinterpret_cast<const float2*>(p);
        e = v.x;
        o = v.y;
    }
};
template <> struct Pair<DT_F16> {
    __device__ __forceinline__ static void load(const uint16_t* p, float& e, float& o) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
        e = float(__builtin_bit_cast(_Float16, uint16_t(v)));
        o = float(__builtin_bit_cast(_Float16, uint16_t(v >> 16)));
    }
};

template <int DT>
__device__ __forceinline__ void load_rows2(const typename Elt<DT>::T* xc, const int (&ro)[kRows2], bool lane_ok,
                                           float (&ev)[kRows2], float (&od)[kRows2]) {
#pragma unroll
    for (int r = 0; r < kRows2; ++r) {
        float e = 0.f, o = 0.f;
        if (lane_ok && ro[r] >= 0) Pair<DT>::load(xc + ro[r], e, o);
        ev[r] = e;
        od[r] = o;
    }
}

// acc[i] += w * X[2i + DR] for the lane's R output rows.
template <int DR>
__device__ __forceinline__ void tap2(float (&acc)[kR2], const float (&X)[kRows2], float w) {
#pragma unroll
    for (int i = 0; i < kR2; ++i) acc[i] = fmaf(w, X[2 * i + DR], acc[i]);
}

// Tap at kernel position Q: column 0 reads the left lane's odd column (lf),
// column 1 the lane's even column, column 2 its odd column.
template <int Q>
__device__ __forceinline__ void tap2_fix(float (&acc)[kR2], const float (&lf)[kRows2], const float (&ev)[kRows2],
                                         const float (&od)[kRows2], float w) {
    if constexpr (Q % 3 == 0) tap2<Q / 3>(acc, lf, w);
    else if constexpr (Q % 3 == 1) tap2<Q / 3>(acc, ev, w);
    else tap2<Q / 3>(acc, od, w);
}

__device__ __forceinline__ void tap2_dyn(int q, float (&acc)[kR2], const float (&lf)[kRows2],
                                         const float (&ev)[kRows2], const float (&od)[kRows2], float w) {
    switch (q) {
        case 0: tap2<0>(acc, lf, w); break;
        case 1: tap2<0>(acc, ev, w); break;
        case 2: tap2<0>(acc, od, w); break;
        case 3: tap2<1>(acc, lf, w); break;
        case 4: tap2<1>(acc, ev, w); break;
        case 5: tap2<1>(acc, od, w); break;
        case 6: tap2<2>(acc, lf, w); break;
        case 7: tap2<2>(acc, ev, w); break;
        default: tap2<2>(acc, od, w); break;
    }
}

struct Ctx2 {
    int ro[kRows2];          // element offset of input column 2j of each row (-1: padding)
    bool lane_ok;
    int cin, plane;
};

template <int DT>
__device__ __forceinline__ void rows_of(const Ctx2& c, const typename Elt<DT>::T* xn, int ci, float (&ev)[kRows2],
                                        float (&od)[kRows2]) {
    const bool ok = unsigned(ci) < unsigned(c.cin);     // malformed channel indices read zeros
    load_rows2<DT>(xn + int64_t(ok ? ci : 0) * c.plane, c.ro, c.lane_ok && ok, ev, od);
}

// Kernels [k0, k1) of one pattern segment whose taps sit at positions Q0..Q3
// (compile-time for the centre+3 shapes, QD = false; read from q[] for other
// masks).  The rows of the next kernel load while this one's FMAs run.
template <int DT, bool QD, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void run_seg2(const Ctx2& c, const typename Elt<DT>::T* xn,
                                         const int32_t* __restrict__ cin_idx,
                                         const typename Elt<DT>::T* __restrict__ vals, int k0, int k1,
                                         const int (&q)[4], float (&acc)[kR2]) {
    using E = Elt<DT>;
    constexpr bool kLeft = Q0 % 3 == 0 || Q1 % 3 == 0 || Q2 % 3 == 0 || Q3 % 3 == 0;
    const bool left = QD ? (q[0] % 3 == 0 || q[1] % 3 == 0 || q[2] % 3 == 0 || q[3] % 3 == 0) : kLeft;
    float ev[kRows2], od[kRows2], ev2[kRows2], od2[kRows2];
    rows_of<DT>(c, xn, cin_idx[k0], ev, od);
    for (int k = k0; k < k1; ++k) {
        if (k + 1 < k1) rows_of<DT>(c, xn, cin_idx[k + 1], ev2, od2);
        float lf[kRows2];
        if (left) {
#pragma unroll
            for (int r = 0; r < kRows2; ++r)
                lf[r] = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, od[r]),
                                                                              kDppShr, 0xf, 0xf, true));
        } else {
#pragma unroll
            for (int r = 0; r < kRows2; ++r) lf[r] = 0.f;          // no column-0 tap reads it
        }
        const float w0 = E::load(vals, int64_t(k) * 4), w1 = E::load(vals, int64_t(k) * 4 + 1);
        const float w2 = E::load(vals, int64_t(k) * 4 + 2), w3 = E::load(vals, int64_t(k) * 4 + 3);
        if constexpr (QD) {
            tap2_dyn(q[0], acc, lf, ev, od, w0);
            tap2_dyn(q[1], acc, lf, ev, od, w1);
            tap2_dyn(q[2], acc, lf, ev, od, w2);
            tap2_dyn(q[3], acc, lf, ev, od, w3);
        } else {
            tap2_fix<Q0>(acc, lf, ev, od, w0);
            tap2_fix<Q1>(acc, lf, ev, od, w1);
            tap2_fix<Q2>(acc, lf, ev, od, w2);
            tap2_fix<Q3>(acc, lf, ev, od, w3);
        }
        if (k + 1 < k1) {
#pragma unroll
            for (int r = 0; r < kRows2; ++r) {
                ev[r] = ev2[r];
                od[r] = od2[r];
            }
        }
    }
}

template <int DT, int MASK>
__device__ __forceinline__ void run_shape2(const Ctx2& c, const typename Elt<DT>::T* xn, const int32_t* cin_idx,
                                           const typename Elt<DT>::T* vals, int k0, int k1, const int (&q)[4],
                                           float (&acc)[kR2]) {
    run_seg2<DT, false, NthBit<MASK, 0>::value(), NthBit<MASK, 1>::value(), NthBit<MASK, 2>::value(),
             NthBit<MASK, 3>::value()>(c, xn, cin_idx, vals, k0, k1, q, acc);
}

#define PSC_S2_CASE(I) \
    case I: run_shape2<DT, kCentre3.code[I]>(c, xn, cin_idx, vals, k0, k1, q, acc); return;
#define PSC_S2_CASE8(I)                                                                             \
    PSC_S2_CASE(I) PSC_S2_CASE(I + 1) PSC_S2_CASE(I + 2) PSC_S2_CASE(I + 3) PSC_S2_CASE(I + 4)      \
    PSC_S2_CASE(I + 5) PSC_S2_CASE(I + 6) PSC_S2_CASE(I + 7)
template <int DT>
__device__ __forceinline__ void run_pattern2(int shape, const Ctx2& c, const typename Elt<DT>::T* xn,
                                             const int32_t* cin_idx, const typename Elt<DT>::T* vals, int k0,
                                             int k1, const int (&q)[4], float (&acc)[kR2]) {
    switch (shape) {
        PSC_S2_CASE8(0)
        PSC_S2_CASE8(8)
        PSC_S2_CASE8(16)
        PSC_S2_CASE8(24)
        PSC_S2_CASE8(32)
        PSC_S2_CASE8(40)
        PSC_S2_CASE8(48)
        default: run_seg2<DT, true, 0, 0, 0, 0>(c, xn, cin_idx, vals, k0, k1, q, acc); return;
    }
}
#undef PSC_S2_CASE8
#undef PSC_S2_CASE

template <int DT>
__global__ __launch_bounds__(256) void k_conv_stride2(const typename Elt<DT>::T* __restrict__ x,
                                                      const int32_t* __restrict__ perm,
                                                      const int32_t* __restrict__ seg_ptr,
                                                      const int32_t* __restrict__ cin_idx,
                                                      const typename Elt<DT>::T* __restrict__ vals,
                                                      const typename Elt<DT>::T* __restrict__ bias,
                                                      typename Elt<DT>::T* __restrict__ y, Geo2 g) {
    using E = Elt<DT>;
    __shared__ float red[4][kR2][64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int gf = wave / g.KS, sp = wave - gf * g.KS;          // filter slot, share
    // XCD-aware block order: the blocks one XCD runs are consecutive logical
    // blocks (same output band group, different filter groups)
    const int b = blockIdx.x;
    int lb = b;
    if (g.nblocks >= 8) {
        const int per = g.nblocks / 8, rem = g.nblocks % 8;
        const int xcd = b % 8, slot = b / 8;
        lb = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
    }
    const int fg = lb % g.groups_x, sg = lb / g.groups_x;
    const int i = fg * g.FW + gf;
    const bool has_filter = i < g.cout;

    const int seg = lane / g.seg_len, j = lane - seg * g.seg_len;
    const int u = sg * g.S + seg;
    bool lane_ok = false;
    int nimg = 0, i0 = 0;
    if (seg < g.S && u < g.units && j < g.OW) {
        lane_ok = true;
        nimg = u / g.RB;
        i0 = (u - nimg * g.RB) * kR2;
    }
    const int plane = g.H * g.W;
    // element offset (inside one channel plane) of input column 2j of each row
    int ro[kRows2];
#pragma unroll
    for (int r = 0; r < kRows2; ++r) {
        const int row = 2 * i0 - 1 + r;
        ro[r] = (row >= 0 && row < g.H) ? row * g.W + 2 * j : -1;
    }
    float acc[kR2];
#pragma unroll
    for (int r = 0; r < kR2; ++r) acc[r] = 0.f;

    if (has_filter) {
        const int* segp = seg_ptr + int64_t(i) * (g.m + 1);
        const int f0 = segp[0], f1 = segp[g.m];
        const int len = f1 - f0;
        const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
        const typename E::T* xn = x + int64_t(nimg) * g.cin * plane;
        Ctx2 c;
#pragma unroll
        for (int r = 0; r < kRows2; ++r) c.ro[r] = ro[r];
        c.lane_ok = lane_ok;
        c.cin = g.cin;
        c.plane = plane;
        for (int p = 0; p < g.m; ++p) {
            int k0 = segp[p], k1 = segp[p + 1];
            k0 = k0 < s0 ? s0 : k0;
            k1 = k1 > s1 ? s1 : k1;                               // malformed pointers stay in the share
            if (k0 >= k1) continue;
            int q[4] = {4, 4, 4, 4}, t = 0;
            const unsigned mk = g.mask[p];
            for (int qq = 0; qq < 9; ++qq)
                if ((mk >> qq) & 1u) {
                    if (t < 4) q[t] = qq;
                    ++t;
                }
            run_pattern2<DT>(g.shape[p], c, xn, cin_idx, vals, k0, k1, q, acc);
        }
    }
    // add the KS partial sums of each filter in share order
    if (g.KS > 1) {
        for (int slot = 0; slot < g.FW; ++slot) {
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < kR2; ++r) red[sp][r][lane] = acc[r];
            }
            __syncthreads();
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < kR2; ++r) {
                    float v = 0.f;
                    for (int t = 0; t < g.KS; ++t) v += red[t][r][lane];
                    acc[r] = v;
                }
            }
            __syncthreads();
        }
    }
    if (!has_filter || !lane_ok) return;
    const int f = perm[i];
    const float bv = bias ? E::load(bias, f) : 0.f;
    typename E::T* yp = y + (int64_t(nimg) * g.cout + f) * (g.OH * g.OW) + j;
#pragma unroll
    for (int r = 0; r < kR2; ++r) {
        const int row = i0 + r;
        if (row < g.OH && (r % g.KS) == sp) {
            float v = acc[r] + bv;
            if (g.relu) v = v > 0.f ? v : 0.f;
            yp[row * g.OW] = E::from_f(v);
        }
    }
}

}  // namespace

// Launch configuration of the stride-2 kernel; false when it does not take
// the call (odd width, more than 63 output columns, a pooled output).
static bool plan_conv_stride2(const PatTable& tab, const ConvArgs& a, ConvForm* form, Geo2* out) {
    if (a.stride != 2 || a.pool || (a.w & 1)) return false;
    const int OH = (a.h - 1) / 2 + 1, OW = (a.w - 1) / 2 + 1;
    if (OW > 63) return false;
    Geo2 g{};
    g.n = a.n;
    g.cin = a.cin;
    g.H = a.h;
    g.W = a.w;
    g.cout = a.cout;
    g.m = tab.m;
    g.OH = OH;
    g.OW = OW;
    g.keep = a.keep;
    g.relu = a.relu;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        g.shape[p] = -1;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    g.seg_len = OW + 1;
    g.S = 65 / (OW + 1);
    g.RB = (OH + kR2 - 1) / kR2;
    g.units = a.n * g.RB;
    g.slots = (g.units + g.S - 1) / g.S;
    g.KS = 1;
    while (g.KS < 4 && int64_t(g.slots) * a.cout * g.KS < 4096 && a.cin >= 16 * g.KS) g.KS *= 2;
    g.FW = 4 / g.KS;
    if (g.FW > a.cout) g.FW = a.cout;
    g.groups_x = (a.cout + g.FW - 1) / g.FW;
    g.nblocks = g.groups_x * g.slots;
    if (form) *form = ConvForm{3, 0, kR2, 1, g.S, 1, g.KS, g.FW, g.nblocks, g.FW * g.KS * 64};
    if (out) *out = g;
    return true;
}

bool describe_conv_stride2(const PatTable& tab, const ConvArgs& a, ConvForm& form) {
    return plan_conv_stride2(tab, a, &form, nullptr);
}

hipError_t launch_conv_stride2(const PatTable& tab, const PackedView& pk, const ConvArgs& a, hipStream_t stream) {
    Geo2 g;
    if (!plan_conv_stride2(tab, a, nullptr, &g)) return hipErrorNotSupported;
    const dim3 grid(unsigned(g.nblocks)), block(unsigned(g.FW * g.KS * 64));
    if (a.dtype == DT_F16)
        hipLaunchKernelGGL(k_conv_stride2<DT_F16>, grid, block, 0, stream, static_cast<const uint16_t*>(a.x),
                           pk.filter_perm, pk.seg_ptr, pk.cin_idx, static_cast<const uint16_t*>(pk.values),
                           static_cast<const uint16_t*>(a.bias), static_cast<uint16_t*>(a.y), g);
    else
        hipLaunchKernelGGL(k_conv_stride2<DT_F32>, grid, block, 0, stream, static_cast<const float*>(a.x),
                           pk.filter_perm, pk.seg_ptr, pk.cin_idx, static_cast<const float*>(pk.values),
                           static_cast<const float*>(a.bias), static_cast<float*>(a.y), g);
    return hipGetLastError();
}

}  // namespace psc
