// Pattern-sparse 3x3 convolution with stride 2 (Sec. 4.1 Eq. 1 with a
// stride; the stage-entry convolutions of the ResNets the paper prunes),
// zero padding 1, for images of even width W with at most 63 output columns.
//
// As in the stride-1 kernels, one wave walks one reordered filter's
// compressed storage (Sec. 3.4) and its lanes hold output pixels: a lane
// owns C adjacent output columns (C = 1, or 2 when W is a multiple of 4) and
// R output rows of a band; a wave holds S bands of full output rows, each
// followed by one zero lane.  Output (i, j) reads input rows 2i-1..2i+1 and
// columns 2j-1..2j+1, so for each kernel a lane loads, for the 2R+1 input
// rows its R output rows need, its 2C input columns in one buffer load (C =
// 1: 8 bytes fp32 / 4 fp16; C = 2: 16 / 8) at an offset fixed per lane and
// row (the channel enters as a scalar offset; padding rows and lanes point
// past the buffer range and read zero); the column left of them -- the left
// lane's last column -- is read by DPP inside the FMA (v_fmac_f32_dpp
// wave_shr:1).  The wave walks the filter's storage one pattern segment after
// another, each through a loop compiled with that centre+3 shape's taps fixed
// (other masks take a loop that dispatches each tap); channel index and
// weights are wave-uniform (scalar buffer loads).  The next kernel's rows
// load while the current kernel's FMAs run.
#include "conv_stream.h"

namespace psc {
namespace {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kR2 = 4;                 // output rows per lane
constexpr int kRows2 = 2 * kR2 + 1;    // input rows per lane and kernel

struct Geo2 {
    int n, cin, H, W, cout, m, OH, OW;
    int C;                             // output columns per lane
    int S, seg_len, RB, units, slots;
    int KS, FW, groups_x, nblocks;
    int64_t keep;
    int x_bytes;
    int relu;
    uint16_t mask[kMaxPatterns];
    int8_t shape[kMaxPatterns];   // centre+3 shape index of each library pattern, -1 = other mask
};

// Raw words of a lane's 2C input columns in each of its 2R+1 rows.
template <int DT, int C> struct Cols {
    static constexpr int NW = DT == DT_F32 ? 2 * C : C;
    uint32_t d[kRows2][NW];
};

// The 2C input columns of each row as fp32: v[c][r] is column 2C j + c.
template <int C> struct ColVals {
    float v[2 * C][kRows2];
};

struct Ctx2 {
    cs::Meta m;
    __amdgpu_buffer_rsrc_t xr;     // x, bounded to its size
    int chan_bytes;                // bytes of one input channel plane
    uint32_t vo[kRows2];           // byte offset of the lane's first column of each row, channel 0 (2^31: padding)
};

template <int DT, int C>
__device__ __forceinline__ void load_cols(const Ctx2& c, int ci, Cols<DT, C>& p) {
    // wave-uniform: an SGPR operand.  A malformed channel index reads zeros
    // or other data of x, never memory outside it (range-checked loads).
    const int soff = __builtin_amdgcn_readfirstlane(ci * c.chan_bytes);
#pragma unroll
    for (int r = 0; r < kRows2; ++r) {
        if constexpr (Cols<DT, C>::NW == 4) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(c.xr, int(c.vo[r]), soff, 0);
            p.d[r][0] = v.x, p.d[r][1] = v.y, p.d[r][2] = v.z, p.d[r][3] = v.w;
        } else if constexpr (Cols<DT, C>::NW == 2) {
            const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(c.xr, int(c.vo[r]), soff, 0);
            p.d[r][0] = v.x, p.d[r][1] = v.y;
        } else {
            p.d[r][0] = __builtin_amdgcn_raw_buffer_load_b32(c.xr, int(c.vo[r]), soff, 0);
        }
    }
}

// The columns as fp32; then an asm the compiler sees as writing the last
// column (the one the right neighbour reads by DPP: no VALU write of it can
// follow) and the two wait states a DPP read needs after a VALU write of its
// source.
template <int DT, int C>
__device__ __forceinline__ void unpack_cols(const Cols<DT, C>& p, ColVals<C>& x) {
#pragma unroll
    for (int r = 0; r < kRows2; ++r) {
#pragma unroll
        for (int q = 0; q < 2 * C; ++q) {
            if constexpr (DT == DT_F32)
                x.v[q][r] = __builtin_bit_cast(float, p.d[r][q]);
            else
                x.v[q][r] = float(__builtin_bit_cast(_Float16, uint16_t(p.d[r][q / 2] >> (16 * (q & 1)))));
        }
    }
    float (&l)[kRows2] = x.v[2 * C - 1];
    asm volatile("" : "+v"(l[0]), "+v"(l[1]), "+v"(l[2]), "+v"(l[3]), "+v"(l[4]));
    asm volatile("" : "+v"(l[5]), "+v"(l[6]), "+v"(l[7]), "+v"(l[8]));
    asm volatile("s_nop 1");
}

// The tap at kernel position Q = 3 ky + kx: for each output column c of the
// lane and each output row i, acc[c][i] += w * x(row 2i + ky - 1, column
// 2(Cj + c) + kx - 1).  Column 2Cj - 1 is the last column of the lane to the
// left (DPP; a lane without one reads zero).
template <int Q, int C>
__device__ __forceinline__ void tap2(float (&acc)[C][kR2], const ColVals<C>& x, float w) {
    constexpr int ky = Q / 3, kx = Q % 3;
#pragma unroll
    for (int c = 0; c < C; ++c) {
#pragma unroll
        for (int i = 0; i < kR2; ++i) {
            const int col = 2 * c + kx - 1;     // input column relative to the lane's first
            if (col < 0)
                asm volatile("v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
                             : "+v"(acc[c][i])
                             : "v"(x.v[2 * C - 1][2 * i + ky]), "v"(w));
            else
                acc[c][i] = __builtin_fmaf(w, x.v[col][2 * i + ky], acc[c][i]);
        }
    }
}

template <int C>
__device__ __forceinline__ void tap2_dyn(int q, float (&acc)[C][kR2], const ColVals<C>& x, float w) {
    switch (q) {
        case 0: tap2<0, C>(acc, x, w); break;
        case 1: tap2<1, C>(acc, x, w); break;
        case 2: tap2<2, C>(acc, x, w); break;
        case 3: tap2<3, C>(acc, x, w); break;
        case 4: tap2<4, C>(acc, x, w); break;
        case 5: tap2<5, C>(acc, x, w); break;
        case 6: tap2<6, C>(acc, x, w); break;
        case 7: tap2<7, C>(acc, x, w); break;
        default: tap2<8, C>(acc, x, w); break;
    }
}

// Kernels [k, e) of one pattern segment share (e > k), two per trip: the
// rows of one load while the other's FMAs run; metadata is read two kernels
// ahead; the single loop exit keeps the accumulators in place.
template <int DT, int C, class TapFn>
__device__ __forceinline__ void run2(const Ctx2& c, int k, int e, float (&acc)[C][kR2], TapFn taps) {
    const int last = e - 1;
    float wA[4], wB[4];
    cs::meta_w<DT>(c.m, k, wA);
    int kk = k + 1 <= last ? k + 1 : last;
    int ciB = cs::meta_ci(c.m, kk);
    cs::meta_w<DT>(c.m, kk, wB);
    Cols<DT, C> pA, pB;
    load_cols<DT, C>(c, cs::meta_ci(c.m, k), pA);
    while (k + 1 < e) {
        load_cols<DT, C>(c, ciB, pB);                            // rows of kernel k+1
        kk = k + 2 <= last ? k + 2 : last;
        const int ciA2 = cs::meta_ci(c.m, kk);
        float wA2[4];
        cs::meta_w<DT>(c.m, kk, wA2);
        kk = k + 3 <= last ? k + 3 : last;
        const int ciB2 = cs::meta_ci(c.m, kk);
        float wB2[4];
        cs::meta_w<DT>(c.m, kk, wB2);
        {
            ColVals<C> x;
            unpack_cols<DT, C>(pA, x);
            taps(acc, x, wA);                                    // kernel k
        }
        load_cols<DT, C>(c, ciA2, pA);                           // rows of kernel k+2
        {
            ColVals<C> x;
            unpack_cols<DT, C>(pB, x);
            taps(acc, x, wB);                                    // kernel k+1
        }
        k += 2;
        wA[0] = wA2[0], wA[1] = wA2[1], wA[2] = wA2[2], wA[3] = wA2[3];
        wB[0] = wB2[0], wB[1] = wB2[1], wB[2] = wB2[2], wB[3] = wB2[3];
        ciB = ciB2;
    }
    if (k < e) {
        ColVals<C> x;
        unpack_cols<DT, C>(pA, x);
        taps(acc, x, wA);
    }
}

template <int DT, int C, int MASK>
__device__ __forceinline__ void run_shape2(const Ctx2& c, int k, int e, float (&acc)[C][kR2]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    run2<DT, C>(c, k, e, acc, [](float (&a)[C][kR2], const ColVals<C>& x, const float (&w)[4]) {
        // the taps without a DPP read first: they put FMAs between the unpack
        // and the DPP reads
        if constexpr (Q0 % 3 != 0) tap2<Q0, C>(a, x, w[0]);
        if constexpr (Q1 % 3 != 0) tap2<Q1, C>(a, x, w[1]);
        if constexpr (Q2 % 3 != 0) tap2<Q2, C>(a, x, w[2]);
        if constexpr (Q3 % 3 != 0) tap2<Q3, C>(a, x, w[3]);
        if constexpr (Q0 % 3 == 0) tap2<Q0, C>(a, x, w[0]);
        if constexpr (Q1 % 3 == 0) tap2<Q1, C>(a, x, w[1]);
        if constexpr (Q2 % 3 == 0) tap2<Q2, C>(a, x, w[2]);
        if constexpr (Q3 % 3 == 0) tap2<Q3, C>(a, x, w[3]);
    });
}

// Any 4-of-9 mask: each tap is chosen per kernel by a uniform branch.
template <int DT, int C>
__device__ __forceinline__ void run_generic2(unsigned mask, const Ctx2& c, int k, int e, float (&acc)[C][kR2]) {
    int q0 = 4, q1 = 4, q2 = 4, q3 = 4, seen = 0;
#pragma unroll
    for (int q = 0; q < 9; ++q) {
        if ((mask >> q) & 1u) {
            if (seen == 0) q0 = q;
            else if (seen == 1) q1 = q;
            else if (seen == 2) q2 = q;
            else if (seen == 3) q3 = q;
            ++seen;
        }
    }
    run2<DT, C>(c, k, e, acc, [=](float (&a)[C][kR2], const ColVals<C>& x, const float (&w)[4]) {
        tap2_dyn<C>(q0, a, x, w[0]);
        tap2_dyn<C>(q1, a, x, w[1]);
        tap2_dyn<C>(q2, a, x, w[2]);
        tap2_dyn<C>(q3, a, x, w[3]);
    });
}

#define PSC_S2_CASE(I) \
    case I: run_shape2<DT, C, kCentre3.code[I]>(c, k, e, acc); return;
#define PSC_S2_CASE8(I)                                                                             \
    PSC_S2_CASE(I) PSC_S2_CASE(I + 1) PSC_S2_CASE(I + 2) PSC_S2_CASE(I + 3) PSC_S2_CASE(I + 4)      \
    PSC_S2_CASE(I + 5) PSC_S2_CASE(I + 6) PSC_S2_CASE(I + 7)
template <int DT, int C>
__device__ __forceinline__ void run_pattern2(int shape, unsigned mask, const Ctx2& c, int k, int e,
                                             float (&acc)[C][kR2]) {
    switch (shape) {
        PSC_S2_CASE8(0)
        PSC_S2_CASE8(8)
        PSC_S2_CASE8(16)
        PSC_S2_CASE8(24)
        PSC_S2_CASE8(32)
        PSC_S2_CASE8(40)
        PSC_S2_CASE8(48)
        default: run_generic2<DT, C>(mask, c, k, e, acc); return;
    }
}
#undef PSC_S2_CASE8
#undef PSC_S2_CASE

template <int DT, int C>
__global__ __launch_bounds__(256) void k_conv_stride2(const typename Elt<DT>::T* __restrict__ x,
                                                      const int32_t* __restrict__ perm,
                                                      const int32_t* __restrict__ seg_ptr,
                                                      const int32_t* __restrict__ cin_idx,
                                                      const typename Elt<DT>::T* __restrict__ vals,
                                                      const typename Elt<DT>::T* __restrict__ bias,
                                                      typename Elt<DT>::T* __restrict__ y, Geo2 g) {
    using E = Elt<DT>;
    __shared__ float red[4][C * kR2][64];
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

    // lane j of a band owns output columns Cj .. Cj + C - 1
    const int seg = lane / g.seg_len, j = lane - seg * g.seg_len;
    const int u = sg * g.S + seg;
    bool lane_ok = false;
    int nimg = 0, i0 = 0;
    if (seg < g.S && u < g.units && C * j < g.OW) {
        lane_ok = true;
        nimg = u / g.RB;
        i0 = (u - nimg * g.RB) * kR2;
    }
    const int plane = g.H * g.W;
    constexpr int ESZ = int(sizeof(typename E::T));
    float acc[C][kR2];
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int r = 0; r < kR2; ++r) acc[c][r] = 0.f;

    if (has_filter) {
        const int* segp = seg_ptr + int64_t(i) * (g.m + 1);
        const int f0 = segp[0], f1 = segp[g.m];
        const int len = f1 - f0;
        const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
        Ctx2 c;
        c.m = cs::Meta{cs::scalar_rsrc(cin_idx, int(g.keep) * 4), cs::scalar_rsrc(vals, int(g.keep) * 4 * ESZ)};
        c.xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes, 0x00020000);
        c.chan_bytes = __builtin_amdgcn_readfirstlane(plane * ESZ);
        // byte offset of input column 2Cj of each of the lane's rows in
        // channel 0 of its image; past the buffer range for padding
#pragma unroll
        for (int r = 0; r < kRows2; ++r) {
            const int row = 2 * i0 - 1 + r;
            c.vo[r] = (lane_ok && row >= 0 && row < g.H)
                          ? uint32_t(nimg * g.cin * plane + row * g.W + 2 * C * j) * uint32_t(ESZ)
                          : 0x80000000u;
        }
        for (int p = 0; p < g.m; ++p) {
            int k0 = segp[p], k1 = segp[p + 1];
            k0 = k0 < s0 ? s0 : k0;
            k1 = k1 > s1 ? s1 : k1;                               // malformed pointers stay in the share
            if (k0 < k1) run_pattern2<DT, C>(g.shape[p], g.mask[p], c, k0, k1, acc);
        }
    }
    // add the KS partial sums of each filter in share order
    if (g.KS > 1) {
        for (int slot = 0; slot < g.FW; ++slot) {
            if (slot == gf) {
#pragma unroll
                for (int c = 0; c < C; ++c)
#pragma unroll
                    for (int r = 0; r < kR2; ++r) red[sp][c * kR2 + r][lane] = acc[c][r];
            }
            __syncthreads();
            if (slot == gf) {
#pragma unroll
                for (int c = 0; c < C; ++c)
#pragma unroll
                    for (int r = 0; r < kR2; ++r) {
                        float v = 0.f;
                        for (int t = 0; t < g.KS; ++t) v += red[t][c * kR2 + r][lane];
                        acc[c][r] = v;
                    }
            }
            __syncthreads();
        }
    }
    if (!has_filter || !lane_ok) return;
    const int f = perm[i];
    const float bv = bias ? E::load(bias, f) : 0.f;
    typename E::T* yp = y + (int64_t(nimg) * g.cout + f) * (g.OH * g.OW) + C * j;
#pragma unroll
    for (int r = 0; r < kR2; ++r) {
        const int row = i0 + r;
        if (row < g.OH && (r % g.KS) == sp) {
#pragma unroll
            for (int c = 0; c < C; ++c) {
                float v = acc[c][r] + bv;
                if (g.relu) v = v > 0.f ? v : 0.f;
                yp[row * g.OW + c] = E::from_f(v);
            }
        }
    }
}

}  // namespace

// Launch configuration of the stride-2 kernel; false when it does not take
// the call (odd width, more than 63 output columns, a pooled output, x
// beyond the 2 GiB a buffer descriptor addresses here).
static bool plan_conv_stride2(const PatTable& tab, const ConvArgs& a, ConvForm* form, Geo2* out) {
    if (a.stride != 2 || a.pool || (a.w & 1)) return false;
    const int OH = (a.h - 1) / 2 + 1, OW = (a.w - 1) / 2 + 1;
    if (OW > 63) return false;
    // buffer descriptors address at most 2 GiB (x) and the packed weights
    const int esz = a.dtype == DT_F16 ? 2 : 4;
    const int64_t x_bytes = int64_t(a.n) * a.cin * a.h * a.w * esz;
    if (x_bytes >= (int64_t(1) << 31) || a.keep * 4 * esz > 0x7fffffff) return false;
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
    g.x_bytes = int(x_bytes);
    g.relu = a.relu;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        g.shape[p] = -1;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    // two output columns per lane when the lane's 4 input columns start on
    // a 16-byte (fp32) / 8-byte (fp16) boundary: W a multiple of 4
    g.C = a.w % 4 == 0 ? 2 : 1;
    const int lanes = (OW + g.C - 1) / g.C;
    g.seg_len = lanes + 1;
    g.S = 65 / (lanes + 1);
    g.RB = (OH + kR2 - 1) / kR2;
    g.units = a.n * g.RB;
    g.slots = (g.units + g.S - 1) / g.S;
    g.KS = 1;
    while (g.KS < 4 && int64_t(g.slots) * a.cout * g.KS < 4096 && a.cin >= 16 * g.KS) g.KS *= 2;
    g.FW = 4 / g.KS;
    if (g.FW > a.cout) g.FW = a.cout;
    g.groups_x = (a.cout + g.FW - 1) / g.FW;
    g.nblocks = g.groups_x * g.slots;
    if (form) *form = ConvForm{3, 0, kR2, g.C, g.S, 1, g.KS, g.FW, g.nblocks, g.FW * g.KS * 64};
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
#define PSC_S2_LAUNCH(DT, T, C)                                                                              \
    hipLaunchKernelGGL((k_conv_stride2<DT, C>), grid, block, 0, stream, static_cast<const T*>(a.x),            \
                       pk.filter_perm, pk.seg_ptr, pk.cin_idx, static_cast<const T*>(pk.values),             \
                       static_cast<const T*>(a.bias), static_cast<T*>(a.y), g)
    if (a.dtype == DT_F16) {
        if (g.C == 2) PSC_S2_LAUNCH(DT_F16, uint16_t, 2);
        else PSC_S2_LAUNCH(DT_F16, uint16_t, 1);
    } else {
        if (g.C == 2) PSC_S2_LAUNCH(DT_F32, float, 2);
        else PSC_S2_LAUNCH(DT_F32, float, 1);
    }
#undef PSC_S2_LAUNCH
    return hipGetLastError();
}

}  // namespace psc
