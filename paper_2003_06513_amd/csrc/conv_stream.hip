// Tuned pattern-sparse 3x3 convolution forward (Sec. 4.1 Eq. 1), built on
// the three compiler optimisations of Sec. 3.4 redesigned for CDNA4:
//
//  * filter kernel reorder -> one wave per reordered filter (or per share of
//    it, below): the filter's kernels, channel indices and weights are
//    wave-uniform and arrive by scalar loads; filters of similar length run
//    side by side;
//  * compressed weight storage -> the wave walks the filter's storage in its
//    own order: one pattern segment after another, each processed by a loop
//    compiled for that pattern's shape (a switch over the 56 centre+3 shapes
//    taken once per segment), so no weight position is ever decoded;
//  * load redundancy elimination -> each lane owns one output column and R
//    output rows; for every kernel it loads the R+2 input rows it needs once
//    into registers and takes the left/right neighbour columns from adjacent
//    lanes with DPP inside the FMA itself (v_fmac_f32_dpp), so one load feeds
//    up to 4 FMAs per row.  The rows of the next kernel load while the
//    current one's FMAs run.  Input rows come through a buffer descriptor:
//    offsets of padding rows and columns are placed past its range, where a
//    buffer load returns zero, so the zero padding costs nothing.
//
// There is no LDS staging and no barrier in the main loop: reuse of an input
// row across the filters that touch it happens in the L1/L2 caches (filters
// of one spatial tile run on the same XCD).
//
// Lane layout: a wave's 64 lanes hold S independent segments.  If the image
// row fits (W <= 63), a segment is one full row band [W columns] and the
// segments are separated by a single lane that holds zero -- the zero padding
// on both sides.  Otherwise a segment is [halo][Wt columns][halo], the halo
// lanes holding the real neighbouring columns (or zero at the image border).
//
// Small grids split each filter over KS waves: wave s takes the s-th of KS
// equal contiguous ranges of the filter's kernels; the partial sums are
// added in share order through LDS, so results are deterministic.
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "launch.h"

namespace psc {
namespace {

// The 56 masks made of the centre and 3 of its 8 neighbours, ascending.
struct Centre3Table {
    uint16_t code[56];
    constexpr Centre3Table() : code{} {
        int n = 0;
        for (int c = 0; c < 512; ++c) {
            int pc = 0;
            for (int b = 0; b < 9; ++b) pc += (c >> b) & 1;
            if (((c >> 4) & 1) && pc == 4) code[n++] = uint16_t(c);
        }
    }
};
constexpr Centre3Table kCentre3{};

constexpr int kMaxSplit = 8;

struct Geo {
    int n, cin, H, W, cout, m;
    int S;          // segments per wave
    int seg_len;    // lanes per segment
    int Wt;         // output columns per segment
    int cols_mode;  // 0: full-row segments with zero separators, 1: haloed column tiles
    int RB, CT;     // row blocks and column tiles per image
    int U;          // work units = n * RB * CT
    int FW, KS;     // filters and shares per filter in a workgroup
    int groups_x;   // filter groups (fastest varying logical block index)
    int nblocks;    // total workgroups
    int x_bytes;    // bytes of x (the buffer range), at most 2^31
    int relu;
    int8_t shape[kMaxPatterns];  // centre+3 shape index of each library pattern, -1 = generic
    uint16_t mask[kMaxPatterns];
};

// ------------------------------------------------------------------ taps
// acc[r] += w * x[r + DR] taken from the lane to the left (DS == 0), the same
// lane (DS == 1) or the lane to the right (DS == 2); lanes without a
// neighbour read 0 (bound_ctrl).  The shifted forms fold the DPP into the FMA
// (the weight must then sit in a VGPR); the s_nop covers the wait states a
// DPP read needs after a VALU write.  All taps are asm so the accumulators
// keep their registers across the taps of a run.
#define PSC_SHR "wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_SHL "wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_FM(i) "v_fmac_f32_dpp %[a" #i "], %[x" #i "], %[w] "
#define PSC_FC(i) "v_fmac_f32_e32 %[a" #i "], %[w], %[x" #i "]\n"
#define PSC_A(i) [a##i] "+v"(acc[i])
#define PSC_X(i) [x##i] "v"(xr[DR + i])

template <int R, int DR, int DS, bool WS> struct Tap;   // WS: weight may stay in an SGPR

#define PSC_TAPS(DSV, WSV, NOP, L, WC)                                                                \
    template <int DR> struct Tap<2, DR, DSV, WSV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[2], const float (&xr)[4], float w) {  \
            asm volatile(NOP L(0) L(1) : PSC_A(0), PSC_A(1) : PSC_X(0), PSC_X(1), [w] WC(w));         \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<4, DR, DSV, WSV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[4], const float (&xr)[6], float w) {  \
            asm volatile(NOP L(0) L(1) L(2) L(3)                                                      \
                         : PSC_A(0), PSC_A(1), PSC_A(2), PSC_A(3)                                     \
                         : PSC_X(0), PSC_X(1), PSC_X(2), PSC_X(3), [w] WC(w));                        \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<7, DR, DSV, WSV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[7], const float (&xr)[9], float w) {  \
            asm volatile(NOP L(0) L(1) L(2) L(3) L(4) L(5) L(6)                                       \
                         : PSC_A(0), PSC_A(1), PSC_A(2), PSC_A(3), PSC_A(4), PSC_A(5), PSC_A(6)       \
                         : PSC_X(0), PSC_X(1), PSC_X(2), PSC_X(3), PSC_X(4), PSC_X(5), PSC_X(6),      \
                           [w] WC(w));                                                                \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<8, DR, DSV, WSV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[8], const float (&xr)[10], float w) { \
            asm volatile(NOP L(0) L(1) L(2) L(3) L(4) L(5) L(6) L(7)                                  \
                         : PSC_A(0), PSC_A(1), PSC_A(2), PSC_A(3), PSC_A(4), PSC_A(5), PSC_A(6),      \
                           PSC_A(7)                                                                   \
                         : PSC_X(0), PSC_X(1), PSC_X(2), PSC_X(3), PSC_X(4), PSC_X(5), PSC_X(6),      \
                           PSC_X(7), [w] WC(w));                                                      \
        }                                                                                             \
    };

#define PSC_L_SHR(i) PSC_FM(i) PSC_SHR "\n"
#define PSC_L_SHL(i) PSC_FM(i) PSC_SHL "\n"
#define PSC_WV(w) "v"(w)
#define PSC_WS(w) "s"(w)
// kernel column 0 reads x at w - 1 (the lane to the left), column 2 at w + 1
// (the lane to the right), column 1 the lane's own column
PSC_TAPS(0, false, "s_nop 4\n", PSC_L_SHR, PSC_WV)
PSC_TAPS(0, true, "s_nop 4\n", PSC_L_SHR, PSC_WV)
PSC_TAPS(1, false, "", PSC_FC, PSC_WV)
PSC_TAPS(1, true, "", PSC_FC, PSC_WS)
PSC_TAPS(2, false, "s_nop 4\n", PSC_L_SHL, PSC_WV)
PSC_TAPS(2, true, "s_nop 4\n", PSC_L_SHL, PSC_WV)
#undef PSC_WS
#undef PSC_WV
#undef PSC_L_SHL
#undef PSC_L_SHR
#undef PSC_TAPS
#undef PSC_X
#undef PSC_A
#undef PSC_FC
#undef PSC_FM
#undef PSC_SHL
#undef PSC_SHR

// fp32 weights arrive in SGPRs (scalar loads); fp16 ones are widened into
// VGPRs.
template <int Q, int R, bool WS>
__device__ __forceinline__ void tap_q(float (&acc)[R], const float (&xr)[R + 2], float wv) {
    Tap<R, Q / 3, Q % 3, WS>::run(acc, xr, wv);
}

template <int R, bool WS>
__device__ __forceinline__ void tap_dyn(int q, float (&acc)[R], const float (&xr)[R + 2], float wv) {
    switch (q) {
        case 0: tap_q<0, R, WS>(acc, xr, wv); break;
        case 1: tap_q<1, R, WS>(acc, xr, wv); break;
        case 2: tap_q<2, R, WS>(acc, xr, wv); break;
        case 3: tap_q<3, R, WS>(acc, xr, wv); break;
        case 4: tap_q<4, R, WS>(acc, xr, wv); break;
        case 5: tap_q<5, R, WS>(acc, xr, wv); break;
        case 6: tap_q<6, R, WS>(acc, xr, wv); break;
        case 7: tap_q<7, R, WS>(acc, xr, wv); break;
        default: tap_q<8, R, WS>(acc, xr, wv); break;
    }
}

// Position of the JJ-th set bit of MASK (ascending).
template <int MASK, int JJ>
struct NthBit {
    static constexpr int value() {
        int seen = 0;
        for (int q = 0; q < 9; ++q)
            if ((MASK >> q) & 1) {
                if (seen == JJ) return q;
                ++seen;
            }
        return -1;
    }
};

// ------------------------------------------------------------------ runs
template <int DT>
struct RunCtx {
    const int32_t* __restrict__ cin_idx;
    const typename Elt<DT>::T* __restrict__ vals;
    __amdgpu_buffer_rsrc_t xr;   // x, bounded to its size
    int chan_bytes;              // bytes of one input channel plane
    int cmax;                    // last input channel
};

template <int DT>
__device__ __forceinline__ void load_w4(const typename Elt<DT>::T* __restrict__ vals, int k, float (&wv)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) wv[j] = Elt<DT>::load(vals, int64_t(k) * 4 + j);
}

// The R+2 input rows of channel ci in this lane's column (zero outside the
// image: those offsets lie past the buffer range).
template <int DT, int R>
__device__ __forceinline__ void load_rows(const RunCtx<DT>& c, const uint32_t (&vo)[R + 2], int ci,
                                          float (&xr)[R + 2]) {
    ci = ci < 0 ? 0 : (ci > c.cmax ? c.cmax : ci);    // a malformed index stays inside x
    const int soff = __builtin_amdgcn_readfirstlane(ci * c.chan_bytes);   // wave-uniform: an SGPR operand
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
        if constexpr (DT == DT_F32)
            xr[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(c.xr, vo[r], soff, 0));
        else
            xr[r] = float(__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(c.xr, vo[r], soff, 0)));
    }
}

// Kernels [k, e) of one pattern segment share (e > k).  Two kernels per
// trip: the rows of one load while the other's FMAs run; metadata is read two
// kernels ahead; the single loop exit keeps the accumulators in place.
template <int DT, int R, class TapFn>
__device__ __forceinline__ void run_kernels(const RunCtx<DT>& c, const uint32_t (&vo)[R + 2], int k, int e,
                                            float (&acc)[R], TapFn taps) {
    const int last = e - 1;
    float wA[4], wB[4];
    load_w4<DT>(c.vals, k, wA);
    int kk = k + 1 <= last ? k + 1 : last;
    int ciB = __builtin_amdgcn_readfirstlane(c.cin_idx[kk]);
    load_w4<DT>(c.vals, kk, wB);
    float xA[R + 2], xB[R + 2];
    load_rows<DT, R>(c, vo, __builtin_amdgcn_readfirstlane(c.cin_idx[k]), xA);
    while (k + 1 < e) {
        load_rows<DT, R>(c, vo, ciB, xB);                      // rows of kernel k+1
        kk = k + 2 <= last ? k + 2 : last;
        const int ciA2 = __builtin_amdgcn_readfirstlane(c.cin_idx[kk]);
        float wA2[4];
        load_w4<DT>(c.vals, kk, wA2);
        kk = k + 3 <= last ? k + 3 : last;
        const int ciB2 = __builtin_amdgcn_readfirstlane(c.cin_idx[kk]);
        float wB2[4];
        load_w4<DT>(c.vals, kk, wB2);
        taps(acc, xA, wA);                                     // kernel k
        load_rows<DT, R>(c, vo, ciA2, xA);                     // rows of kernel k+2
        taps(acc, xB, wB);                                     // kernel k+1
        k += 2;
        wA[0] = wA2[0], wA[1] = wA2[1], wA[2] = wA2[2], wA[3] = wA2[3];
        wB[0] = wB2[0], wB[1] = wB2[1], wB[2] = wB2[2], wB[3] = wB2[3];
        ciB = ciB2;
    }
    if (k < e) taps(acc, xA, wA);
}

template <int DT, int R, int MASK>
__device__ __forceinline__ void run_shape(const RunCtx<DT>& c, const uint32_t (&vo)[R + 2], int k, int e,
                                          float (&acc)[R]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    constexpr bool WS = DT == DT_F32;
    run_kernels<DT, R>(c, vo, k, e, acc, [](float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
        tap_q<Q0, R, WS>(a, x, w[0]);
        tap_q<Q1, R, WS>(a, x, w[1]);
        tap_q<Q2, R, WS>(a, x, w[2]);
        tap_q<Q3, R, WS>(a, x, w[3]);
    });
}

// Any 4-of-9 mask: the taps are chosen per kernel by uniform branches.
template <int DT, int R>
__device__ __forceinline__ void run_generic(unsigned mask, const RunCtx<DT>& c, const uint32_t (&vo)[R + 2],
                                            int k, int e, float (&acc)[R]) {
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
    constexpr bool WS = DT == DT_F32;
    run_kernels<DT, R>(c, vo, k, e, acc, [=](float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
        tap_dyn<R, WS>(q0, a, x, w[0]);
        tap_dyn<R, WS>(q1, a, x, w[1]);
        tap_dyn<R, WS>(q2, a, x, w[2]);
        tap_dyn<R, WS>(q3, a, x, w[3]);
    });
}

#define PSC_SHAPE_CASE(I) \
    case I: run_shape<DT, R, kCentre3.code[I]>(c, vo, k, e, acc); return;
#define PSC_SHAPE_CASE8(I)                                                                     \
    PSC_SHAPE_CASE(I) PSC_SHAPE_CASE(I + 1) PSC_SHAPE_CASE(I + 2) PSC_SHAPE_CASE(I + 3)        \
    PSC_SHAPE_CASE(I + 4) PSC_SHAPE_CASE(I + 5) PSC_SHAPE_CASE(I + 6) PSC_SHAPE_CASE(I + 7)

template <int DT, int R>
__device__ __forceinline__ void run_pattern(int shape, unsigned mask, const RunCtx<DT>& c,
                                            const uint32_t (&vo)[R + 2], int k, int e, float (&acc)[R]) {
    switch (shape) {
        PSC_SHAPE_CASE8(0)
        PSC_SHAPE_CASE8(8)
        PSC_SHAPE_CASE8(16)
        PSC_SHAPE_CASE8(24)
        PSC_SHAPE_CASE8(32)
        PSC_SHAPE_CASE8(40)
        PSC_SHAPE_CASE8(48)
        default: run_generic<DT, R>(mask, c, vo, k, e, acc); return;
    }
}
#undef PSC_SHAPE_CASE8
#undef PSC_SHAPE_CASE

// ------------------------------------------------------------------ kernel
template <int DT, int R>
__global__ __launch_bounds__(512) void k_conv_stream(const typename Elt<DT>::T* __restrict__ x,
                                                     const int32_t* __restrict__ perm,
                                                     const int32_t* __restrict__ seg_ptr,
                                                     const int32_t* __restrict__ cin_idx,
                                                     const typename Elt<DT>::T* __restrict__ vals,
                                                     const typename Elt<DT>::T* __restrict__ bias,
                                                     typename Elt<DT>::T* __restrict__ y, Geo g) {
    using E = Elt<DT>;
    constexpr int ROWS = R + 2;
    __shared__ float red[kMaxSplit][R][64];     // partial sums of the shares of one filter

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int gf = wave / g.KS, sp = wave - gf * g.KS;   // filter slot, share

    // XCD-aware block order: the hardware deals consecutive blocks out to the
    // 8 XCDs in turn; remap so that the blocks one XCD runs are consecutive
    // logical blocks, which share a spatial tile (its input rows stay in that
    // XCD's L2) and differ in their filter group.
    const int b = blockIdx.x;
    int lb = b;
    if (g.nblocks >= 8) {
        const int per = g.nblocks / 8, rem = g.nblocks % 8;
        const int xcd = b % 8, slot = b / 8;
        lb = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
    }
    const int fg = lb % g.groups_x, sgrp = lb / g.groups_x;
    const int i = fg * g.FW + gf;                        // reordered filter of this wave
    const bool has_filter = i < g.cout;

    // ---- lane geometry
    const int s = lane / g.seg_len, cidx = lane - s * g.seg_len;
    const int u = sgrp * g.S + s;
    int ld_col = -1, out_col = -1, nimg = 0, h0 = 0;
    if (s < g.S && u < g.U) {
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
    const int plane = g.H * g.W;
    // byte offset of this lane's column in each of its R+2 input rows of
    // channel 0; 2^31 (past the buffer range, reads zero) for padding
    uint32_t vo[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        const int row = h0 - 1 + r;
        vo[r] = (ld_col >= 0 && row >= 0 && row < g.H)
                    ? uint32_t(nimg * g.cin * plane + row * g.W + ld_col) * uint32_t(sizeof(typename E::T))
                    : 0x80000000u;
    }

    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;

    if (has_filter) {
        const RunCtx<DT> ctx{cin_idx, vals,
                             __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0),
                                                               g.x_bytes, 0x00020000),
                             __builtin_amdgcn_readfirstlane(plane * int(sizeof(typename E::T))), g.cin - 1};
        const int* segp = seg_ptr + i * (g.m + 1);
        const int f0 = segp[0], f1 = segp[g.m];
        // share sp: the sp-th of KS equal contiguous ranges of the filter's
        // kernels, which crosses few pattern segments
        const int len = f1 - f0;
        const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
        for (int p = 0; p < g.m; ++p) {
            int k0 = segp[p], k1 = segp[p + 1];
            k0 = k0 < s0 ? s0 : k0;
            k1 = k1 > s1 ? s1 : k1;                         // malformed pointers stay in the share
            if (k0 < k1) run_pattern<DT, R>(g.shape[p], g.mask[p], ctx, vo, k0, k1, acc);
        }
    }

    // ---- add the KS partial sums of each filter in share order
    if (g.KS > 1) {
        // the KS waves of filter slot gf use red[0..KS) of their own barrier
        // phase: slots are processed one after another
        for (int slot = 0; slot < g.FW; ++slot) {
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < R; ++r) red[sp][r][lane] = acc[r];
            }
            __syncthreads();
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    float v = 0.f;
                    for (int t = 0; t < g.KS; ++t) v += red[t][r][lane];
                    acc[r] = v;
                }
            }
            __syncthreads();
        }
    }
    if (!has_filter || out_col < 0) return;
    const int f = perm[i];
    const float bv = bias ? E::load(bias, f) : 0.f;
    typename E::T* yp = y + (nimg * g.cout + f) * plane + out_col;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        // the KS waves of a filter hold the same sums; share t stores rows t, t+KS, ...
        const int row = h0 + r;
        if (row < g.H && (r % g.KS) == sp) {
            float v = acc[r] + bv;
            if (g.relu) v = v > 0.f ? v : 0.f;
            yp[row * g.W] = E::from_f(v);
        }
    }
}

template <int DT, int R>
hipError_t launch_r(const PackedView& pk, const ConvArgs& a, const Geo& g, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    hipLaunchKernelGGL((k_conv_stream<DT, R>), dim3(unsigned(g.nblocks)), dim3(unsigned(g.FW * g.KS * 64)), 0,
                       stream, static_cast<const T*>(a.x), pk.filter_perm, pk.seg_ptr, pk.cin_idx,
                       static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), static_cast<T*>(a.y), g);
    return hipGetLastError();
}

}  // namespace

// Launch configuration.  Rows per lane R minimise the lane-rows issued
// (ceil(units / S) * R, larger R on ties); a workgroup holds 4 filters, or
// fewer filters split into KS shares (KS doubles up to 8) while the grid
// holds under 4 waves per SIMD.  Returns hipErrorNotSupported when x exceeds
// the 2 GiB a buffer descriptor addresses here.
hipError_t launch_conv_stream(const PatTable& tab, const PackedView& pk, const ConvArgs& a,
                              hipStream_t stream) {
    const int64_t x_bytes = int64_t(a.n) * a.cin * a.h * a.w * (a.dtype == DT_F16 ? 2 : 4);
    if (x_bytes > (int64_t(1) << 31)) return hipErrorNotSupported;
    Geo g;
    std::memset(&g, 0, sizeof g);
    g.n = a.n;
    g.cin = a.cin;
    g.H = a.h;
    g.W = a.w;
    g.cout = a.cout;
    g.m = tab.m;
    g.relu = a.relu;
    g.x_bytes = int(x_bytes > 0x7fffffff ? 0x7fffffff : x_bytes);
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.shape[p] = -1;
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    // lane layout: full-row segments if they use the lanes at least as well
    // as haloed column tiles
    const int S_rows = a.w <= 63 ? 65 / (a.w + 1) : 0;
    const int use_rows = S_rows * a.w;
    int ct = (a.w + 61) / 62, use_cols = 0;
    for (int t = ct; t <= a.w && t <= 64; ++t) {
        const int wt = (a.w + t - 1) / t;
        const int use = (64 / (wt + 2)) * a.w / t;
        if (use > use_cols) {
            use_cols = use;
            ct = t;
        }
    }
    if (S_rows > 0 && use_rows >= use_cols) {
        g.cols_mode = 0;
        g.S = S_rows;
        g.seg_len = a.w + 1;
        g.Wt = a.w;
        g.CT = 1;
    } else {
        const int Wt = (a.w + ct - 1) / ct;
        g.cols_mode = 1;
        g.S = 64 / (Wt + 2);
        g.seg_len = Wt + 2;
        g.Wt = Wt;
        g.CT = ct;
    }
    // rows per lane
    const int cand[4] = {8, 7, 4, 2};
    int R = 8;
    int64_t best = -1;
    for (int rr : cand) {
        const int64_t units = int64_t(a.n) * ((a.h + rr - 1) / rr) * g.CT;
        const int64_t cost = (units + g.S - 1) / g.S * rr;
        if (best < 0 || cost < best) {
            best = cost;
            R = rr;
        }
    }
    g.RB = (a.h + R - 1) / R;
    g.U = a.n * g.RB * g.CT;
    const int sgroups = (g.U + g.S - 1) / g.S;
    g.KS = 1;
    while (g.KS < kMaxSplit && int64_t(sgroups) * a.cout * g.KS < 4096 && a.cin >= 16 * g.KS) g.KS *= 2;
    if (const char* t = getenv("PSC_CONV_TUNE")) {   // experiments: "KS=2"
        if (const char* q = strstr(t, "KS=")) g.KS = atoi(q + 3);
        if (g.KS < 1) g.KS = 1;
        if (g.KS > kMaxSplit) g.KS = kMaxSplit;
    }
    g.FW = g.KS >= 4 ? 1 : 4 / g.KS;
    if (g.FW > a.cout) g.FW = a.cout;
    const int fgroups = (a.cout + g.FW - 1) / g.FW;
    g.groups_x = fgroups;
    g.nblocks = fgroups * sgroups;
    switch (R) {
        case 8: return a.dtype == DT_F16 ? launch_r<DT_F16, 8>(pk, a, g, stream)
                                         : launch_r<DT_F32, 8>(pk, a, g, stream);
        case 7: return a.dtype == DT_F16 ? launch_r<DT_F16, 7>(pk, a, g, stream)
                                         : launch_r<DT_F32, 7>(pk, a, g, stream);
        case 4: return a.dtype == DT_F16 ? launch_r<DT_F16, 4>(pk, a, g, stream)
                                         : launch_r<DT_F32, 4>(pk, a, g, stream);
        default: return a.dtype == DT_F16 ? launch_r<DT_F16, 2>(pk, a, g, stream)
                                          : launch_r<DT_F32, 2>(pk, a, g, stream);
    }
}

}  // namespace psc
