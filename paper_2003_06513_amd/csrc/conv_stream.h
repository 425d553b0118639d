// Kernel templates of the tuned pattern-sparse 3x3 convolution forward (Sec. 4.1 Eq. 1), built on
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
// Input rows reach the registers one of two ways.  Direct: buffer loads
// straight into registers.  Staged (full-row segments, throughput-bound
// grids): the wave copies the contiguous rows its segments need into its own
// LDS area with 64-byte-aligned 1 KiB buffer-to-LDS loads, two copies in
// turn, and reads its rows from there -- a row load that straddles 128-byte
// lines costs the vector memory path twice as much as an aligned one, and
// image rows rarely start on a line.  Neither form has a barrier in the main
// loop; reuse of an input row across the filters that touch it happens in
// the L1/L2 caches (filters of one spatial tile run on the same XCD).
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
#pragma once
#include <cstring>

#include "common.h"
#include "launch.h"

// Scalar buffer loads (the LLVM intrinsic, declared by its name).
typedef int32_t psc_i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t psc_i32x2 __attribute__((ext_vector_type(2)));
typedef float psc_f32x4 __attribute__((ext_vector_type(4)));
__device__ int32_t psc_sbuf_i32(psc_i32x4, int32_t, int32_t) __asm("llvm.amdgcn.s.buffer.load.i32");
__device__ psc_i32x2 psc_sbuf_i32x2(psc_i32x4, int32_t, int32_t) __asm("llvm.amdgcn.s.buffer.load.v2i32");
__device__ psc_f32x4 psc_sbuf_f32x4(psc_i32x4, int32_t, int32_t) __asm("llvm.amdgcn.s.buffer.load.v4f32");

namespace psc {
namespace cs {

constexpr int kMaxSplit = 8;
// Waves (one share per filter) from which a grid of 28..63-column images
// (and fp16 images of any width) takes the wide form: 6 per SIMD.  Measured:
// 3584 waves 7 % slower than the one-column form, 7168 waves 17 % faster,
// batch-1 grids of up to 1024 waves 0-15 % slower.
constexpr int64_t kWideMinWaves = 6144;

typedef psc_i32x4 int32x4;

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
    int keep;       // kept kernels (entries of cin_idx)
    int relu;
    int pool;       // 1: y is the 2x2/2 max-pool of the output (R even, full-row segments)
    int lds;        // 1: input rows staged through per-wave LDS (full-row segments only)
    int region;     // LDS bytes reserved per run of rows
    int wave_bytes; // LDS bytes per wave: nruns regions + a zero area
    int R;          // rows per lane (the kernel's template argument)
    int form;       // 0: one column per lane (k_conv_stream), 1: 4 columns per lane (k_conv_wide)
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

// WS: the weight may stay in an SGPR; NW: the asm starts with the two wait
// states a DPP read needs after a VALU write of one of its operands.
template <int R, int DR, int DS, bool WS, bool NW> struct Tap;

#define PSC_TAPS(DSV, WSV, NWV, NOP, L, WC)                                                           \
    template <int DR> struct Tap<2, DR, DSV, WSV, NWV> {                                             \
        __device__ __forceinline__ static void run(float (&acc)[2], const float (&xr)[4], float w) {  \
            asm volatile(NOP L(0) L(1) : PSC_A(0), PSC_A(1) : PSC_X(0), PSC_X(1), [w] WC(w));         \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<4, DR, DSV, WSV, NWV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[4], const float (&xr)[6], float w) {  \
            asm volatile(NOP L(0) L(1) L(2) L(3)                                                      \
                         : PSC_A(0), PSC_A(1), PSC_A(2), PSC_A(3)                                     \
                         : PSC_X(0), PSC_X(1), PSC_X(2), PSC_X(3), [w] WC(w));                        \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<7, DR, DSV, WSV, NWV> {                                                  \
        __device__ __forceinline__ static void run(float (&acc)[7], const float (&xr)[9], float w) {  \
            asm volatile(NOP L(0) L(1) L(2) L(3) L(4) L(5) L(6)                                       \
                         : PSC_A(0), PSC_A(1), PSC_A(2), PSC_A(3), PSC_A(4), PSC_A(5), PSC_A(6)       \
                         : PSC_X(0), PSC_X(1), PSC_X(2), PSC_X(3), PSC_X(4), PSC_X(5), PSC_X(6),      \
                           [w] WC(w));                                                                \
        }                                                                                             \
    };                                                                                                \
    template <int DR> struct Tap<8, DR, DSV, WSV, NWV> {                                                  \
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
PSC_TAPS(0, false, true, "s_nop 1\n", PSC_L_SHR, PSC_WV)
PSC_TAPS(0, false, false, "", PSC_L_SHR, PSC_WV)
PSC_TAPS(1, false, false, "", PSC_FC, PSC_WV)
PSC_TAPS(1, true, false, "", PSC_FC, PSC_WS)
PSC_TAPS(2, false, true, "s_nop 1\n", PSC_L_SHL, PSC_WV)
PSC_TAPS(2, false, false, "", PSC_L_SHL, PSC_WV)
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

// Tap at position Q of the 3x3 kernel.  Same-column taps take the weight
// from an SGPR when WS (fp32 scalar loads); the shifted (DPP) taps take it
// from a VGPR and, unless NW is false, start with two wait states.
template <int Q, int R, bool WS, bool NW = true>
__device__ __forceinline__ void tap_q(float (&acc)[R], const float (&xr)[R + 2], float wv) {
    if constexpr (Q % 3 == 1)
        Tap<R, Q / 3, 1, WS, false>::run(acc, xr, wv);
    else
        Tap<R, Q / 3, Q % 3, false, NW>::run(acc, xr, wv);
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

// Copy of a weight into a VGPR, as an asm statement so that it stays ahead
// of the taps that follow it.
__device__ __forceinline__ float to_vgpr(float w) {
    float v;
    asm volatile("v_mov_b32 %0, %1" : "=v"(v) : "s"(w));
    return v;
}

// The 4 taps of one kernel of a centre+3 shape.  fp32 with R >= 3: the
// weights of the shifted taps are copied to VGPRs first, the same-column
// taps (the centre at least) run next and the shifted taps last, so at least
// R FMAs separate any VALU write from a DPP read and the shifted taps need no
// wait states.  Otherwise the taps run in position order with wait states.
template <int J, int Q, int R>
__device__ __forceinline__ void tap_same(float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
    if constexpr (Q % 3 == 1) tap_q<Q, R, true>(a, x, w[J]);
}
template <int J, int Q, int R>
__device__ __forceinline__ void tap_shift(float (&a)[R], const float (&x)[R + 2], const float (&wv)[4]) {
    if constexpr (Q % 3 != 1) tap_q<Q, R, false, false>(a, x, wv[J]);
}
template <int DT, int R, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void kernel_taps(float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
    if constexpr (DT == DT_F32 && R >= 3) {
        float wv[4] = {w[0], w[1], w[2], w[3]};
        if constexpr (Q0 % 3 != 1) wv[0] = to_vgpr(w[0]);
        if constexpr (Q1 % 3 != 1) wv[1] = to_vgpr(w[1]);
        if constexpr (Q2 % 3 != 1) wv[2] = to_vgpr(w[2]);
        if constexpr (Q3 % 3 != 1) wv[3] = to_vgpr(w[3]);
        tap_same<0, Q0, R>(a, x, w);
        tap_same<1, Q1, R>(a, x, w);
        tap_same<2, Q2, R>(a, x, w);
        tap_same<3, Q3, R>(a, x, w);
        tap_shift<0, Q0, R>(a, x, wv);
        tap_shift<1, Q1, R>(a, x, wv);
        tap_shift<2, Q2, R>(a, x, wv);
        tap_shift<3, Q3, R>(a, x, wv);
    } else {
        constexpr bool WS = DT == DT_F32;
        tap_q<Q0, R, WS>(a, x, w[0]);
        tap_q<Q1, R, WS>(a, x, w[1]);
        tap_q<Q2, R, WS>(a, x, w[2]);
        tap_q<Q3, R, WS>(a, x, w[3]);
    }
}

// ------------------------------------------------------------------ runs
struct RunCtx;

// Scalar buffer loads (wave-uniform, into SGPRs) of the packed kernels'
// channel indices and weights: 32-bit offsets from a descriptor, no 64-bit
// address arithmetic per kernel.

__device__ __forceinline__ int32x4 scalar_rsrc(const void* p, int bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    return int32x4{int32_t(uint32_t(a)), int32_t(uint32_t(a >> 32) & 0xffffu), bytes, 0x00020000};
}

struct Meta {
    int32x4 ci;   // cin_idx, keep entries
    int32x4 w;    // values, keep * 4 weights
};

// Channel index of kernel k (callers keep k inside the filter's kernels).
__device__ __forceinline__ int meta_ci(const Meta& m, int k) { return psc_sbuf_i32(m.ci, k * 4, 0); }

// The 4 weights of kernel k as floats (fp32: SGPRs; fp16: widened).
template <int DT>
__device__ __forceinline__ void meta_w(const Meta& m, int k, float (&w)[4]) {
    if constexpr (DT == DT_F32) {
        const psc_f32x4 v = psc_sbuf_f32x4(m.w, k * 16, 0);
        w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
    } else {
        const psc_i32x2 v = psc_sbuf_i32x2(m.w, k * 8, 0);
        w[0] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(v.x))));
        w[1] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(v.x) >> 16)));
        w[2] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(v.y))));
        w[3] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(v.y) >> 16)));
    }
}

struct RunCtx {
    Meta m;
    __amdgpu_buffer_rsrc_t xr;   // x, bounded to its size
    int chan_bytes;              // bytes of one input channel plane
};

// The R+2 input rows of channel ci in this lane's column (zero outside the
// image: those offsets lie past the buffer range).
template <int DT, int R>
__device__ __forceinline__ void load_rows(const RunCtx& c, const uint32_t (&vo)[R + 2], int ci,
                                          float (&xr)[R + 2]) {
    // every offset of a buffer load is range-checked: a malformed channel
    // index reads zeros or other data of x, never memory outside it
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
__device__ __forceinline__ void run_kernels(const RunCtx& c, const uint32_t (&vo)[R + 2], int k, int e,
                                            float (&acc)[R], TapFn taps) {
    const int last = e - 1;
    float wA[4], wB[4];
    meta_w<DT>(c.m, k, wA);
    int kk = k + 1 <= last ? k + 1 : last;
    int ciB = meta_ci(c.m, kk);
    meta_w<DT>(c.m, kk, wB);
    float xA[R + 2], xB[R + 2];
    load_rows<DT, R>(c, vo, meta_ci(c.m, k), xA);
    while (k + 1 < e) {
        load_rows<DT, R>(c, vo, ciB, xB);                      // rows of kernel k+1
        kk = k + 2 <= last ? k + 2 : last;
        const int ciA2 = meta_ci(c.m, kk);
        float wA2[4];
        meta_w<DT>(c.m, kk, wA2);
        kk = k + 3 <= last ? k + 3 : last;
        const int ciB2 = meta_ci(c.m, kk);
        float wB2[4];
        meta_w<DT>(c.m, kk, wB2);
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
__device__ __forceinline__ void run_shape(const RunCtx& c, const uint32_t (&vo)[R + 2], int k, int e,
                                          float (&acc)[R]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    run_kernels<DT, R>(c, vo, k, e, acc, [](float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
        kernel_taps<DT, R, Q0, Q1, Q2, Q3>(a, x, w);
    });
}

// Any 4-of-9 mask: the taps are chosen per kernel by uniform branches.
template <int DT, int R>
__device__ __forceinline__ void run_generic(unsigned mask, const RunCtx& c, const uint32_t (&vo)[R + 2],
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

// ------------------------------------------------------------------ LDS-staged rows
// A 64-lane dword load runs at full rate only when every quarter-wave's 64
// bytes lie in one 128-byte line.  Image rows start at arbitrary 4-byte
// offsets, so a direct row load usually straddles lines and costs about twice
// as much.  In the staged form a wave copies, per kernel, the input rows its
// segments need -- for full-row segments these are contiguous "runs" of the
// channel plane, one per image the wave touches -- into its own LDS area with
// buffer-to-LDS loads that start on 64-byte boundaries, and then each lane
// reads its rows from LDS.  The copy of the next kernel's rows overlaps the
// current kernel's FMAs; no other wave touches the area, so no barrier is
// needed.
constexpr int kMaxRuns = 4;
constexpr int kMaxDma = 4;     // buffer-to-LDS loads (1 KiB each: 16 bytes a lane) per run
constexpr int kLdsCopy = 4096; // bytes between the two copies of a wave's runs

typedef __attribute__((address_space(3))) void lds_void_t;

// NR: runs per wave the code is compiled for (1, or up to kMaxRuns).
template <int NR>
struct LdsCtx {
    Meta m;
    __amdgpu_buffer_rsrc_t xr;            // x, bounded to its size
    int chan_bytes;                       // bytes of one input channel plane
    int nruns;
    int run_base[NR];                     // byte offset in x of run j, channel 0
    int run_lds[NR];                      // LDS address of run j's first byte
    int run_len[NR];                      // bytes of run j
    uint32_t vlane;                       // lane * 16
};

// s_waitcnt immediates (GFX9 encoding): wait on one counter only.
constexpr int kWaitVm0 = 0x0F70;          // vmcnt(0)
constexpr int kWaitLgkm0 = 0xC07F;        // lgkmcnt(0)

#define PSC_DMA(Q) \
    __builtin_amdgcn_raw_ptr_buffer_load_lds(c.xr, dst, 16, c.vlane, soff, (Q) * 1024, 0)

// Copy the runs of channel ci into this wave's LDS area.  Each load moves
// 1 KiB (16 bytes a lane) from a 64-byte boundary on; the LDS destination is
// shifted back by the same misalignment, so byte t of run j always lands at
// run_lds[j] + t.  Bytes past the end of x read as zero (every offset of a
// buffer load is range-checked).
template <int NR>
__device__ __forceinline__ void dma_rows(const LdsCtx<NR>& c, int ci, int buf) {
#if defined(__HIP_DEVICE_COMPILE__)   // the 16-byte form exists only for the gfx950 device pass
    // a malformed channel index reads zeros or other data of x (every offset
    // of a buffer load is range-checked)
    const int coff = ci * c.chan_bytes;
#pragma unroll
    for (int j = 0; j < NR; ++j) {
        if (NR == 1 || j < c.nruns) {
            const int start = c.run_base[j] + coff;
            const int mis = start & 63;
            const int soff = start - mis;
            lds_void_t* dst = (lds_void_t*)(uintptr_t)(uint32_t)(c.run_lds[j] + buf * kLdsCopy - mis);
            const int cnt = (mis + c.run_len[j] + 1023) >> 10;
            PSC_DMA(0);
            if (cnt > 1) PSC_DMA(1);
            if (cnt > 2) PSC_DMA(2);
            if (cnt > 3) PSC_DMA(3);
        }
    }
#endif
}
#undef PSC_DMA

// The R+2 rows of this lane from LDS copy OFF / kLdsCopy (lo: LDS byte
// addresses in copy 0; padding rows and columns point at a zeroed area that
// both copies share).
template <int DT, int R, int OFF>
__device__ __forceinline__ void read_rows(const uint32_t (&lo)[R + 2], float (&xr)[R + 2]) {
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
        if constexpr (DT == DT_F32)
            xr[r] = *(const __attribute__((address_space(3))) float*)(uintptr_t)(lo[r] + OFF);
        else
            xr[r] = float(*(const __attribute__((address_space(3))) _Float16*)(uintptr_t)(lo[r] + OFF));
    }
}

// One kernel whose rows sit (or are arriving) in copy B of the wave's LDS
// area: wait for them, start the copy of kernel k+1 (channel ci; also across
// the segment end, for the next segment) into the other copy, read this
// lane's rows and run the FMAs with the weights w of kernel k; then refill w
// and ci with the weights of kernel k+2 and the channel of kernel k+3, for
// the next trip of the same copy.
template <int DT, int R, int NR, int B, class TapFn>
__device__ __forceinline__ void lds_trip(const LdsCtx<NR>& c, const uint32_t (&lo)[R + 2], int k, int s1,
                                         float (&w)[4], int& ci, float (&acc)[R], TapFn taps) {
    const int last = s1 - 1;
    __builtin_amdgcn_s_waitcnt(kWaitVm0);                // rows of kernel k are in LDS
    asm volatile("" ::: "memory");
    if (k + 1 < s1) dma_rows<NR>(c, ci, B ^ 1);           // rows of kernel k+1
    float xr[R + 2];
    read_rows<DT, R, B * kLdsCopy>(lo, xr);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);              // rows in registers
    asm volatile("" ::: "memory");
    taps(acc, xr, w);
    meta_w<DT>(c.m, k + 2 <= last ? k + 2 : last, w);
    ci = meta_ci(c.m, k + 3 <= last ? k + 3 : last);
}

// Kernels [k, e) of one pattern segment, the first one's rows in copy B0.
// Pairs of kernels per trip, one in each copy.  Each copy has its own set of
// weight and channel registers, refilled two kernels ahead, so every
// prefetch is consumed only after the loop's back edge.  An odd last kernel
// runs after the loop: the single loop exit keeps the accumulators in place.
// Returns the copy that kernel e's rows go to.
template <int DT, int R, int NR, int B0, class TapFn>
__device__ __forceinline__ int run_pairs_lds(const LdsCtx<NR>& c, const uint32_t (&lo)[R + 2], int k, int e,
                                             int s1, float (&acc)[R], TapFn taps) {
    const int last = s1 - 1;
    float wA[4], wB[4];
    meta_w<DT>(c.m, k, wA);
    meta_w<DT>(c.m, k + 1 <= last ? k + 1 : last, wB);
    int ciA = meta_ci(c.m, k + 1 <= last ? k + 1 : last);
    int ciB = meta_ci(c.m, k + 2 <= last ? k + 2 : last);
    while (k + 1 < e) {
        lds_trip<DT, R, NR, B0>(c, lo, k, s1, wA, ciA, acc, taps);
        lds_trip<DT, R, NR, B0 ^ 1>(c, lo, k + 1, s1, wB, ciB, acc, taps);
        k += 2;
    }
    if (k < e) {
        lds_trip<DT, R, NR, B0>(c, lo, k, s1, wA, ciA, acc, taps);
        return B0 ^ 1;
    }
    return B0;
}

template <int DT, int R, int NR, class TapFn>
__device__ __forceinline__ int run_kernels_lds(const LdsCtx<NR>& c, const uint32_t (&lo)[R + 2], int k, int e,
                                               int s1, int par, float (&acc)[R], TapFn taps) {
    return par == 0 ? run_pairs_lds<DT, R, NR, 0>(c, lo, k, e, s1, acc, taps)
                    : run_pairs_lds<DT, R, NR, 1>(c, lo, k, e, s1, acc, taps);
}

template <int DT, int R, int NR, int MASK>
__device__ __forceinline__ int run_shape_lds(const LdsCtx<NR>& c, const uint32_t (&lo)[R + 2], int k, int e,
                                             int s1, int par, float (&acc)[R]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    return run_kernels_lds<DT, R, NR>(c, lo, k, e, s1, par, acc,
                                      [](float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
        kernel_taps<DT, R, Q0, Q1, Q2, Q3>(a, x, w);
    });
}

template <int DT, int R, int NR>
__device__ __forceinline__ int run_generic_lds(unsigned mask, const LdsCtx<NR>& c, const uint32_t (&lo)[R + 2],
                                               int k, int e, int s1, int par, float (&acc)[R]) {
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
    return run_kernels_lds<DT, R, NR>(c, lo, k, e, s1, par, acc,
                                      [=](float (&a)[R], const float (&x)[R + 2], const float (&w)[4]) {
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
__device__ __forceinline__ void run_pattern(int shape, unsigned mask, const RunCtx& c,
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

#define PSC_SHAPE_CASE(I) \
    case I: return run_shape_lds<DT, R, NR, kCentre3.code[I]>(c, lo, k, e, s1, par, acc);
#define PSC_SHAPE_CASE8(I)                                                                     \
    PSC_SHAPE_CASE(I) PSC_SHAPE_CASE(I + 1) PSC_SHAPE_CASE(I + 2) PSC_SHAPE_CASE(I + 3)        \
    PSC_SHAPE_CASE(I + 4) PSC_SHAPE_CASE(I + 5) PSC_SHAPE_CASE(I + 6) PSC_SHAPE_CASE(I + 7)

template <int DT, int R, int NR>
__device__ __forceinline__ int run_pattern_lds(int shape, unsigned mask, const LdsCtx<NR>& c,
                                               const uint32_t (&lo)[R + 2], int k, int e, int s1, int par,
                                               float (&acc)[R]) {
    switch (shape) {
        PSC_SHAPE_CASE8(0)
        PSC_SHAPE_CASE8(8)
        PSC_SHAPE_CASE8(16)
        PSC_SHAPE_CASE8(24)
        PSC_SHAPE_CASE8(32)
        PSC_SHAPE_CASE8(40)
        PSC_SHAPE_CASE8(48)
        default: return run_generic_lds<DT, R, NR>(mask, c, lo, k, e, s1, par, acc);
    }
}
#undef PSC_SHAPE_CASE8
#undef PSC_SHAPE_CASE

// ------------------------------------------------------------------ wide rows
// Images 28..252 columns wide, width a multiple of 4: a lane owns 4 adjacent
// output columns and R rows of a full-row band, and each input row arrives as
// one aligned load per lane (16 bytes fp32, 8 bytes fp16), so one load
// instruction feeds 4 columns' taps.  The neighbour columns left of the
// lane's first and right of its last column come from the adjacent lanes
// through DPP; the other taps read the lane's own values.  Segments are
// padded to a multiple of 4 lanes (with rows on 64-byte boundaries, every
// 4-lane group of a load stays in one 64-byte block).

// One output row of a tap: a[c] += w * x[c + DS - 1] over the lane's 4
// columns, with x[-1] / x[4] taken from the lane to the left / right.
template <int DS> struct TapRow4;
#define PSC_A4 [a0] "+v"(a[0]), [a1] "+v"(a[1]), [a2] "+v"(a[2]), [a3] "+v"(a[3])
#define PSC_X4 [x0] "v"(x[0]), [x1] "v"(x[1]), [x2] "v"(x[2]), [x3] "v"(x[3])
template <> struct TapRow4<1> {
    __device__ __forceinline__ static void run(float* a, const float* x, float ws, float) {
        asm volatile("v_fmac_f32_e32 %[a0], %[ws], %[x0]\n"
                     "v_fmac_f32_e32 %[a1], %[ws], %[x1]\n"
                     "v_fmac_f32_e32 %[a2], %[ws], %[x2]\n"
                     "v_fmac_f32_e32 %[a3], %[ws], %[x3]\n"
                     : PSC_A4 : PSC_X4, [ws] "s"(ws));
    }
};
template <> struct TapRow4<0> {
    __device__ __forceinline__ static void run(float* a, const float* x, float ws, float wv) {
        asm volatile("v_fmac_f32_dpp %[a0], %[x3], %[wv] wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
                     "v_fmac_f32_e32 %[a1], %[ws], %[x0]\n"
                     "v_fmac_f32_e32 %[a2], %[ws], %[x1]\n"
                     "v_fmac_f32_e32 %[a3], %[ws], %[x2]\n"
                     : PSC_A4 : PSC_X4, [ws] "s"(ws), [wv] "v"(wv));
    }
};
template <> struct TapRow4<2> {
    __device__ __forceinline__ static void run(float* a, const float* x, float ws, float wv) {
        asm volatile("v_fmac_f32_e32 %[a0], %[ws], %[x1]\n"
                     "v_fmac_f32_e32 %[a1], %[ws], %[x2]\n"
                     "v_fmac_f32_e32 %[a2], %[ws], %[x3]\n"
                     "v_fmac_f32_dpp %[a3], %[x0], %[wv] wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
                     : PSC_A4 : PSC_X4, [ws] "s"(ws), [wv] "v"(wv));
    }
};
#undef PSC_X4
#undef PSC_A4

// Tap at kernel position Q over the lane's R rows; x[r] holds the 4 columns
// of input row r (r = 0 is the row above the lane's first output row).
template <int Q, int R>
__device__ __forceinline__ void tap4(float (&acc)[4 * R], const float (&x)[R + 2][4], float ws, float wv) {
#pragma unroll
    for (int r = 0; r < R; ++r) TapRow4<Q % 3>::run(&acc[4 * r], x[r + Q / 3], ws, wv);
}

template <int J, int Q, int R>
__device__ __forceinline__ void tap4_same(float (&a)[4 * R], const float (&x)[R + 2][4], const float (&w)[4]) {
    if constexpr (Q % 3 == 1) tap4<Q, R>(a, x, w[J], 0.f);
}
template <int J, int Q, int R>
__device__ __forceinline__ void tap4_shift(float (&a)[4 * R], const float (&x)[R + 2][4], const float (&w)[4],
                                           const float (&wv)[4]) {
    if constexpr (Q % 3 != 1) tap4<Q, R>(a, x, w[J], wv[J]);
}

// The 4 taps of one kernel: the shifted taps' weights are copied to VGPRs
// first and the same-column taps (the centre at least: 4R FMAs) run before
// the shifted ones, so no DPP read follows a VALU write of its operands
// within two wait states.
template <int R, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void kernel_taps4(float (&a)[4 * R], const float (&x)[R + 2][4], const float (&w)[4]) {
    float wv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (Q0 % 3 != 1) wv[0] = to_vgpr(w[0]);
    if constexpr (Q1 % 3 != 1) wv[1] = to_vgpr(w[1]);
    if constexpr (Q2 % 3 != 1) wv[2] = to_vgpr(w[2]);
    if constexpr (Q3 % 3 != 1) wv[3] = to_vgpr(w[3]);
    tap4_same<0, Q0, R>(a, x, w);
    tap4_same<1, Q1, R>(a, x, w);
    tap4_same<2, Q2, R>(a, x, w);
    tap4_same<3, Q3, R>(a, x, w);
    tap4_shift<0, Q0, R>(a, x, w, wv);
    tap4_shift<1, Q1, R>(a, x, w, wv);
    tap4_shift<2, Q2, R>(a, x, w, wv);
    tap4_shift<3, Q3, R>(a, x, w, wv);
}

template <int R>
__device__ __forceinline__ void kernel_taps4_dyn(const int (&q)[4], float (&a)[4 * R], const float (&x)[R + 2][4],
                                                 const float (&w)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float wv = to_vgpr(w[j]);
        asm volatile("s_nop 1" ::: "memory");   // wait states before the DPP read of wv
        switch (q[j]) {
            case 0: tap4<0, R>(a, x, w[j], wv); break;
            case 1: tap4<1, R>(a, x, w[j], wv); break;
            case 2: tap4<2, R>(a, x, w[j], wv); break;
            case 3: tap4<3, R>(a, x, w[j], wv); break;
            case 4: tap4<4, R>(a, x, w[j], wv); break;
            case 5: tap4<5, R>(a, x, w[j], wv); break;
            case 6: tap4<6, R>(a, x, w[j], wv); break;
            case 7: tap4<7, R>(a, x, w[j], wv); break;
            default: tap4<8, R>(a, x, w[j], wv); break;
        }
    }
}

// The R+2 input rows (4 columns each) of channel ci for this lane (fp32).
template <int R>
__device__ __forceinline__ void load_rows4(const RunCtx& c, const uint32_t (&vo)[R + 2], int ci,
                                           float (&x)[R + 2][4]) {
    const int soff = __builtin_amdgcn_readfirstlane(ci * c.chan_bytes);
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
        const psc_f32x4 v = __builtin_bit_cast(psc_f32x4, __builtin_amdgcn_raw_buffer_load_b128(c.xr, vo[r], soff, 0));
        x[r][0] = v.x, x[r][1] = v.y, x[r][2] = v.z, x[r][3] = v.w;
    }
}

// fp16: the R+2 rows as raw words (4 halves in 2 words per row), widened
// just before their taps.
template <int R> struct Half4Rows {
    uint32_t d[R + 2][2];
};

template <int R>
__device__ __forceinline__ void load_rows4_f16(const RunCtx& c, const uint32_t (&vo)[R + 2], int ci,
                                               Half4Rows<R>& p) {
    const int soff = __builtin_amdgcn_readfirstlane(ci * c.chan_bytes);
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
        const psc_i32x2 v = __builtin_bit_cast(psc_i32x2, __builtin_amdgcn_raw_buffer_load_b64(c.xr, vo[r], soff, 0));
        p.d[r][0] = uint32_t(v.x), p.d[r][1] = uint32_t(v.y);
    }
}

// Widen to fp32; then an asm the compiler sees as writing the first and last
// column of every row (the ones the neighbours read by DPP: no VALU write of
// them can follow) and the two wait states a DPP read needs after a VALU
// write of its source.
template <int R>
__device__ __forceinline__ void unpack_rows4(const Half4Rows<R>& p, float (&x)[R + 2][4]) {
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            x[r][q] = float(__builtin_bit_cast(_Float16, uint16_t(p.d[r][q / 2] >> (16 * (q & 1)))));
    }
#pragma unroll
    for (int r = 0; r < R + 2; ++r) asm volatile("" : "+v"(x[r][0]), "+v"(x[r][3]));
    asm volatile("s_nop 1");
}

// Kernels [k, e) of one pattern segment share; two per trip as in the
// one-column form.
template <int DT, int R, class TapFn>
__device__ __forceinline__ void run_kernels4(const RunCtx& c, const uint32_t (&vo)[R + 2], int k, int e,
                                             float (&acc)[4 * R], TapFn taps) {
    const int last = e - 1;
    float wA[4], wB[4];
    meta_w<DT>(c.m, k, wA);
    int kk = k + 1 <= last ? k + 1 : last;
    int ciB = meta_ci(c.m, kk);
    meta_w<DT>(c.m, kk, wB);
    if constexpr (DT == DT_F32) {
        float xA[R + 2][4], xB[R + 2][4];
        load_rows4<R>(c, vo, meta_ci(c.m, k), xA);
        while (k + 1 < e) {
            load_rows4<R>(c, vo, ciB, xB);                     // rows of kernel k+1
            kk = k + 2 <= last ? k + 2 : last;
            const int ciA2 = meta_ci(c.m, kk);
            float wA2[4];
            meta_w<DT>(c.m, kk, wA2);
            kk = k + 3 <= last ? k + 3 : last;
            const int ciB2 = meta_ci(c.m, kk);
            float wB2[4];
            meta_w<DT>(c.m, kk, wB2);
            taps(acc, xA, wA);                                 // kernel k
            load_rows4<R>(c, vo, ciA2, xA);                    // rows of kernel k+2
            taps(acc, xB, wB);                                 // kernel k+1
            k += 2;
            wA[0] = wA2[0], wA[1] = wA2[1], wA[2] = wA2[2], wA[3] = wA2[3];
            wB[0] = wB2[0], wB[1] = wB2[1], wB[2] = wB2[2], wB[3] = wB2[3];
            ciB = ciB2;
        }
        if (k < e) taps(acc, xA, wA);
    } else {
        Half4Rows<R> pA, pB;
        load_rows4_f16<R>(c, vo, meta_ci(c.m, k), pA);
        while (k + 1 < e) {
            load_rows4_f16<R>(c, vo, ciB, pB);                 // rows of kernel k+1
            kk = k + 2 <= last ? k + 2 : last;
            const int ciA2 = meta_ci(c.m, kk);
            float wA2[4];
            meta_w<DT>(c.m, kk, wA2);
            kk = k + 3 <= last ? k + 3 : last;
            const int ciB2 = meta_ci(c.m, kk);
            float wB2[4];
            meta_w<DT>(c.m, kk, wB2);
            {
                float x[R + 2][4];
                unpack_rows4<R>(pA, x);
                taps(acc, x, wA);                              // kernel k
            }
            load_rows4_f16<R>(c, vo, ciA2, pA);                // rows of kernel k+2
            {
                float x[R + 2][4];
                unpack_rows4<R>(pB, x);
                taps(acc, x, wB);                              // kernel k+1
            }
            k += 2;
            wA[0] = wA2[0], wA[1] = wA2[1], wA[2] = wA2[2], wA[3] = wA2[3];
            wB[0] = wB2[0], wB[1] = wB2[1], wB[2] = wB2[2], wB[3] = wB2[3];
            ciB = ciB2;
        }
        if (k < e) {
            float x[R + 2][4];
            unpack_rows4<R>(pA, x);
            taps(acc, x, wA);
        }
    }
}

template <int DT, int R, int MASK>
__device__ __forceinline__ void run_shape4(const RunCtx& c, const uint32_t (&vo)[R + 2], int k, int e,
                                           float (&acc)[4 * R]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    run_kernels4<DT, R>(c, vo, k, e, acc, [](float (&a)[4 * R], const float (&x)[R + 2][4], const float (&w)[4]) {
        kernel_taps4<R, Q0, Q1, Q2, Q3>(a, x, w);
    });
}

template <int DT, int R>
__device__ __forceinline__ void run_generic4(unsigned mask, const RunCtx& c, const uint32_t (&vo)[R + 2], int k,
                                             int e, float (&acc)[4 * R]) {
    int q[4] = {4, 4, 4, 4}, seen = 0;
#pragma unroll
    for (int p = 0; p < 9; ++p) {
        if ((mask >> p) & 1u) {
            if (seen == 0) q[0] = p;
            else if (seen == 1) q[1] = p;
            else if (seen == 2) q[2] = p;
            else if (seen == 3) q[3] = p;
            ++seen;
        }
    }
    run_kernels4<DT, R>(c, vo, k, e, acc, [=](float (&a)[4 * R], const float (&x)[R + 2][4], const float (&w)[4]) {
        kernel_taps4_dyn<R>(q, a, x, w);
    });
}

#define PSC_SHAPE_CASE(I) \
    case I: run_shape4<DT, R, kCentre3.code[I]>(c, vo, k, e, acc); return;
#define PSC_SHAPE_CASE8(I)                                                                     \
    PSC_SHAPE_CASE(I) PSC_SHAPE_CASE(I + 1) PSC_SHAPE_CASE(I + 2) PSC_SHAPE_CASE(I + 3)        \
    PSC_SHAPE_CASE(I + 4) PSC_SHAPE_CASE(I + 5) PSC_SHAPE_CASE(I + 6) PSC_SHAPE_CASE(I + 7)
template <int DT, int R>
__device__ __forceinline__ void run_pattern4(int shape, unsigned mask, const RunCtx& c, const uint32_t (&vo)[R + 2],
                                             int k, int e, float (&acc)[4 * R]) {
    switch (shape) {
        PSC_SHAPE_CASE8(0)
        PSC_SHAPE_CASE8(8)
        PSC_SHAPE_CASE8(16)
        PSC_SHAPE_CASE8(24)
        PSC_SHAPE_CASE8(32)
        PSC_SHAPE_CASE8(40)
        PSC_SHAPE_CASE8(48)
        default: run_generic4<DT, R>(mask, c, vo, k, e, acc); return;
    }
}
#undef PSC_SHAPE_CASE8
#undef PSC_SHAPE_CASE

// Wide form of the kernel: same blocks, shares, reduction and epilogue as
// the one-column form, 4 columns per lane.  With 4 rows per lane the
// compiler is held to 128 VGPRs (4 waves per SIMD).
template <int DT, int R>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(R <= 2 ? 6 : 4))) void k_conv_wide(
    const typename Elt<DT>::T* __restrict__ x, const int32_t* __restrict__ perm, const int32_t* __restrict__ seg_ptr,
    const int32_t* __restrict__ cin_idx, const typename Elt<DT>::T* __restrict__ vals,
    const typename Elt<DT>::T* __restrict__ bias, typename Elt<DT>::T* __restrict__ y, Geo g) {
    using E = Elt<DT>;
    constexpr int ESZ = int(sizeof(typename E::T));
    constexpr int ROWS = R + 2;
    extern __shared__ float psc_smem4[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int gf = wave / g.KS, sp = wave - gf * g.KS;
    const int b = blockIdx.x;
    int lb = b;
    if (g.nblocks >= 8) {
        const int per = g.nblocks / 8, rem = g.nblocks % 8;
        const int xcd = b % 8, slot = b / 8;
        lb = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
    }
    const int fg = lb % g.groups_x, sgrp = lb / g.groups_x;
    const int i = fg * g.FW + gf;
    const bool has_filter = i < g.cout;

    // ---- lane geometry: lane cidx of segment s holds columns 4*cidx .. +3
    const int s = lane / g.seg_len, cidx = lane - s * g.seg_len;
    const int u = sgrp * g.S + s;
    int col0 = -1, nimg = 0, h0 = 0;
    if (s < g.S && u < g.U) {
        nimg = u / g.RB;
        h0 = (u % g.RB) * R;
        if (4 * cidx < g.W) col0 = 4 * cidx;
    }
    const int plane = g.H * g.W;
    uint32_t vo[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        const int row = h0 - 1 + r;
        vo[r] = (col0 >= 0 && row >= 0 && row < g.H) ? uint32_t(nimg * g.cin * plane + row * g.W + col0) * uint32_t(ESZ)
                                                     : 0x80000000u;
    }
    float acc[4 * R];
#pragma unroll
    for (int r = 0; r < 4 * R; ++r) acc[r] = 0.f;

    const int* segp = seg_ptr + i * (g.m + 1);
    if (has_filter) {
        const int f0 = segp[0], f1 = segp[g.m];
        const int len = f1 - f0;
        const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
        const RunCtx ctx{Meta{scalar_rsrc(cin_idx, g.keep * 4), scalar_rsrc(vals, g.keep * 4 * ESZ)},
                         __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes,
                                                           0x00020000),
                         __builtin_amdgcn_readfirstlane(plane * ESZ)};
        for (int p = 0; p < g.m; ++p) {
            int k0 = segp[p], k1 = segp[p + 1];
            k0 = k0 < s0 ? s0 : k0;
            k1 = k1 > s1 ? s1 : k1;
            if (k0 < k1) run_pattern4<DT, R>(g.shape[p], g.mask[p], ctx, vo, k0, k1, acc);
        }
    }

    if (g.KS > 1) {
        float (*red)[4 * R][64] = reinterpret_cast<float (*)[4 * R][64]>(psc_smem4);
        for (int slot = 0; slot < g.FW; ++slot) {
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < 4 * R; ++r) red[sp][r][lane] = acc[r];
            }
            __syncthreads();
            if (slot == gf) {
#pragma unroll
                for (int r = 0; r < 4 * R; ++r) {
                    float v = 0.f;
                    for (int t = 0; t < g.KS; ++t) v += red[t][r][lane];
                    acc[r] = v;
                }
            }
            __syncthreads();
        }
    }
    if (!has_filter || col0 < 0) return;
    const int f = perm[i];
    const float bv = bias ? E::load(bias, f) : 0.f;
    if constexpr (R % 2 == 0) {
        if (g.pool) {
            // 2x2/2 max-pool: the lane's 4 columns give 2 pooled columns
            const int OH = g.H / 2, OW = g.W / 2;
            typename E::T* yp = y + (nimg * g.cout + f) * (OH * OW) + col0 / 2;
#pragma unroll
            for (int j = 0; j < R / 2; ++j) {
                const int prow = h0 / 2 + j;
                if (prow < OH && (j % g.KS) == sp) {
                    const float* a0 = &acc[8 * j];
                    float p0 = fmaxf(fmaxf(a0[0], a0[1]), fmaxf(a0[4], a0[5])) + bv;
                    float p1 = fmaxf(fmaxf(a0[2], a0[3]), fmaxf(a0[6], a0[7])) + bv;
                    if (g.relu) {
                        p0 = p0 > 0.f ? p0 : 0.f;
                        p1 = p1 > 0.f ? p1 : 0.f;
                    }
                    yp[prow * OW] = E::from_f(p0);
                    yp[prow * OW + 1] = E::from_f(p1);
                }
            }
            return;
        }
    }
    typename E::T* yp = y + (nimg * g.cout + f) * plane + col0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = h0 + r;
        if (row < g.H && (r % g.KS) == sp) {
            psc_f32x4 v{acc[4 * r] + bv, acc[4 * r + 1] + bv, acc[4 * r + 2] + bv, acc[4 * r + 3] + bv};
            if (g.relu) {
                v.x = v.x > 0.f ? v.x : 0.f;
                v.y = v.y > 0.f ? v.y : 0.f;
                v.z = v.z > 0.f ? v.z : 0.f;
                v.w = v.w > 0.f ? v.w : 0.f;
            }
            if constexpr (DT == DT_F32) {
                *reinterpret_cast<psc_f32x4*>(yp + row * g.W) = v;
            } else {
                // 4 halves, 8 bytes: col0 and the width are multiples of 4
                const uint32_t lo = uint32_t(E::from_f(v.x)) | (uint32_t(E::from_f(v.y)) << 16);
                const uint32_t hi = uint32_t(E::from_f(v.z)) | (uint32_t(E::from_f(v.w)) << 16);
                *reinterpret_cast<psc_i32x2*>(yp + row * g.W) = psc_i32x2{int32_t(lo), int32_t(hi)};
            }
        }
    }
}

// ------------------------------------------------------------------ kernel
// LDS = true stages the input rows through per-wave LDS (full-row segments
// only; NR: runs per wave compiled for); LDS = false loads them straight
// into registers.
template <int DT, int R, bool LDS, int NR>
__global__ __launch_bounds__(512) void k_conv_stream(const typename Elt<DT>::T* __restrict__ x,
                                                     const int32_t* __restrict__ perm,
                                                     const int32_t* __restrict__ seg_ptr,
                                                     const int32_t* __restrict__ cin_idx,
                                                     const typename Elt<DT>::T* __restrict__ vals,
                                                     const typename Elt<DT>::T* __restrict__ bias,
                                                     typename Elt<DT>::T* __restrict__ y, Geo g) {
    using E = Elt<DT>;
    constexpr int ROWS = R + 2;
    constexpr int ESZ = int(sizeof(typename E::T));
    // dynamic LDS: the per-wave row areas (LDS form), then, after all
    // kernels, the partial sums of the KS shares of a filter
    extern __shared__ float psc_smem[];

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

    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;

    const int* segp = seg_ptr + i * (g.m + 1);
    int s0 = 0, s1 = 0;
    if (has_filter) {
        const int f0 = segp[0], f1 = segp[g.m];
        // share sp: the sp-th of KS equal contiguous ranges of the filter's
        // kernels, which crosses few pattern segments
        const int len = f1 - f0;
        s0 = f0 + len * sp / g.KS;
        s1 = f0 + len * (sp + 1) / g.KS;
    }
    const auto xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes,
                                                      0x00020000);
    const Meta meta{scalar_rsrc(cin_idx, g.keep * 4), scalar_rsrc(vals, g.keep * 4 * ESZ)};

    if constexpr (!LDS) {
        // byte offset of this lane's column in each of its R+2 input rows of
        // channel 0; 2^31 (past the buffer range, reads zero) for padding
        uint32_t vo[ROWS];
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            const int row = h0 - 1 + r;
            vo[r] = (ld_col >= 0 && row >= 0 && row < g.H)
                        ? uint32_t(nimg * g.cin * plane + row * g.W + ld_col) * uint32_t(ESZ)
                        : 0x80000000u;
        }
        if (has_filter) {
            const RunCtx ctx{meta, xr, __builtin_amdgcn_readfirstlane(plane * ESZ)};
            for (int p = 0; p < g.m; ++p) {
                int k0 = segp[p], k1 = segp[p + 1];
                k0 = k0 < s0 ? s0 : k0;
                k1 = k1 > s1 ? s1 : k1;                     // malformed pointers stay in the share
                if (k0 < k1) run_pattern<DT, R>(g.shape[p], g.mask[p], ctx, vo, k0, k1, acc);
            }
        }
    } else {
        // ---- this wave's LDS area: nruns regions of g.region bytes (run j's
        // data starts 64 bytes in), then 64 zeroed bytes that padding reads
        const uint32_t area = uint32_t(uintptr_t((const __attribute__((address_space(3))) void*)psc_smem)) +
                              uint32_t(wave * g.wave_bytes);
        // copy 0 of the runs, copy 1 kLdsCopy bytes later, then the zero
        // area; padding reads of copy 1 land kLdsCopy past the zero area,
        // which is zeroed too
        const uint32_t zero_at = area + uint32_t(g.wave_bytes - 64 - kLdsCopy);
        if (lane < 16) *(__attribute__((address_space(3))) float*)(uintptr_t)(zero_at + lane * 4) = 0.f;
        if (lane < 16) *(__attribute__((address_space(3))) float*)(uintptr_t)(zero_at + kLdsCopy + lane * 4) = 0.f;
        // runs: the wave's segments grouped by image; run j covers the rows
        // of image n_first + j that its segments need
        const int RBn = g.RB;
        const int u_first = sgrp * g.S;
        const int u_last = (u_first + g.S < g.U ? u_first + g.S : g.U) - 1;
        const int n_first = u_first / RBn;
        LdsCtx<NR> ctx;
        ctx.m = meta;
        ctx.xr = xr;
        ctx.chan_bytes = __builtin_amdgcn_readfirstlane(plane * ESZ);
        ctx.nruns = __builtin_amdgcn_readfirstlane(u_first <= u_last ? u_last / RBn - n_first + 1 : 0);
        ctx.vlane = uint32_t(lane) * 16u;
#pragma unroll
        for (int j = 0; j < NR; ++j) {
            const int n = n_first + j;
            const int ua = u_first > n * RBn ? u_first : n * RBn;
            const int ub = u_last < n * RBn + RBn - 1 ? u_last : n * RBn + RBn - 1;
            int row_lo = (ua - n * RBn) * R - 1, row_hi = (ub - n * RBn + 1) * R + 1;
            row_lo = row_lo < 0 ? 0 : row_lo;
            row_hi = row_hi > g.H ? g.H : row_hi;
            // wave-uniform values: SGPR operands of the copies
            ctx.run_base[j] = __builtin_amdgcn_readfirstlane((n * g.cin * plane + row_lo * g.W) * ESZ);
            ctx.run_lds[j] = __builtin_amdgcn_readfirstlane(int(area) + j * g.region + 64);
            ctx.run_len[j] = __builtin_amdgcn_readfirstlane(j < ctx.nruns ? (row_hi - row_lo) * g.W * ESZ : 0);
        }
        // LDS byte address of each of this lane's rows (zero area for padding)
        uint32_t lo[ROWS];
        {
            const int jn = nimg - n_first;
            const int ua = u_first > nimg * RBn ? u_first : nimg * RBn;
            int row_lo = (ua - nimg * RBn) * R - 1;
            row_lo = row_lo < 0 ? 0 : row_lo;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int row = h0 - 1 + r;
                lo[r] = (ld_col >= 0 && row >= 0 && row < g.H)
                            ? area + uint32_t(jn * g.region + 64 + ((row - row_lo) * g.W + ld_col) * ESZ)
                            : zero_at;
            }
        }
        if (has_filter && s0 < s1) {
            dma_rows<NR>(ctx, meta_ci(meta, s0), 0);
            int par = 0;
            for (int p = 0; p < g.m; ++p) {
                int k0 = segp[p], k1 = segp[p + 1];
                k0 = k0 < s0 ? s0 : k0;
                k1 = k1 > s1 ? s1 : k1;                     // malformed pointers stay in the share
                if (k0 < k1) par = run_pattern_lds<DT, R, NR>(g.shape[p], g.mask[p], ctx, lo, k0, k1, s1, par, acc);
            }
        }
        __builtin_amdgcn_s_waitcnt(kWaitVm0);            // no copy into LDS is left in flight
    }

    // ---- add the KS partial sums of each filter in share order
    if (g.KS > 1) {
        float (*red)[R][64] = reinterpret_cast<float (*)[R][64]>(psc_smem);
        // the partial sums reuse the row areas: wait until every wave is done
        if constexpr (LDS) __syncthreads();
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
    if constexpr (R % 2 == 0) {
        if (g.pool) {
            // 2x2/2 max-pool of the output: rows 2j, 2j+1 of the lane, then
            // the column pair (even column, the lane to its right)
            float v[R / 2];
#pragma unroll
            for (int j = 0; j < R / 2; ++j) {
                const float m = fmaxf(acc[2 * j], acc[2 * j + 1]);
                v[j] = fmaxf(m, __shfl_down(m, 1));
            }
            if (!has_filter || out_col < 0 || (out_col & 1)) return;
            const int f = perm[i];
            const float bv = bias ? E::load(bias, f) : 0.f;
            const int OH = g.H / 2, OW = g.W / 2;
            typename E::T* yp = y + (nimg * g.cout + f) * (OH * OW) + out_col / 2;
#pragma unroll
            for (int j = 0; j < R / 2; ++j) {
                const int prow = h0 / 2 + j;
                if (prow < OH && (j % g.KS) == sp) {
                    float o = v[j] + bv;
                    if (g.relu) o = o > 0.f ? o : 0.f;
                    yp[prow * OW] = E::from_f(o);
                }
            }
            return;
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
hipError_t launch_wide(const PackedView& pk, const ConvArgs& a, const Geo& g, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    const int waves = g.FW * g.KS;
    const size_t smem = g.KS > 1 ? size_t(g.KS) * 4 * R * 64 * sizeof(float) : 0;
    hipLaunchKernelGGL((k_conv_wide<DT, R>), dim3(unsigned(g.nblocks)), dim3(unsigned(waves * 64)), smem, stream,
                       static_cast<const T*>(a.x), pk.filter_perm, pk.seg_ptr, pk.cin_idx,
                       static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), static_cast<T*>(a.y), g);
    return hipGetLastError();
}

template <int DT, int R>
hipError_t launch_r(const PackedView& pk, const ConvArgs& a, const Geo& g, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    const int waves = g.FW * g.KS;
    const size_t red = g.KS > 1 ? size_t(g.KS) * R * 64 * sizeof(float) : 0;
    const size_t rows = g.lds ? size_t(waves) * g.wave_bytes : 0;
    const size_t smem = red > rows ? red : rows;
    if (g.lds == 1)
        hipLaunchKernelGGL((k_conv_stream<DT, R, true, 1>), dim3(unsigned(g.nblocks)), dim3(unsigned(waves * 64)),
                           smem, stream, static_cast<const T*>(a.x), pk.filter_perm, pk.seg_ptr, pk.cin_idx,
                           static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), static_cast<T*>(a.y),
                           g);
    else if (g.lds > 1)
        hipLaunchKernelGGL((k_conv_stream<DT, R, true, kMaxRuns>), dim3(unsigned(g.nblocks)),
                           dim3(unsigned(waves * 64)), smem, stream, static_cast<const T*>(a.x), pk.filter_perm,
                           pk.seg_ptr, pk.cin_idx, static_cast<const T*>(pk.values), static_cast<const T*>(a.bias),
                           static_cast<T*>(a.y), g);
    else
        hipLaunchKernelGGL((k_conv_stream<DT, R, false, 1>), dim3(unsigned(g.nblocks)), dim3(unsigned(waves * 64)),
                           smem, stream, static_cast<const T*>(a.x), pk.filter_perm, pk.seg_ptr, pk.cin_idx,
                           static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), static_cast<T*>(a.y),
                           g);
    return hipGetLastError();
}

}  // namespace cs
}  // namespace psc
