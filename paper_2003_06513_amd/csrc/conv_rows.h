// Pattern-sparse 3x3 convolution, stride 1, zero padding 1 (Sec. 4.1 Eq. 1
// with the compiler optimisations of Sec. 3.4) for planes of at most 28
// columns: ONE OUTPUT ROW PER LANE.
//
// The column-per-lane kernels (conv_stream.h) load, for every kernel, R+2
// single elements per lane (one per input row of its column) for 4R FMAs.
// On small planes at large batch that load path is the bound.  Here a lane
// owns a whole output row of one image -- W accumulators -- and per kernel
// loads its own input row with 16-byte loads; the rows above and below come
// from the neighbouring lanes by DPP inside the FMA (v_fmac_f32_dpp
// wave_shr:1 / wave_shl:1), and the left and right neighbours of a column are
// other registers of the same lane.  So each loaded element feeds up to 12
// FMAs (load redundancy elimination at the register level), and a kernel
// costs 1..7 load instructions instead of R+2.
//
// Lane layout: a wave holds S = 64 / (H+1) images; image s occupies lanes
// s(H+1) .. s(H+1)+H-1 (row r in lane s(H+1)+r) and lane s(H+1)+H holds zero:
// the padding row below image s and above image s+1.  Padding columns cost
// nothing: the FMAs that would read them are left out at compile time.
//
// Stride 2 (ST = 2; the stage-entry convolutions): a lane owns output row i,
// OW = W/2 columns; it loads input rows 2i and 2i+1 (W values each) and takes
// row 2i-1 -- the odd row of the lane to the left -- by DPP.  Output column c
// reads input columns 2c-1, 2c and 2c+1, all registers of the lane.
//
// As in the other kernels, one wave walks one reordered filter's compressed
// storage (filter kernel reorder, compressed weight storage): pattern segment
// by pattern segment, each through a loop compiled for its centre+3 shape,
// with channel index and weights wave-uniform in SGPRs (scalar buffer loads).
// The next kernel's row loads while the current kernel's FMAs run.  Small
// grids split each filter over KS waves whose partial sums are added through
// LDS in share order (deterministic).
#pragma once

#include "conv_stream.h"

namespace psc {
namespace rw {

constexpr int kMaxShares = 8;

struct RGeo {
    int n, cin, H, W, cout, m;
    int ST, OH, OW; // stride, output rows and columns
    int S;          // images per wave
    int seg_len;    // lanes per image: OH rows + 1 zero lane
    int groups;     // image groups: ceil(n / S)
    int FW, KS;     // filters and shares per filter in a workgroup
    int groups_x;   // filter groups (fastest varying logical block index)
    int nblocks;
    int x_bytes;    // bytes of x (the buffer range), below 2^31
    int keep;
    int relu;
    int staged;     // fp32, stride 1 on 16 x 16, stride 2 on 8 x 8 and 16 x 16 planes: the planes go through LDS
    int8_t shape[kMaxPatterns];  // centre+3 shape index of each library pattern, -1 = other mask
    uint16_t mask[kMaxPatterns];
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Raw words of one lane's input row(s): stride 1, the row; stride 2, the even
// row then the odd row.  fp16 rows of odd width start at a 2-byte boundary:
// the lane loads the 16-byte window from the 4-byte boundary at or below the
// row start and shifts it by the 2 bytes if needed.
template <int DT, int W, int ST>
struct RowWords {
    static constexpr int ESZ = DT == DT_F32 ? 4 : 2;
    static constexpr bool ODD = DT == DT_F16 && (W & 1);
    static constexpr int BYTES = ODD ? 16 : W * ESZ;   // per row
    static constexpr int NW = BYTES / 4;               // words per row
    static_assert(BYTES % 4 == 0, "rows are loaded in whole dwords");
    static_assert(!ODD || W <= 7, "the shifted window holds 7 halves");
    static_assert(ST == 1 || (!ODD && W % 2 == 0), "stride-2 rows have an even width");
    uint32_t d[ST * NW];
    uint32_t sh;   // ODD: 0 or 16, the bit shift of the row start in the window
};

// Whole-row loads of BYTES bytes at byte offset vo + soff into d[0..BYTES/4).
template <int BYTES>
__device__ __forceinline__ void load_row_words(__amdgpu_buffer_rsrc_t xr, uint32_t vo, int soff, uint32_t* d) {
#pragma unroll
    for (int o = 0; o < BYTES; o += 16) {
        const int left = BYTES - o;
        if (left >= 16) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(xr, int(vo + o), soff, 0);
            d[o / 4] = v.x, d[o / 4 + 1] = v.y, d[o / 4 + 2] = v.z, d[o / 4 + 3] = v.w;
        } else if (left == 12) {
            const u32x3 v = __builtin_amdgcn_raw_buffer_load_b96(xr, int(vo + o), soff, 0);
            d[o / 4] = v.x, d[o / 4 + 1] = v.y, d[o / 4 + 2] = v.z;
        } else if (left == 8) {
            const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(xr, int(vo + o), soff, 0);
            d[o / 4] = v.x, d[o / 4 + 1] = v.y;
        } else {
            d[o / 4] = __builtin_amdgcn_raw_buffer_load_b32(xr, int(vo + o), soff, 0);
        }
    }
}

// Load the words at byte offset vo + soff (and, stride 2, the odd row at
// vo2 + soff).  A buffer load returns zero for any offset past the range of
// x: padding lanes and rows pass 2^31.
template <int DT, int W, int ST>
__device__ __forceinline__ void load_words(__amdgpu_buffer_rsrc_t xr, uint32_t vo, uint32_t vo2, int soff,
                                           int x_bytes, bool valid, RowWords<DT, W, ST>& rw) {
    using RWd = RowWords<DT, W, ST>;
    if constexpr (RWd::ODD) {
        const uint32_t t = vo + uint32_t(soff);
        const uint32_t at = t & ~3u;
        rw.sh = (t & 2u) << 3;
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(xr, int(at), 0, 0);
        rw.d[0] = v.x, rw.d[1] = v.y, rw.d[2] = v.z, rw.d[3] = v.w;
        // the window of a row that starts on a 4-byte boundary reaches 2
        // bytes past the row; for the last row of x those lie past the range,
        // so its 7th half is loaded on its own
        if (valid && int64_t(at) + 16 > int64_t(x_bytes)) {
            const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(xr, int(at + 12), 0, 0);
            rw.d[3] = (rw.d[3] & 0xffff0000u) | h;
        }
    } else {
        load_row_words<RWd::BYTES>(xr, vo, soff, rw.d);
        if constexpr (ST == 2) load_row_words<RWd::BYTES>(xr, vo2, soff, rw.d + RWd::NW);
    }
}

// The input values as fp32 (fp16 widened exactly): e, the row (stride 2:
// the even row); o, stride 2 only, the odd row.
template <int W, int ST>
struct RowVals {
    float e[W];
    float o[ST == 2 ? W : 1];
};

template <int DT, int W>
__device__ __forceinline__ void unpack_words(const uint32_t* d, uint32_t sh, float (&x)[W]) {
    constexpr int NW = RowWords<DT, W, 1>::NW;
    if constexpr (DT == DT_F32) {
#pragma unroll
        for (int j = 0; j < W; ++j) x[j] = __builtin_bit_cast(float, d[j]);
    } else {
        uint32_t s[NW];
        if constexpr (RowWords<DT, W, 1>::ODD) {
#pragma unroll
            for (int i = 0; i + 1 < NW; ++i) s[i] = __builtin_amdgcn_alignbit(d[i + 1], d[i], sh);
            s[NW - 1] = d[NW - 1] >> sh;
        } else {
#pragma unroll
            for (int i = 0; i < NW; ++i) s[i] = d[i];
        }
#pragma unroll
        for (int j = 0; j < W; ++j)
            x[j] = float(__builtin_bit_cast(_Float16, uint16_t(s[j / 2] >> (16 * (j & 1)))));
    }
}

// After the values are final: an asm the compiler sees as writing the DPP
// source row (so no VALU write of it can follow), then the two wait states a
// DPP read needs after a VALU write of its source.
template <int W>
__device__ __forceinline__ void settle_row(float (&x)[W]) {
#pragma unroll
    for (int j = 0; j < W; j += 4) {
        if (j + 3 < W) asm volatile("" : "+v"(x[j]), "+v"(x[j + 1]), "+v"(x[j + 2]), "+v"(x[j + 3]));
        else
            for (int t = j; t < W; ++t) asm volatile("" : "+v"(x[t]));
    }
    asm volatile("s_nop 1");
}

template <int DT, int W, int ST>
__device__ __forceinline__ void unpack_vals(const RowWords<DT, W, ST>& rw, RowVals<W, ST>& v) {
    unpack_words<DT, W>(rw.d, rw.sh, v.e);
    if constexpr (ST == 2) {
        unpack_words<DT, W>(rw.d + RowWords<DT, W, ST>::NW, 0u, v.o);
        settle_row<W>(v.o);
    } else {
        settle_row<W>(v.e);
    }
}

// The tap at kernel position Q = 3 ky + kx, stride 1: acc[c] += w * x(row
// r + ky - 1, column c + kx - 1).  Row r - 1 is the lane to the left
// (wave_shr), row r + 1 the lane to the right (wave_shl); lanes without a
// neighbour read zero (bound_ctrl).  Columns outside the row are skipped.
// Stride 2: acc[c] += w * x(row 2i + ky - 1, column 2c + kx - 1) with row
// 2i - 1 the odd row of the lane to the left, 2i the even and 2i + 1 the odd
// row of the lane.
#define PSC_DPP_SHR "v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_DPP_SHL "v_fmac_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
template <int Q, int W, int ST>
__device__ __forceinline__ void tap_row(float (&acc)[W / ST], const RowVals<W, ST>& x, float w) {
    constexpr int ky = Q / 3, kx = Q % 3;
    if constexpr (ST == 1) {
        constexpr int c0 = kx == 0 ? 1 : 0, c1 = kx == 2 ? W - 1 : W;
#pragma unroll
        for (int c = c0; c < c1; ++c) {
            if constexpr (ky == 1)
                acc[c] = __builtin_fmaf(w, x.e[c + kx - 1], acc[c]);
            else if constexpr (ky == 0)
                asm volatile(PSC_DPP_SHR : "+v"(acc[c]) : "v"(x.e[c + kx - 1]), "v"(w));
            else
                asm volatile(PSC_DPP_SHL : "+v"(acc[c]) : "v"(x.e[c + kx - 1]), "v"(w));
        }
    } else {
        constexpr int c0 = kx == 0 ? 1 : 0;
#pragma unroll
        for (int c = c0; c < W / 2; ++c) {
            if constexpr (ky == 0)
                asm volatile(PSC_DPP_SHR : "+v"(acc[c]) : "v"(x.o[2 * c + kx - 1]), "v"(w));
            else if constexpr (ky == 1)
                acc[c] = __builtin_fmaf(w, x.e[2 * c + kx - 1], acc[c]);
            else
                acc[c] = __builtin_fmaf(w, x.o[2 * c + kx - 1], acc[c]);
        }
    }
}
#undef PSC_DPP_SHL
#undef PSC_DPP_SHR

template <int W, int ST>
__device__ __forceinline__ void tap_row_dyn(int q, float (&acc)[W / ST], const RowVals<W, ST>& x, float w) {
    switch (q) {
        case 0: tap_row<0, W, ST>(acc, x, w); break;
        case 1: tap_row<1, W, ST>(acc, x, w); break;
        case 2: tap_row<2, W, ST>(acc, x, w); break;
        case 3: tap_row<3, W, ST>(acc, x, w); break;
        case 4: tap_row<4, W, ST>(acc, x, w); break;
        case 5: tap_row<5, W, ST>(acc, x, w); break;
        case 6: tap_row<6, W, ST>(acc, x, w); break;
        case 7: tap_row<7, W, ST>(acc, x, w); break;
        default: tap_row<8, W, ST>(acc, x, w); break;
    }
}

struct RowCtx {
    cs::Meta m;
    __amdgpu_buffer_rsrc_t xr;   // x, bounded to its size
    int chan_bytes;              // bytes of one input channel plane
    int x_bytes;
    uint32_t vo;                 // byte offset of this lane's (even) row in channel 0 (2^31: padding)
    uint32_t vo2;                // stride 2: the odd row (2^31: padding)
    bool valid;
};

template <int DT, int W, int ST>
__device__ __forceinline__ void row_of(const RowCtx& c, int ci, RowWords<DT, W, ST>& rw) {
    // wave-uniform: an SGPR operand.  A malformed channel index reads zeros
    // or other data of x, never memory outside it (range-checked loads).
    const int soff = __builtin_amdgcn_readfirstlane(ci * c.chan_bytes);
    load_words<DT, W, ST>(c.xr, c.vo, c.vo2, soff, c.x_bytes, c.valid, rw);
}

// Kernels [k, e) of one pattern segment share (e > k), two per trip: the row
// of one loads while the other's FMAs run; metadata is read two kernels
// ahead; the single loop exit keeps the accumulators in place.
template <int DT, int W, int ST, class TapFn>
__device__ __forceinline__ void run_rows(const RowCtx& c, int k, int e, float (&acc)[W / ST], TapFn taps) {
    const int last = e - 1;
    float wA[4], wB[4];
    cs::meta_w<DT>(c.m, k, wA);
    int kk = k + 1 <= last ? k + 1 : last;
    int ciB = cs::meta_ci(c.m, kk);
    cs::meta_w<DT>(c.m, kk, wB);
    RowWords<DT, W, ST> rA, rB;
    row_of<DT, W, ST>(c, cs::meta_ci(c.m, k), rA);
    while (k + 1 < e) {
        row_of<DT, W, ST>(c, ciB, rB);                           // row of kernel k+1
        kk = k + 2 <= last ? k + 2 : last;
        const int ciA2 = cs::meta_ci(c.m, kk);
        float wA2[4];
        cs::meta_w<DT>(c.m, kk, wA2);
        kk = k + 3 <= last ? k + 3 : last;
        const int ciB2 = cs::meta_ci(c.m, kk);
        float wB2[4];
        cs::meta_w<DT>(c.m, kk, wB2);
        {
            RowVals<W, ST> x;
            unpack_vals<DT, W, ST>(rA, x);
            taps(acc, x, wA);                                    // kernel k
        }
        row_of<DT, W, ST>(c, ciA2, rA);                          // row of kernel k+2
        {
            RowVals<W, ST> x;
            unpack_vals<DT, W, ST>(rB, x);
            taps(acc, x, wB);                                    // kernel k+1
        }
        k += 2;
        wA[0] = wA2[0], wA[1] = wA2[1], wA[2] = wA2[2], wA[3] = wA2[3];
        wB[0] = wB2[0], wB[1] = wB2[1], wB[2] = wB2[2], wB[3] = wB2[3];
        ciB = ciB2;
    }
    if (k < e) {
        RowVals<W, ST> x;
        unpack_vals<DT, W, ST>(rA, x);
        taps(acc, x, wA);
    }
}

// The four taps of a fixed centre+3 mask.  The taps that read the DPP source
// row through DPP go last: the others put FMAs between the settle and the DPP
// reads.
template <int W, int ST, int MASK>
struct ShapeTaps {
    __device__ __forceinline__ void operator()(float (&a)[W / ST], const RowVals<W, ST>& x,
                                               const float (&w)[4]) const {
        constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
        constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
        constexpr int DR = 0;   // ky of the taps read by DPP (the row above)
        if constexpr (Q0 / 3 != DR && (ST == 2 || Q0 / 3 == 1)) tap_row<Q0, W, ST>(a, x, w[0]);
        if constexpr (Q1 / 3 != DR && (ST == 2 || Q1 / 3 == 1)) tap_row<Q1, W, ST>(a, x, w[1]);
        if constexpr (Q2 / 3 != DR && (ST == 2 || Q2 / 3 == 1)) tap_row<Q2, W, ST>(a, x, w[2]);
        if constexpr (Q3 / 3 != DR && (ST == 2 || Q3 / 3 == 1)) tap_row<Q3, W, ST>(a, x, w[3]);
        if constexpr (!(Q0 / 3 != DR && (ST == 2 || Q0 / 3 == 1))) tap_row<Q0, W, ST>(a, x, w[0]);
        if constexpr (!(Q1 / 3 != DR && (ST == 2 || Q1 / 3 == 1))) tap_row<Q1, W, ST>(a, x, w[1]);
        if constexpr (!(Q2 / 3 != DR && (ST == 2 || Q2 / 3 == 1))) tap_row<Q2, W, ST>(a, x, w[2]);
        if constexpr (!(Q3 / 3 != DR && (ST == 2 || Q3 / 3 == 1))) tap_row<Q3, W, ST>(a, x, w[3]);
    }
};

// Any 4-of-9 mask: each tap is chosen per kernel by a uniform branch.
template <int W, int ST>
struct GenericTaps {
    int q0 = 4, q1 = 4, q2 = 4, q3 = 4;
    __device__ __forceinline__ explicit GenericTaps(unsigned mask) {
        int seen = 0;
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
    }
    __device__ __forceinline__ void operator()(float (&a)[W / ST], const RowVals<W, ST>& x,
                                               const float (&w)[4]) const {
        tap_row_dyn<W, ST>(q0, a, x, w[0]);
        tap_row_dyn<W, ST>(q1, a, x, w[1]);
        tap_row_dyn<W, ST>(q2, a, x, w[2]);
        tap_row_dyn<W, ST>(q3, a, x, w[3]);
    }
};

template <int DT, int W, int ST, int MASK>
__device__ __forceinline__ void run_shape_rows(const RowCtx& c, int k, int e, float (&acc)[W / ST]) {
    run_rows<DT, W, ST>(c, k, e, acc, ShapeTaps<W, ST, MASK>{});
}

template <int DT, int W, int ST>
__device__ __forceinline__ void run_generic_rows(unsigned mask, const RowCtx& c, int k, int e,
                                                 float (&acc)[W / ST]) {
    run_rows<DT, W, ST>(c, k, e, acc, GenericTaps<W, ST>(mask));
}

#define PSC_ROWS_CASE(I) \
    case I: run_shape_rows<DT, W, ST, kCentre3.code[I]>(c, k, e, acc); return;
#define PSC_ROWS_CASE8(I)                                                                           \
    PSC_ROWS_CASE(I) PSC_ROWS_CASE(I + 1) PSC_ROWS_CASE(I + 2) PSC_ROWS_CASE(I + 3)                 \
    PSC_ROWS_CASE(I + 4) PSC_ROWS_CASE(I + 5) PSC_ROWS_CASE(I + 6) PSC_ROWS_CASE(I + 7)

template <int DT, int W, int ST>
__device__ __forceinline__ void run_pattern_rows(int shape, unsigned mask, const RowCtx& c, int k, int e,
                                                 float (&acc)[W / ST]) {
    switch (shape) {
        PSC_ROWS_CASE8(0)
        PSC_ROWS_CASE8(8)
        PSC_ROWS_CASE8(16)
        PSC_ROWS_CASE8(24)
        PSC_ROWS_CASE8(32)
        PSC_ROWS_CASE8(40)
        PSC_ROWS_CASE8(48)
        default: run_generic_rows<DT, W, ST>(mask, c, k, e, acc); return;
    }
}
#undef PSC_ROWS_CASE8
#undef PSC_ROWS_CASE

// ------------------------------------------------------------ LDS-staged rows
// Three fp32 geometries in which each lane needs whole rows of its image
// that lie 64 or 128 bytes apart from its neighbours': stride 1 on 16 x 16
// planes (3 images a wave, row r, 64 bytes), stride 2 on 8 x 8 (12 images,
// input rows 2r and 2r+1, 64 bytes) and on 16 x 16 (7 images, 128 bytes).
// Loaded directly, each 16-byte load of the wave touches 24 or more
// 128-byte lines per KiB.  Staged, the wave copies the channel planes of a
// kernel (3 or 7 KiB, whole planes) into its own LDS area with 1 KiB
// buffer-to-LDS loads of 8 lines each, and every lane then reads its rows
// with 16-byte LDS reads.  The copy of the next kernel overlaps the current
// kernel's FMAs.  With two copies it starts before this kernel's reads;
// with one (7 KiB planes, to keep 20+ waves per CU) right after them.  No
// other wave touches the area, so no barrier is needed.
//
// A plane is NCH chunks of 16 bytes; lane r of an image needs the LC chunks
// LC r .. LC r + LC-1 and reads chunk LC r + j in its j-th read.  Image s
// keeps that chunk at position LC r + ((j + s + r / (16 / LC)) mod LC) of
// its block, which spreads one read of neighbouring rows and images over the
// LDS banks (without it the 16 x 16 stride-2 form took 1.8x as long).
template <int W, int ST>
struct Stage {
    static constexpr int H = W;                     // square planes only
    static constexpr int OH = H / ST;
    static constexpr int S = 64 / (OH + 1);         // images per wave
    static constexpr int PLANE = H * W * 4;         // bytes of one fp32 channel plane
    static constexpr int NCH = PLANE / 16;          // chunks per plane
    static constexpr int LC = ST * W / 4;           // chunks a lane reads
    static constexpr int RD = 16 / LC;              // rows per step of the rotation
    static constexpr int ZERO = S * PLANE;          // offset of the bytes padding lanes read (zero)
    static constexpr int COPY = ZERO + 16 * LC;     // bytes between the copies
    static constexpr int NB = LC == 4 ? 2 : 1;      // copies
    static constexpr int WAVE = NB * COPY;          // LDS bytes per wave
    static constexpr int ND = S * NCH / 64;         // buffer-to-LDS loads per kernel
    static_assert((LC == 4 || LC == 8) && S * NCH == 64 * ND, "whole planes in whole 1 KiB loads");
};

constexpr bool staged_geometry(int dtype, int w, int h, int stride) {
    return dtype == DT_F32 && h == w && ((stride == 2 && (w == 8 || w == 16)) || (stride == 1 && w == 16));
}

template <int W, int ST>
struct RowLds {
    cs::Meta m;
    __amdgpu_buffer_rsrc_t xr;         // x, bounded to its size
    uint32_t vo[Stage<W, ST>::ND];     // load j: byte offset in x (channel 0) of the chunk this lane moves, 2^31 past the batch
    uint32_t area;                     // LDS address of this wave's area (wave-uniform)
};

// Copy the planes of channel ci into copy B (0 when there is one copy).  A buffer-to-LDS load writes
// lane L's 16 bytes at its LDS base + 16 L; load j covers positions 64 j ..
// 64 j + 63 of the wave's chunks.  Images past the batch read zero (offset
// 2^31, past the buffer range).
template <int W, int ST, int B>
__device__ __forceinline__ void dma_stage(const RowLds<W, ST>& c, int ci) {
#if defined(__HIP_DEVICE_COMPILE__)   // the 16-byte form exists only for the gfx950 device pass
    using G = Stage<W, ST>;
    const int soff = __builtin_amdgcn_readfirstlane(ci * G::PLANE);
#pragma unroll
    for (int j = 0; j < G::ND; ++j) {
        cs::lds_void_t* dst = (cs::lds_void_t*)(uintptr_t)(c.area + uint32_t(B * G::COPY + j * 1024));
        __builtin_amdgcn_raw_ptr_buffer_load_lds(c.xr, dst, 16, c.vo[j], soff, 0, 0);
    }
#endif
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// One kernel whose planes sit (or are arriving) in copy B: wait for them,
// start the copy of kernel k+1 (channel ci; also across the pattern segment's
// end) into the other copy, read this lane's rows and run the FMAs with the
// weights w of kernel k; then refill w and ci with the weights of kernel k+2
// and the channel of kernel k+3, for the next trip of the same copy.
template <int W, int ST, int B, class TapFn>
__device__ __forceinline__ void stage_trip(const RowLds<W, ST>& c, const uint32_t (&lo)[Stage<W, ST>::LC], int k,
                                           int s1, float (&w)[4], int& ci, float (&acc)[W / ST], TapFn taps) {
    using G = Stage<W, ST>;
    constexpr int LC = G::LC;
    constexpr int BR = G::NB == 2 ? B : 0;               // the copy this kernel's planes sit in
    const int last = s1 - 1;
    __builtin_amdgcn_s_waitcnt(cs::kWaitVm0);            // planes of kernel k are in LDS
    asm volatile("" ::: "memory");
    if constexpr (G::NB == 2)
        if (k + 1 < s1) dma_stage<W, ST, BR ^ 1>(c, ci); // planes of kernel k+1
    f32x4 v[LC];
#pragma unroll
    for (int j = 0; j < LC; ++j)
        v[j] = *(const __attribute__((address_space(3))) f32x4*)(uintptr_t)(lo[j] + BR * G::COPY);
    __builtin_amdgcn_s_waitcnt(cs::kWaitLgkm0);          // rows in registers
    asm volatile("" ::: "memory");
    // one copy: it is free again once the rows are in registers
    if constexpr (G::NB == 1)
        if (k + 1 < s1) dma_stage<W, ST, 0>(c, ci);      // planes of kernel k+1
    // chunks 0 .. LC/ST - 1 hold the (even) row, stride 2: then the odd row
    RowVals<W, ST> x;
#pragma unroll
    for (int j = 0; j < LC; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (ST == 1 || j < LC / 2) x.e[4 * j + t] = v[j][t];
            else x.o[4 * (j - LC / 2) + t] = v[j][t];
        }
    if constexpr (ST == 2) settle_row<W>(x.o);
    else settle_row<W>(x.e);
    taps(acc, x, w);
    // the FMAs stay ahead of the next trip's wait: moved past it, they would
    // wait for the copy just started
#pragma unroll
    for (int t = 0; t < W / ST; ++t) asm volatile("" : "+v"(acc[t]));
    cs::meta_w<DT_F32>(c.m, k + 2 <= last ? k + 2 : last, w);
    ci = cs::meta_ci(c.m, k + 3 <= last ? k + 3 : last);
}

// Kernels [k, e) of one pattern segment of the share that ends at s1, the
// first one's planes in copy B0; returns the copy that kernel e's planes go
// to.  Each copy has its own weight and channel registers, refilled two
// kernels ahead.
template <int W, int ST, int B0, class TapFn>
__device__ __forceinline__ int stage_pairs(const RowLds<W, ST>& c, const uint32_t (&lo)[Stage<W, ST>::LC], int k,
                                           int e, int s1, float (&acc)[W / ST], TapFn taps) {
    const int last = s1 - 1;
    float wA[4], wB[4];
    cs::meta_w<DT_F32>(c.m, k, wA);
    cs::meta_w<DT_F32>(c.m, k + 1 <= last ? k + 1 : last, wB);
    int ciA = cs::meta_ci(c.m, k + 1 <= last ? k + 1 : last);
    int ciB = cs::meta_ci(c.m, k + 2 <= last ? k + 2 : last);
    while (k + 1 < e) {
        stage_trip<W, ST, B0>(c, lo, k, s1, wA, ciA, acc, taps);
        stage_trip<W, ST, B0 ^ 1>(c, lo, k + 1, s1, wB, ciB, acc, taps);
        k += 2;
    }
    if (k < e) {
        stage_trip<W, ST, B0>(c, lo, k, s1, wA, ciA, acc, taps);
        return B0 ^ 1;
    }
    return B0;
}

template <int W, int ST, class TapFn>
__device__ __forceinline__ int stage_kernels(const RowLds<W, ST>& c, const uint32_t (&lo)[Stage<W, ST>::LC], int k,
                                             int e, int s1, int par, float (&acc)[W / ST], TapFn taps) {
    return par == 0 ? stage_pairs<W, ST, 0>(c, lo, k, e, s1, acc, taps)
                    : stage_pairs<W, ST, 1>(c, lo, k, e, s1, acc, taps);
}

#define PSC_STG_CASE(I) \
    case I: return stage_kernels<W, ST>(c, lo, k, e, s1, par, acc, ShapeTaps<W, ST, kCentre3.code[I]>{});
#define PSC_STG_CASE8(I)                                                                            \
    PSC_STG_CASE(I) PSC_STG_CASE(I + 1) PSC_STG_CASE(I + 2) PSC_STG_CASE(I + 3)                     \
    PSC_STG_CASE(I + 4) PSC_STG_CASE(I + 5) PSC_STG_CASE(I + 6) PSC_STG_CASE(I + 7)

template <int W, int ST>
__device__ __forceinline__ int stage_pattern(int shape, unsigned mask, const RowLds<W, ST>& c,
                                             const uint32_t (&lo)[Stage<W, ST>::LC], int k, int e, int s1, int par,
                                             float (&acc)[W / ST]) {
    switch (shape) {
        PSC_STG_CASE8(0)
        PSC_STG_CASE8(8)
        PSC_STG_CASE8(16)
        PSC_STG_CASE8(24)
        PSC_STG_CASE8(32)
        PSC_STG_CASE8(40)
        PSC_STG_CASE8(48)
        default: return stage_kernels<W, ST>(c, lo, k, e, s1, par, acc, GenericTaps<W, ST>(mask));
    }
}
#undef PSC_STG_CASE8
#undef PSC_STG_CASE

// STG: the LDS-staged form (fp32: stride 1 on 16 x 16 planes, stride 2 on 8 x 8 and 16 x 16).
template <int DT, int W, int ST, bool STG>
__global__ __launch_bounds__(512) void k_conv_rows(const typename Elt<DT>::T* __restrict__ x,
                                                   const int32_t* __restrict__ perm,
                                                   const int32_t* __restrict__ seg_ptr,
                                                   const int32_t* __restrict__ cin_idx,
                                                   const typename Elt<DT>::T* __restrict__ vals,
                                                   const typename Elt<DT>::T* __restrict__ bias,
                                                   typename Elt<DT>::T* __restrict__ y, RGeo g) {
    using E = Elt<DT>;
    constexpr int ESZ = int(sizeof(typename E::T));
    constexpr int OW = W / ST;                // output columns (stride 2: W even)
    // KS > 1: [KS][OW][64] partial sums; STG: first the waves' staging areas
    extern __shared__ float psc_rows_red[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int gf = wave / g.KS, sp = wave - gf * g.KS;   // filter slot, share

    // XCD-aware block order: the hardware deals consecutive blocks out to the
    // 8 XCDs in turn; remap so that one XCD runs consecutive logical blocks,
    // which share an image group (its rows stay in that XCD's L2) and differ
    // in their filter group.
    const int b = blockIdx.x;
    int lb = b;
    if (g.nblocks >= 8) {
        const int per = g.nblocks / 8, rem = g.nblocks % 8;
        const int xcd = b % 8, slot = b / 8;
        lb = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot;
    }
    const int fg = lb % g.groups_x, grp = lb / g.groups_x;
    const int i = fg * g.FW + gf;                        // reordered filter of this wave
    const bool has_filter = i < g.cout;

    // ---- lane geometry: image s of the group, output row r (r == OH: the zero lane)
    const int s = lane / g.seg_len, r = lane - s * g.seg_len;
    const int img = grp * g.S + s;
    const bool valid = s < g.S && img < g.n && r < g.OH;
    const int plane = g.H * g.W;

    float acc[OW];
#pragma unroll
    for (int c = 0; c < OW; ++c) acc[c] = 0.f;

    if constexpr (STG) {
        using G = Stage<W, ST>;
        static_assert(staged_geometry(DT, W, W, ST), "no staged form for this geometry");
        constexpr int LC = G::LC;
        // this wave's area: per copy the planes, then 16 LC zero bytes that
        // padding lanes read
        const uint32_t area = uint32_t(uintptr_t((const __attribute__((address_space(3))) void*)psc_rows_red)) +
                              uint32_t(wave * G::WAVE);
#pragma unroll
        for (int b = 0; b < G::NB; ++b)
            if (lane < 4 * LC)
                *(__attribute__((address_space(3))) float*)(uintptr_t)(area + b * G::COPY + G::ZERO + lane * 4) = 0.f;
        // LDS address (copy 0) of the chunk this lane reads in each of its LC reads
        uint32_t lo[LC];
#pragma unroll
        for (int j = 0; j < LC; ++j)
            lo[j] = s < G::S && r < G::OH
                        ? area + uint32_t(s * G::PLANE + 16 * (LC * r + ((j + s + r / G::RD) & (LC - 1))))
                        : area + uint32_t(G::ZERO + 16 * j);
        if (has_filter) {
            const int* segp = seg_ptr + i * (g.m + 1);
            const int f0 = segp[0], f1 = segp[g.m];
            const int len = f1 - f0;
            const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
            RowLds<W, ST> ctx;
            ctx.m = cs::Meta{cs::scalar_rsrc(cin_idx, g.keep * 4), cs::scalar_rsrc(vals, g.keep * 4 * ESZ)};
            ctx.xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes,
                                                       0x00020000);
            ctx.area = __builtin_amdgcn_readfirstlane(area);
            // load j, lane L: position q of image slot t's block, holding
            // chunk LC rr + ((q - t - rr / RD) mod LC) of the plane (rr = q / LC)
#pragma unroll
            for (int j = 0; j < G::ND; ++j) {
                const int pos = 64 * j + lane, t = pos / G::NCH, q = pos - t * G::NCH, rr = q / LC;
                const int chunk = LC * rr + ((q - t - rr / G::RD) & (LC - 1));
                const int im = grp * G::S + t;
                ctx.vo[j] = im < g.n ? uint32_t(im * g.cin * G::PLANE + chunk * 16) : 0x80000000u;
            }
            if (s0 < s1) {
                dma_stage<W, ST, 0>(ctx, cs::meta_ci(ctx.m, s0));
                int par = 0;
                for (int p = 0; p < g.m; ++p) {
                    int k0 = segp[p], k1 = segp[p + 1];
                    k0 = k0 < s0 ? s0 : k0;
                    k1 = k1 > s1 ? s1 : k1;                 // malformed pointers stay in the share
                    if (k0 < k1) par = stage_pattern<W, ST>(g.shape[p], g.mask[p], ctx, lo, k0, k1, s1, par, acc);
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(cs::kWaitVm0);        // no copy into LDS is left in flight
    } else if (has_filter) {
        const int* segp = seg_ptr + i * (g.m + 1);
        const int f0 = segp[0], f1 = segp[g.m];
        // share sp: the sp-th of KS equal contiguous ranges of the filter's kernels
        const int len = f1 - f0;
        const int s0 = f0 + len * sp / g.KS, s1 = f0 + len * (sp + 1) / g.KS;
        RowCtx ctx;
        ctx.m = cs::Meta{cs::scalar_rsrc(cin_idx, g.keep * 4), cs::scalar_rsrc(vals, g.keep * 4 * ESZ)};
        ctx.xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes, 0x00020000);
        ctx.chan_bytes = __builtin_amdgcn_readfirstlane(plane * ESZ);
        ctx.x_bytes = g.x_bytes;
        // input row ST*r of channel 0 of the lane's image (stride 2: and row
        // 2r+1, zero past the last row)
        ctx.vo = valid ? uint32_t((img * g.cin * g.H + ST * r) * g.W) * uint32_t(ESZ) : 0x80000000u;
        ctx.vo2 = valid && ST == 2 && 2 * r + 1 < g.H ? ctx.vo + uint32_t(g.W * ESZ) : 0x80000000u;
        ctx.valid = valid;
        for (int p = 0; p < g.m; ++p) {
            int k0 = segp[p], k1 = segp[p + 1];
            k0 = k0 < s0 ? s0 : k0;
            k1 = k1 > s1 ? s1 : k1;                     // malformed pointers stay in the share
            if (k0 < k1) run_pattern_rows<DT, W, ST>(g.shape[p], g.mask[p], ctx, k0, k1, acc);
        }
    }

    // ---- add the KS partial sums of each filter in share order
    if (g.KS > 1) {
        float (*red)[OW][64] = reinterpret_cast<float (*)[OW][64]>(psc_rows_red);
        // the partial sums reuse the staging areas: wait until every wave is done
        if constexpr (STG) __syncthreads();
        for (int slot = 0; slot < g.FW; ++slot) {
            if (slot == gf) {
#pragma unroll
                for (int c = 0; c < OW; ++c) red[sp][c][lane] = acc[c];
            }
            __syncthreads();
            if (slot == gf) {
#pragma unroll
                for (int c = 0; c < OW; ++c) {
                    float v = 0.f;
                    for (int t = 0; t < g.KS; ++t) v += red[t][c][lane];
                    acc[c] = v;
                }
            }
            __syncthreads();
        }
    }
    if (!has_filter || !valid) return;
    const int f = perm[i];
    const float bv = bias ? E::load(bias, f) : 0.f;
    typename E::T* yp = y + (int64_t(img) * g.cout + f) * (g.OH * OW) + r * OW;
#pragma unroll
    for (int c = 0; c < OW; ++c) {
        // the KS waves of a filter hold the same sums; share t stores columns t, t+KS, ...
        if ((c % g.KS) == sp) {
            float v = acc[c] + bv;
            if (g.relu) v = v > 0.f ? v : 0.f;
            yp[c] = E::from_f(v);
        }
    }
}

template <int DT, int W, int ST>
hipError_t launch_rows(const PackedView& pk, const ConvArgs& a, const RGeo& g, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    const int waves = g.FW * g.KS;
    const size_t red = g.KS > 1 ? size_t(g.KS) * (W / ST) * 64 * sizeof(float) : 0;
    if constexpr (staged_geometry(DT, W, W, ST)) {
        if (g.staged) {
            const size_t stage = size_t(waves) * Stage<W, ST>::WAVE;
            hipLaunchKernelGGL((k_conv_rows<DT, W, ST, true>), dim3(unsigned(g.nblocks)), dim3(unsigned(waves * 64)),
                               stage > red ? stage : red, stream, static_cast<const T*>(a.x), pk.filter_perm,
                               pk.seg_ptr, pk.cin_idx, static_cast<const T*>(pk.values),
                               static_cast<const T*>(a.bias), static_cast<T*>(a.y), g);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((k_conv_rows<DT, W, ST, false>), dim3(unsigned(g.nblocks)), dim3(unsigned(waves * 64)), red,
                       stream, static_cast<const T*>(a.x), pk.filter_perm, pk.seg_ptr, pk.cin_idx,
                       static_cast<const T*>(pk.values), static_cast<const T*>(a.bias), static_cast<T*>(a.y), g);
    return hipGetLastError();
}

}  // namespace rw
}  // namespace psc
