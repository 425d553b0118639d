// Tuned pattern-sparse 3x3 convolution forward (Sec. 4.1 Eq. 1), built on
// the three compiler optimisations of Sec. 3.4 redesigned for CDNA4:
//
//  * filter kernel reorder -> one wave per reordered filter: the filter's
//    kernel list, channel indices, pattern ids and weights are wave-uniform
//    and read with scalar loads; consecutive (similar-length) filters share a
//    workgroup so its waves finish together;
//  * compressed weight storage -> kernels of one pattern are contiguous, so
//    the pattern decides the code path once per run of kernels (a switch over
//    the 56 centre+3 shapes, each a fully unrolled tap sequence), never per
//    weight;
//  * load redundancy elimination -> an input tile (channel chunk x (R+2) rows
//    x 64 columns) is staged once in LDS and reused by every filter of the
//    workgroup; inside a wave each lane owns one output column and R output
//    rows, loads each needed input row of a channel once into a register and
//    obtains the left/right neighbour columns from adjacent lanes (DPP), so
//    one LDS read feeds up to 4 FMAs per row.
//
// Lane layout: a wave's 64 lanes hold S independent segments.  If the image
// row fits (W <= 63), a segment is one full row band [W columns] and the
// segments are separated by a single lane that holds zero -- the zero padding
// on both sides.  Otherwise a segment is [halo][Wt columns][halo], the halo
// lanes holding the real neighbouring columns (or zero at the image border).
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

struct Geo {
    int n, cin, H, W, cout, m;
    int S;          // segments per wave
    int seg_len;    // lanes per segment
    int Wt;         // output columns per segment
    int cols_mode;  // 0: full-row segments with zero separators, 1: haloed column tiles
    int RB, CT;     // row blocks and column tiles per image
    int U;          // work units = n * RB * CT
    int C;          // input channels per LDS chunk
    int relu;
    int8_t shape[kMaxPatterns];  // centre+3 shape index of each library pattern, -1 = generic
    uint16_t mask[kMaxPatterns];
};

// Lane shifts across the whole wave: dst[l] = src[l-1] (right) or src[l+1]
// (left); lanes without a source read 0.
__device__ __forceinline__ float from_left(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x138,
                                                                 0xf, 0xf, true));
}
__device__ __forceinline__ float from_right(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x130,
                                                                 0xf, 0xf, true));
}

// One tap at kernel position (DR, DS) for R output rows.
template <int DR, int DS, int R>
__device__ __forceinline__ void tap(float (&acc)[R], const float (&xr)[R + 2], float wv) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        float xv = xr[r + DR];
        if constexpr (DS == 0) xv = from_left(xv);
        if constexpr (DS == 2) xv = from_right(xv);
        acc[r] = fmaf(wv, xv, acc[r]);
    }
}

template <int Q, int R>
__device__ __forceinline__ void tap_q(float (&acc)[R], const float (&xr)[R + 2], float wv) {
    tap<Q / 3, Q % 3, R>(acc, xr, wv);
}

// Position of the J-th set bit of MASK (ascending).
template <int MASK, int J>
struct NthBit {
    static constexpr int value() {
        int seen = 0;
        for (int q = 0; q < 9; ++q)
            if ((MASK >> q) & 1) {
                if (seen == J) return q;
                ++seen;
            }
        return -1;
    }
};

template <int DT>
__device__ __forceinline__ void load_w4(const typename Elt<DT>::T* __restrict__ vals, int k, float (&wv)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) wv[j] = Elt<DT>::load(vals, int64_t(k) * 4 + j);
}

// Runs kernels k.. of one pattern (shape MASK) while their channel lies in
// the staged chunk; returns the first kernel not processed.
template <int DT, int R, int MASK>
__device__ __forceinline__ int run_shape(int k, int e, int c_end, int c0,
                                         const int32_t* __restrict__ cin_idx,
                                         const typename Elt<DT>::T* __restrict__ vals,
                                         const float* __restrict__ xs_lane, float (&acc)[R]) {
    constexpr int Q0 = NthBit<MASK, 0>::value(), Q1 = NthBit<MASK, 1>::value();
    constexpr int Q2 = NthBit<MASK, 2>::value(), Q3 = NthBit<MASK, 3>::value();
    for (; k < e; ++k) {
        const int ci = __builtin_amdgcn_readfirstlane(cin_idx[k]);
        if (unsigned(ci - c0) >= unsigned(c_end - c0)) break;   // also stops on malformed ci < c0
        float wv[4];
        load_w4<DT>(vals, k, wv);
        const float* b = xs_lane + (ci - c0) * (R + 2) * 64;
        float xr[R + 2];
#pragma unroll
        for (int r = 0; r < R + 2; ++r) xr[r] = b[r * 64];
        tap_q<Q0, R>(acc, xr, wv[0]);
        tap_q<Q1, R>(acc, xr, wv[1]);
        tap_q<Q2, R>(acc, xr, wv[2]);
        tap_q<Q3, R>(acc, xr, wv[3]);
    }
    return k;
}

// Any 4-of-9 mask: the taps are decoded per kernel (a uniform branch per tap).
template <int R>
__device__ __forceinline__ void tap_dyn(int q, float (&acc)[R], const float (&xr)[R + 2], float wv) {
    switch (q) {
        case 0: tap_q<0, R>(acc, xr, wv); break;
        case 1: tap_q<1, R>(acc, xr, wv); break;
        case 2: tap_q<2, R>(acc, xr, wv); break;
        case 3: tap_q<3, R>(acc, xr, wv); break;
        case 4: tap_q<4, R>(acc, xr, wv); break;
        case 5: tap_q<5, R>(acc, xr, wv); break;
        case 6: tap_q<6, R>(acc, xr, wv); break;
        case 7: tap_q<7, R>(acc, xr, wv); break;
        default: tap_q<8, R>(acc, xr, wv); break;
    }
}

template <int DT, int R>
__device__ __forceinline__ int run_generic(unsigned mask, int k, int e, int c_end, int c0,
                                        const int32_t* __restrict__ cin_idx,
                                        const typename Elt<DT>::T* __restrict__ vals,
                                        const float* __restrict__ xs_lane, float (&acc)[R]) {
    int qs[4];
    int j = 0;
    for (int q = 0; q < 9; ++q)
        if ((mask >> q) & 1u) qs[j++] = q;
    for (; k < e; ++k) {
        const int ci = __builtin_amdgcn_readfirstlane(cin_idx[k]);
        if (unsigned(ci - c0) >= unsigned(c_end - c0)) break;   // also stops on malformed ci < c0
        float wv[4];
        load_w4<DT>(vals, k, wv);
        const float* b = xs_lane + (ci - c0) * (R + 2) * 64;
        float xr[R + 2];
#pragma unroll
        for (int r = 0; r < R + 2; ++r) xr[r] = b[r * 64];
#pragma unroll
        for (int t = 0; t < 4; ++t) tap_dyn<R>(qs[t], acc, xr, wv[t]);
    }
    return k;
}

#define PSC_SHAPE_CASE(I) \
    case I: return run_shape<DT, R, kCentre3.code[I]>(k, e, c_end, c0, cin_idx, vals, xs_lane, acc);
#define PSC_SHAPE_CASE8(I)                                                                     \
    PSC_SHAPE_CASE(I) PSC_SHAPE_CASE(I + 1) PSC_SHAPE_CASE(I + 2) PSC_SHAPE_CASE(I + 3)        \
    PSC_SHAPE_CASE(I + 4) PSC_SHAPE_CASE(I + 5) PSC_SHAPE_CASE(I + 6) PSC_SHAPE_CASE(I + 7)

template <int DT, int R>
__device__ __forceinline__ int run_pattern(int shape, unsigned mask, int k, int e, int c_end, int c0,
                                           const int32_t* __restrict__ cin_idx,
                                           const typename Elt<DT>::T* __restrict__ vals,
                                           const float* __restrict__ xs_lane, float (&acc)[R]) {
    switch (shape) {
        PSC_SHAPE_CASE8(0)
        PSC_SHAPE_CASE8(8)
        PSC_SHAPE_CASE8(16)
        PSC_SHAPE_CASE8(24)
        PSC_SHAPE_CASE8(32)
        PSC_SHAPE_CASE8(40)
        PSC_SHAPE_CASE8(48)
        default: return run_generic<DT, R>(mask, k, e, c_end, c0, cin_idx, vals, xs_lane, acc);
    }
}
#undef PSC_SHAPE_CASE8
#undef PSC_SHAPE_CASE

template <int DT, int R, int FW>
__global__ __launch_bounds__(FW * 64) void k_conv_tiled(const typename Elt<DT>::T* __restrict__ x,
                                                        const int32_t* __restrict__ perm,
                                                        const int32_t* __restrict__ seg_ptr,
                                                        const int32_t* __restrict__ cin_idx,
                                                        const typename Elt<DT>::T* __restrict__ vals,
                                                        const typename Elt<DT>::T* __restrict__ bias,
                                                        typename Elt<DT>::T* __restrict__ y, Geo g) {
    using E = Elt<DT>;
    extern __shared__ float smem[];
    float* xs = smem;                                   // [C][R+2][64]
    int* cur = reinterpret_cast<int*>(smem + g.C * (R + 2) * 64);   // [FW][m]

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int i = blockIdx.y * FW + wave;               // reordered filter of this wave
    const bool has_filter = i < g.cout;

    // ---- lane geometry
    const int s = lane / g.seg_len, c = lane - s * g.seg_len;
    const int u = blockIdx.x * g.S + s;
    int ld_col = -1, out_col = -1, nimg = 0, h0 = 0;
    if (s < g.S && u < g.U) {
        nimg = u / (g.RB * g.CT);
        const int rb = (u / g.CT) % g.RB, ct = u % g.CT;
        h0 = rb * R;
        if (!g.cols_mode) {
            if (c < g.W) ld_col = out_col = c;
        } else {
            const int col = ct * g.Wt + c - 1;
            if (col >= 0 && col < g.W) ld_col = col;
            if (c >= 1 && c <= g.Wt && col < g.W) out_col = col;
        }
    }
    const int plane = g.H * g.W;
    const int x_lane = nimg * g.cin * plane + (ld_col < 0 ? 0 : ld_col);

    const int m = g.m;
    const int* segp = seg_ptr + (has_filter ? i : 0) * (m + 1);
    for (int p = lane; p < m; p += 64) cur[wave * m + p] = segp[p];

    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;

    const float* xs_lane = xs + lane;
    const int rows = R + 2;
    for (int c0 = 0; c0 < g.cin; c0 += g.C) {
        // ---- stage x[n][c0 .. c0+C)[h0-1 .. h0+R][lane columns] into LDS
        for (int e = wave; e < g.C * rows; e += FW) {
            const int cc = e / rows, r = e - cc * rows;
            const int row = h0 - 1 + r, ch = c0 + cc;
            float v = 0.f;
            if (ld_col >= 0 && row >= 0 && row < g.H && ch < g.cin)
                v = E::load(x, x_lane + ch * plane + row * g.W);
            xs[e * 64 + lane] = v;
        }
        __syncthreads();
        if (has_filter) {
            const int c_end = c0 + g.C;
            for (int p = 0; p < m; ++p) {
                int k = __builtin_amdgcn_readfirstlane(cur[wave * m + p]);
                const int e = segp[p + 1];
                if (k >= e) continue;
                if (__builtin_amdgcn_readfirstlane(cin_idx[k]) >= c_end) continue;
                k = run_pattern<DT, R>(g.shape[p], g.mask[p], k, e, c_end, c0, cin_idx, vals, xs_lane,
                                       acc);
                if (lane == 0) cur[wave * m + p] = k;
            }
        }
        __syncthreads();
    }
    if (!has_filter || out_col < 0) return;
    const int f = perm[i];
    const float b = bias ? E::load(bias, f) : 0.f;
    typename E::T* yp = y + (nimg * g.cout + f) * plane + out_col;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = h0 + r;
        if (row < g.H) {
            float v = acc[r] + b;
            if (g.relu) v = v > 0.f ? v : 0.f;
            yp[row * g.W] = E::from_f(v);
        }
    }
}

constexpr int kFW = 8;   // filters (waves) per workgroup

template <int DT, int R>
hipError_t launch_r(const PackedView& pk, const ConvArgs& a, Geo g, hipStream_t stream, size_t lds) {
    using T = typename Elt<DT>::T;
    auto kern = k_conv_tiled<DT, R, kFW>;
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (err != hipSuccess) return err;
    const dim3 grid(unsigned((g.U + g.S - 1) / g.S), unsigned((a.cout + kFW - 1) / kFW));
    hipLaunchKernelGGL(kern, grid, dim3(kFW * 64), lds, stream, static_cast<const T*>(a.x), pk.filter_perm,
                       pk.seg_ptr, pk.cin_idx, static_cast<const T*>(pk.values),
                       static_cast<const T*>(a.bias), static_cast<T*>(a.y), g);
    return hipGetLastError();
}

int pick_rows(int H) {
    // fewest wasted rows, larger R on ties
    const int cand[4] = {8, 7, 4, 2};
    int best = 8, waste = 1 << 30;
    for (int rr : cand) {
        const int wst = (H + rr - 1) / rr * rr - H;
        if (wst < waste) {
            waste = wst;
            best = rr;
        }
    }
    return best;
}

}  // namespace

hipError_t launch_conv_tiled(const PatTable& tab, const PackedView& pk, const ConvArgs& a,
                             hipStream_t stream) {
    Geo g;
    g.n = a.n;
    g.cin = a.cin;
    g.H = a.h;
    g.W = a.w;
    g.cout = a.cout;
    g.m = tab.m;
    g.relu = a.relu;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.shape[p] = -1;
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    const int R = pick_rows(a.h);
    g.RB = (a.h + R - 1) / R;
    // lane layout: full-row segments if they use the lanes at least as well
    // as haloed column tiles
    const int S_rows = a.w <= 63 ? 65 / (a.w + 1) : 0;
    const int use_rows = S_rows * a.w;
    // haloed column tiles: the tile count that keeps the most useful lanes
    int ct = (a.w + 61) / 62, use_cols = 0;
    for (int t = ct; t <= a.w && t <= 64; ++t) {
        const int wt = (a.w + t - 1) / t;
        const int use = (64 / (wt + 2)) * a.w / t;
        if (use > use_cols) {
            use_cols = use;
            ct = t;
        }
    }
    const int Wt = (a.w + ct - 1) / ct;
    const int S_cols = 64 / (Wt + 2);
    if (S_rows > 0 && use_rows >= use_cols) {
        g.cols_mode = 0;
        g.S = S_rows;
        g.seg_len = a.w + 1;
        g.Wt = a.w;
        g.CT = 1;
    } else {
        g.cols_mode = 1;
        g.S = S_cols;
        g.seg_len = Wt + 2;
        g.Wt = Wt;
        g.CT = ct;
    }
    g.U = a.n * g.RB * g.CT;
    // channel chunk: as much as fits in 64 KiB of LDS next to the cursors
    const size_t cur_bytes = size_t(kFW) * tab.m * 4;
    const size_t per_ch = size_t(R + 2) * 64 * 4;
    int C = int((65536 - cur_bytes) / per_ch);
    if (C > a.cin) C = a.cin;
    if (C < 1) C = 1;
    g.C = C;
    const size_t lds = size_t(C) * per_ch + cur_bytes;
    switch (R) {
        case 8: return a.dtype == DT_F16 ? launch_r<DT_F16, 8>(pk, a, g, stream, lds)
                                         : launch_r<DT_F32, 8>(pk, a, g, stream, lds);
        case 7: return a.dtype == DT_F16 ? launch_r<DT_F16, 7>(pk, a, g, stream, lds)
                                         : launch_r<DT_F32, 7>(pk, a, g, stream, lds);
        case 4: return a.dtype == DT_F16 ? launch_r<DT_F16, 4>(pk, a, g, stream, lds)
                                         : launch_r<DT_F32, 4>(pk, a, g, stream, lds);
        default: return a.dtype == DT_F16 ? launch_r<DT_F16, 2>(pk, a, g, stream, lds)
                                          : launch_r<DT_F32, 2>(pk, a, g, stream, lds);
    }
}

}  // namespace psc
