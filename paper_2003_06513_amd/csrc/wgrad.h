// Weight gradients of the 3x3 layer (stride 1, zero padding 1): for a kernel
// (f, ci) and each of its taps t at position (r_t, s_t),
//
//   dW_t = sum over images and output pixels (i, j) of
//          dy[n, f, i, j] * x[n, ci, i + r_t - 1, j + s_t - 1].
//
// Used for the masked gradient of the retraining function (Sec. 3.3: the 4
// stored values of each kept kernel, nothing for pruned weights) and for the
// dense gradient of the ADMM primal step (Sec. 4.3 Eq. 4: all 9 positions
// of every (f, ci)).
//
// Layout of the work.  The kernels of one filter all read the same dy plane,
// so a wave takes one filter and a chunk of up to KC of its kernels (KC
// consecutive kernels of one pattern segment in storage order; dense: KC
// consecutive input channels) and one share of the images: for every output
// band of the share it loads the R rows of dy once and, for each kernel of
// the chunk, the R+2 rows of x around them, so one dy load feeds KC kernels.
// The lane layout is the forward's: a lane owns one column and R rows of a
// band (a wave holds S bands of full rows separated by a zero lane, or a
// column tile with one halo lane on each side), or, for widths that are
// multiples of 4, 4 adjacent columns and R rows (each row one 16-byte fp32 /
// 8-byte fp16 load), or, for small planes at large batch, one image row.
// Rows come through buffer loads at offsets fixed per lane and row, the
// channel entering as a scalar offset and padding reading zero; the left and
// right neighbour columns of x are read by DPP inside the FMA.  The taps of a
// chunk are compiled for its centre+3 shape (other masks dispatch each tap).
// At the end of a chunk the KC x 4 per-lane sums are added across the wave
// by a reduce-scatter (each step halves the values a lane holds).  The
// chunks of a filter are dealt round-robin to G waves; when a wave has a
// single band group, its chunks run as a pipeline (the next chunk's rows
// load during the current one's FMAs and reduction).  With several image
// shares the share sums go to a workspace and a second kernel adds them in
// share order, so results do not depend on scheduling; the bias gradient is
// summed in parts that are added the same way.
#pragma once
#include "common.h"
#include "launch.h"
#include "conv_rows.h"

namespace psc {
namespace wg {

constexpr int kKC = 4;           // kernels per chunk

struct WGeo {
    int n, cin, cout, H, W;
    int S;          // bands (segments) per wave
    int seg_len;    // lanes per segment
    int Wt;         // output columns per segment
    int cols_mode;  // 0: full-row segments with zero separators, 1: haloed column tiles
    int rows;       // 1: one image row per lane (small planes at large batch; S images per wave)
    int wide;       // 1: 4 columns per lane (full-row segments padded to a multiple of 4 lanes)
    int pipe;       // 1: one slot per wave, chunks pipelined (masked gradients, one-column layout)
    int RB, CT;     // row bands and column tiles per image
    int units;      // n * RB * CT (rows: n)
    int slots;      // waves' worth of units: ceil(units / S)
    int G;          // waves sharing one filter's chunks (round-robin)
    int KS;         // image shares (ranges of slots)
    int64_t nk;     // kernels
    int dense;      // 1: kernel k is (k / cin, k % cin) with all 9 taps
    int m;
    int x_bytes, dy_bytes;   // buffer ranges
    uint16_t mask[kMaxPatterns];
    int8_t shape[kMaxPatterns];   // centre+3 shape index of each library pattern, -1 = other mask
};

#define PSC_W_SHR "v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_W_SHL "v_fmac_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
// acc += sum_r x(column c + kx - 1, row r + ky) * dy[r]: column c - 1 is the
// lane to the left (DPP wave_shr), c + 1 the lane to the right (wave_shl);
// lanes without a neighbour read zero.
template <int R, int Q>
__device__ __forceinline__ void wtap(float& acc, const float (&x)[R + 2], const float (&dyr)[R]) {
    constexpr int ky = Q / 3, kx = Q % 3;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if constexpr (kx == 1)
            acc = __builtin_fmaf(x[r + ky], dyr[r], acc);
        else if constexpr (kx == 0)
            asm volatile(PSC_W_SHR : "+v"(acc) : "v"(x[r + ky]), "v"(dyr[r]));
        else
            asm volatile(PSC_W_SHL : "+v"(acc) : "v"(x[r + ky]), "v"(dyr[r]));
    }
}
#undef PSC_W_SHL
#undef PSC_W_SHR

template <int R>
__device__ __forceinline__ void wtap_dyn(int q, float& acc, const float (&x)[R + 2], const float (&dyr)[R]) {
    switch (q) {
        case 0: wtap<R, 0>(acc, x, dyr); break;
        case 1: wtap<R, 1>(acc, x, dyr); break;
        case 2: wtap<R, 2>(acc, x, dyr); break;
        case 3: wtap<R, 3>(acc, x, dyr); break;
        case 4: wtap<R, 4>(acc, x, dyr); break;
        case 5: wtap<R, 5>(acc, x, dyr); break;
        case 6: wtap<R, 6>(acc, x, dyr); break;
        case 7: wtap<R, 7>(acc, x, dyr); break;
        default: wtap<R, 8>(acc, x, dyr); break;
    }
}

// R rows of one column through a buffer descriptor (offsets past its range
// read zero), widened to fp32.
template <int DT, int N>
__device__ __forceinline__ void load_col(__amdgpu_buffer_rsrc_t rs, const uint32_t (&vo)[N], int soff,
                                         float (&v)[N]) {
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if constexpr (DT == DT_F32)
            v[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, int(vo[r]), soff, 0));
        else
            v[r] = float(__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(rs, int(vo[r]), soff, 0)));
    }
}

// Values the compiler sees as written by an asm (no VALU write of them can
// follow), then the two wait states a DPP read needs after a VALU write of
// its source.
template <int N>
__device__ __forceinline__ void settle(float (&v)[N]) {
#pragma unroll
    for (int j = 0; j < N; j += 2) {
        if (j + 1 < N) asm volatile("" : "+v"(v[j]), "+v"(v[j + 1]));
        else asm volatile("" : "+v"(v[j]));
    }
    asm volatile("s_nop 1");
}

// Sum of each of the V values over the 64 lanes of the wave.  Reduce-scatter
// while more than one value is left: at each step the lanes whose bit d is
// set keep the upper half of their values and hand the lower half to their
// partner lane^d (which keeps the lower half), so every step halves the
// values a lane holds; the last value is then summed over the remaining
// lanes.  Returns the value index (0..V-1) lane holds at the end; every lane
// with the same index holds the same sum.
template <int V, int H, int D>
__device__ __forceinline__ void reduce_scatter_step(float (&a)[V], int lane, int& idx) {
    if constexpr (H >= 1) {
        const bool up = (lane & D) != 0;
#pragma unroll
        for (int j = 0; j < H; ++j) {
            const float send = up ? a[j] : a[j + H];
            const float keep = up ? a[j + H] : a[j];
            a[j] = keep + __shfl_xor(send, D);
        }
        if (up) idx += H;
        reduce_scatter_step<V, H / 2, D / 2>(a, lane, idx);
    } else {
#pragma unroll
        for (int d = D; d >= 1; d /= 2) a[0] += __shfl_xor(a[0], d);
    }
}

template <int V>
__device__ __forceinline__ int wave_reduce_scatter(float (&a)[V], int lane) {
    static_assert((V & (V - 1)) == 0 && V >= 2 && V <= 64, "V is a power of two from 2 to 64");
    int idx = 0;
    reduce_scatter_step<V, V / 2, 32>(a, lane, idx);
    return idx;
}

struct WCtx {
    __amdgpu_buffer_rsrc_t xs, dys;
    int chan_bytes;
};

// The chunk [k0, k0 + kc) of one filter: kernels of one pattern segment with
// taps Q (masked, NT = 4; QD: the positions come from q[] at run time), or the
// dense kernels (f, ci0 + j) with all 9 taps.  Sums over the bands of slots
// [sl0, sl1) go to out[(k0 + j) * NT + t], written by the lanes that hold
// them after the reduction.
template <int DT, int R, int NT, bool QD, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void run_chunk(const WGeo& g, const WCtx& c, const int32_t* __restrict__ cin_idx,
                                          int f, int k0, int kc, int ci0, const int (&q)[4], int sl0, int sl1,
                                          int lane, float* __restrict__ out) {
    constexpr int ESZ = DT == DT_F32 ? 4 : 2;
    float acc[kKC][NT];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[j][t] = 0.f;
    int ci[kKC];
#pragma unroll
    for (int j = 0; j < kKC; ++j) {
        const int kj = k0 + (j < kc ? j : 0);
        // malformed channel indices read zeros (a range-checked load past x)
        const int cj = g.dense ? ci0 + (j < kc ? j : 0) : cin_idx[kj];
        ci[j] = __builtin_amdgcn_readfirstlane(unsigned(cj) < unsigned(g.cin) ? cj : 0x7fffffff / c.chan_bytes);
    }
    const int seg = lane / g.seg_len, cidx = lane - seg * g.seg_len;
    for (int sl = sl0; sl < sl1; ++sl) {
        const int u = sl * g.S + seg;
        int ld_col = -1, out_col = -1, nimg = 0, h0 = 0;
        if (seg < g.S && u < g.units) {
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
        uint32_t vy[R], vx[R + 2];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = h0 + r;
            vy[r] = (out_col >= 0 && row < g.H)
                        ? uint32_t(((nimg * g.cout + f) * g.H + row) * g.W + out_col) * uint32_t(ESZ)
                        : 0x80000000u;
        }
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            const int row = h0 - 1 + r;
            vx[r] = (ld_col >= 0 && row >= 0 && row < g.H)
                        ? uint32_t((nimg * g.cin * g.H + row) * g.W + ld_col) * uint32_t(ESZ)
                        : 0x80000000u;
        }
        float dyr[R];
        load_col<DT, R>(c.dys, vy, 0, dyr);
        float xk[kKC][R + 2];
#pragma unroll
        for (int j = 0; j < kKC; ++j)
            if (j < kc) load_col<DT, R + 2>(c.xs, vx, ci[j] * c.chan_bytes, xk[j]);
#pragma unroll
        for (int j = 0; j < kKC; ++j) {
            if (j < kc) {
                settle<R + 2>(xk[j]);
                if constexpr (NT == 9) {
                    wtap<R, 0>(acc[j][0], xk[j], dyr);
                    wtap<R, 1>(acc[j][1], xk[j], dyr);
                    wtap<R, 2>(acc[j][2], xk[j], dyr);
                    wtap<R, 3>(acc[j][3], xk[j], dyr);
                    wtap<R, 4>(acc[j][4], xk[j], dyr);
                    wtap<R, 5>(acc[j][5], xk[j], dyr);
                    wtap<R, 6>(acc[j][6], xk[j], dyr);
                    wtap<R, 7>(acc[j][7], xk[j], dyr);
                    wtap<R, 8>(acc[j][8], xk[j], dyr);
                } else if constexpr (QD) {
                    wtap_dyn<R>(q[0], acc[j][0], xk[j], dyr);
                    wtap_dyn<R>(q[1], acc[j][1], xk[j], dyr);
                    wtap_dyn<R>(q[2], acc[j][2], xk[j], dyr);
                    wtap_dyn<R>(q[3], acc[j][3], xk[j], dyr);
                } else {
                    wtap<R, Q0>(acc[j][0], xk[j], dyr);
                    wtap<R, Q1>(acc[j][1], xk[j], dyr);
                    wtap<R, Q2>(acc[j][2], xk[j], dyr);
                    wtap<R, Q3>(acc[j][3], xk[j], dyr);
                }
            }
        }
    }
    if constexpr (NT == 4) {
        float a[kKC * 4];
#pragma unroll
        for (int j = 0; j < kKC; ++j)
#pragma unroll
            for (int t = 0; t < 4; ++t) a[j * 4 + t] = acc[j][t];
        const int v = wave_reduce_scatter<kKC * 4>(a, lane);
        // lanes with the same index hold the same sum: the lowest one writes it
        if ((lane & (64 / (kKC * 4) - 1)) == 0 && v / 4 < kc) out[int64_t(k0 + v / 4) * 4 + (v % 4)] = a[0];
    } else {
#pragma unroll
        for (int j = 0; j < kKC; ++j)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                float v = acc[j][t];
                for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
                acc[j][t] = v;
            }
        if (lane == 0)
#pragma unroll
            for (int j = 0; j < kKC; ++j)
                if (j < kc)
#pragma unroll
                    for (int t = 0; t < NT; ++t) out[int64_t(k0 + j) * NT + t] = acc[j][t];
    }
}

// ---- one band group per wave (small planes at small batch): the wave's dy
// rows are loaded once, and the channel indices and x rows of its next chunk
// load while the current chunk's FMAs and wave reduction run.  A wave takes
// the chunks j = grp, grp + G, ... of its filter (counted over the pattern
// segments in storage order).

// Per-lane byte offsets of the R dy rows and the R+2 x rows (channel 0) of
// slot sl in the one-column layout; past the buffer range for padding.
template <int DT, int R>
__device__ __forceinline__ void slot_offsets(const WGeo& g, int f, int sl, int lane, uint32_t (&vy)[R],
                                             uint32_t (&vx)[R + 2]) {
    constexpr int ESZ = DT == DT_F32 ? 4 : 2;
    const int seg = lane / g.seg_len, cidx = lane - seg * g.seg_len;
    const int u = sl * g.S + seg;
    int ld_col = -1, out_col = -1, nimg = 0, h0 = 0;
    if (seg < g.S && u < g.units) {
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
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = h0 + r;
        vy[r] = (out_col >= 0 && row < g.H) ? uint32_t(((nimg * g.cout + f) * g.H + row) * g.W + out_col) * uint32_t(ESZ)
                                            : 0x80000000u;
    }
#pragma unroll
    for (int r = 0; r < R + 2; ++r) {
        const int row = h0 - 1 + r;
        vx[r] = (ld_col >= 0 && row >= 0 && row < g.H)
                    ? uint32_t((nimg * g.cin * g.H + row) * g.W + ld_col) * uint32_t(ESZ)
                    : 0x80000000u;
    }
}

// One chunk of the wave's sequence: kernels [k0, k0 + kc) of segment p.
struct WChunk {
    int p, k0, kc;
    bool valid;
};

// The chunk with index j of the filter (j counted over the segments from
// segment p on, whose first chunk has index jb), or invalid past the end.
__device__ __forceinline__ WChunk chunk_at(const WGeo& g, const int32_t* segp, int p, int jb, int j) {
    for (; p < g.m; ++p) {
        const int a = segp[p], b = segp[p + 1];
        const int nc = b > a ? (b - a + kKC - 1) / kKC : 0;
        if (j < jb + nc) {
            const int k0 = a + (j - jb) * kKC;
            return WChunk{p, k0, b - k0 < kKC ? b - k0 : kKC, true};
        }
        jb += nc;
    }
    return WChunk{g.m, 0, 0, false};
}

template <int DT, int R>
__device__ __forceinline__ void load_chunk(const WGeo& g, const WCtx& c, const int32_t* __restrict__ cin_idx,
                                           const WChunk& ch, const uint32_t (&vx)[R + 2], float (&xk)[kKC][R + 2]) {
#pragma unroll
    for (int j = 0; j < kKC; ++j) {
        if (j < ch.kc) {
            const int cj = cin_idx[ch.k0 + j];
            // malformed channel indices read zeros (a range-checked load past x)
            const int ci = __builtin_amdgcn_readfirstlane(unsigned(cj) < unsigned(g.cin) ? cj : 0x7fffffff / c.chan_bytes);
            load_col<DT, R + 2>(c.xs, vx, ci * c.chan_bytes, xk[j]);
        }
    }
}

template <int R, bool QD, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void chunk_taps(float (&acc)[kKC][4], float (&xk)[kKC][R + 2], const float (&dyr)[R],
                                           int kc, const int (&q)[4]) {
#pragma unroll
    for (int j = 0; j < kKC; ++j) {
        if (j < kc) {
            settle<R + 2>(xk[j]);
            if constexpr (QD) {
                wtap_dyn<R>(q[0], acc[j][0], xk[j], dyr);
                wtap_dyn<R>(q[1], acc[j][1], xk[j], dyr);
                wtap_dyn<R>(q[2], acc[j][2], xk[j], dyr);
                wtap_dyn<R>(q[3], acc[j][3], xk[j], dyr);
            } else {
                wtap<R, Q0>(acc[j][0], xk[j], dyr);
                wtap<R, Q1>(acc[j][1], xk[j], dyr);
                wtap<R, Q2>(acc[j][2], xk[j], dyr);
                wtap<R, Q3>(acc[j][3], xk[j], dyr);
            }
        }
    }
}

#define PSC_WP_CASE(I)                                                                                      \
    case I:                                                                                                 \
        chunk_taps<R, false, NthBit<kCentre3.code[I], 0>::value(), NthBit<kCentre3.code[I], 1>::value(),    \
                   NthBit<kCentre3.code[I], 2>::value(), NthBit<kCentre3.code[I], 3>::value()>(acc, xk, dyr, \
                                                                                               kc, q);      \
        return;
#define PSC_WP_CASE8(I)                                                                             \
    PSC_WP_CASE(I) PSC_WP_CASE(I + 1) PSC_WP_CASE(I + 2) PSC_WP_CASE(I + 3) PSC_WP_CASE(I + 4)      \
    PSC_WP_CASE(I + 5) PSC_WP_CASE(I + 6) PSC_WP_CASE(I + 7)
template <int R>
__device__ __forceinline__ void chunk_taps_pattern(int shape, float (&acc)[kKC][4], float (&xk)[kKC][R + 2],
                                                   const float (&dyr)[R], int kc, const int (&q)[4]) {
    switch (shape) {
        PSC_WP_CASE8(0)
        PSC_WP_CASE8(8)
        PSC_WP_CASE8(16)
        PSC_WP_CASE8(24)
        PSC_WP_CASE8(32)
        PSC_WP_CASE8(40)
        PSC_WP_CASE8(48)
        default: chunk_taps<R, true, 0, 0, 0, 0>(acc, xk, dyr, kc, q); return;
    }
}
#undef PSC_WP_CASE8
#undef PSC_WP_CASE

// The chunk's kc x 4 sums over the wave, written by the lanes that hold them.
__device__ __forceinline__ void chunk_write(float (&acc)[kKC][4], int k0, int kc, int lane, float* __restrict__ out) {
    float a[kKC * 4];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) a[j * 4 + t] = acc[j][t];
    const int v = wave_reduce_scatter<kKC * 4>(a, lane);
    if ((lane & (64 / (kKC * 4) - 1)) == 0 && v / 4 < kc) out[int64_t(k0 + v / 4) * 4 + (v % 4)] = a[0];
}

__device__ __forceinline__ void pattern_taps(unsigned mk, int (&q)[4]) {
    int t = 0;
    q[0] = q[1] = q[2] = q[3] = 4;
    for (int u = 0; u < 9; ++u)
        if ((mk >> u) & 1u) {
            if (t < 4) q[t] = u;
            ++t;
        }
}

// One chunk of the pipeline: the next chunk's rows start loading into xn,
// then the current chunk's taps and reduction run on xc.
template <int DT, int R>
__device__ __forceinline__ WChunk pipe_step(const WGeo& g, const WCtx& c, const int32_t* segp,
                                            const int32_t* __restrict__ cin_idx, const uint32_t (&vx)[R + 2],
                                            const float (&dyr)[R], const WChunk& cur, int jc,
                                            float (&xc)[kKC][R + 2], float (&xn)[kKC][R + 2], int lane,
                                            float* __restrict__ out) {
    const WChunk nx = chunk_at(g, segp, cur.p, jc - (cur.k0 - segp[cur.p]) / kKC, jc + g.G);
    if (nx.valid) load_chunk<DT, R>(g, c, cin_idx, nx, vx, xn);
    float acc[kKC][4];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[j][t] = 0.f;
    int q[4];
    pattern_taps(g.mask[cur.p], q);
    chunk_taps_pattern<R>(g.shape[cur.p], acc, xc, dyr, cur.kc, q);
    chunk_write(acc, cur.k0, cur.kc, lane, out);
    return nx;
}

template <int DT, int R>
__device__ __forceinline__ void run_filter_pipe(const WGeo& g, const WCtx& c, const int32_t* segp,
                                                const int32_t* __restrict__ cin_idx, int f, int grp, int lane,
                                                float* __restrict__ out) {
    uint32_t vy[R], vx[R + 2];
    slot_offsets<DT, R>(g, f, 0, lane, vy, vx);
    float dyr[R];
    load_col<DT, R>(c.dys, vy, 0, dyr);
    WChunk cA = chunk_at(g, segp, 0, 0, grp);
    if (!cA.valid) return;
    int jA = grp;
    float xA[kKC][R + 2], xB[kKC][R + 2];
    load_chunk<DT, R>(g, c, cin_idx, cA, vx, xA);
    while (true) {
        const WChunk cB = pipe_step<DT, R>(g, c, segp, cin_idx, vx, dyr, cA, jA, xA, xB, lane, out);
        if (!cB.valid) break;
        cA = pipe_step<DT, R>(g, c, segp, cin_idx, vx, dyr, cB, jA + g.G, xB, xA, lane, out);
        jA += 2 * g.G;
        if (!cA.valid) break;
    }
}

// ---- four columns per lane.  A lane owns columns 4c..4c+3 and R rows of a
// full-row band; segments are padded to a multiple of 4 lanes, so every
// segment ends in at least one zero lane.  Per band a lane loads its R dy rows
// and, for each kernel of the chunk, its R+2 x rows, each as one load; the
// column left of the lane's four is the left lane's last (DPP wave_shr), the
// one right of them the right lane's first (wave_shl).

// R rows of 4 columns through a buffer descriptor, widened to fp32.
template <int DT, int N>
__device__ __forceinline__ void load_row4(__amdgpu_buffer_rsrc_t rs, const uint32_t (&vo)[N], int soff,
                                          float (&v)[N][4]) {
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if constexpr (DT == DT_F32) {
            // the words are copied out before the casts: hipcc compiles a bit
            // cast of a vector-element lvalue as a read of element 0
            const rw::u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(rs, int(vo[r]), soff, 0);
            const uint32_t w0 = w.x, w1 = w.y, w2 = w.z, w3 = w.w;
            v[r][0] = __builtin_bit_cast(float, w0), v[r][1] = __builtin_bit_cast(float, w1);
            v[r][2] = __builtin_bit_cast(float, w2), v[r][3] = __builtin_bit_cast(float, w3);
        } else {
            const rw::u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(rs, int(vo[r]), soff, 0);
            v[r][0] = float(__builtin_bit_cast(_Float16, uint16_t(w.x)));
            v[r][1] = float(__builtin_bit_cast(_Float16, uint16_t(w.x >> 16)));
            v[r][2] = float(__builtin_bit_cast(_Float16, uint16_t(w.y)));
            v[r][3] = float(__builtin_bit_cast(_Float16, uint16_t(w.y >> 16)));
        }
    }
}

#define PSC_W_SHR "v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_W_SHL "v_fmac_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
// Column c of row r of the tap at kernel position Q: acc += x(row r + ky,
// column c + kx - 1) * dy(row r, column c).
template <int Q, int C, int R>
__device__ __forceinline__ void wtap4_at(float& acc, const float (&x)[R + 2][4], const float (&dy)[R][4], int r) {
    constexpr int ky = Q / 3, col = C + Q % 3 - 1;
    if constexpr (col < 0)
        asm volatile(PSC_W_SHR : "+v"(acc) : "v"(x[r + ky][3]), "v"(dy[r][C]));
    else if constexpr (col > 3)
        asm volatile(PSC_W_SHL : "+v"(acc) : "v"(x[r + ky][0]), "v"(dy[r][C]));
    else
        acc = __builtin_fmaf(x[r + ky][col], dy[r][C], acc);
}
#undef PSC_W_SHL
#undef PSC_W_SHR

template <int Q, int R>
__device__ __forceinline__ void wtap4(float& acc, const float (&x)[R + 2][4], const float (&dy)[R][4]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        wtap4_at<Q, 0, R>(acc, x, dy, r);
        wtap4_at<Q, 1, R>(acc, x, dy, r);
        wtap4_at<Q, 2, R>(acc, x, dy, r);
        wtap4_at<Q, 3, R>(acc, x, dy, r);
    }
}

template <int R>
__device__ __forceinline__ void wtap4_dyn(int q, float& acc, const float (&x)[R + 2][4], const float (&dy)[R][4]) {
    switch (q) {
        case 0: wtap4<0, R>(acc, x, dy); break;
        case 1: wtap4<1, R>(acc, x, dy); break;
        case 2: wtap4<2, R>(acc, x, dy); break;
        case 3: wtap4<3, R>(acc, x, dy); break;
        case 4: wtap4<4, R>(acc, x, dy); break;
        case 5: wtap4<5, R>(acc, x, dy); break;
        case 6: wtap4<6, R>(acc, x, dy); break;
        case 7: wtap4<7, R>(acc, x, dy); break;
        default: wtap4<8, R>(acc, x, dy); break;
    }
}

// The chunk [k0, k0 + kc) as in run_chunk, four columns per lane.
template <int DT, int R, int NT, bool QD, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void run_chunk_wide(const WGeo& g, const WCtx& c, const int32_t* __restrict__ cin_idx,
                                               int f, int k0, int kc, int ci0, const int (&q)[4], int sl0, int sl1,
                                               int lane, float* __restrict__ out) {
    constexpr int ESZ = DT == DT_F32 ? 4 : 2;
    float acc[kKC][NT];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[j][t] = 0.f;
    int ci[kKC];
#pragma unroll
    for (int j = 0; j < kKC; ++j) {
        const int kj = k0 + (j < kc ? j : 0);
        // malformed channel indices read zeros (a range-checked load past x)
        const int cj = g.dense ? ci0 + (j < kc ? j : 0) : cin_idx[kj];
        ci[j] = __builtin_amdgcn_readfirstlane(unsigned(cj) < unsigned(g.cin) ? cj : 0x7fffffff / c.chan_bytes);
    }
    const int seg = lane / g.seg_len, cidx = lane - seg * g.seg_len;
    for (int sl = sl0; sl < sl1; ++sl) {
        const int u = sl * g.S + seg;
        int col0 = -1, nimg = 0, h0 = 0;
        if (seg < g.S && u < g.units) {
            nimg = u / g.RB;
            h0 = (u - nimg * g.RB) * R;
            if (4 * cidx < g.W) col0 = 4 * cidx;
        }
        uint32_t vy[R], vx[R + 2];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int row = h0 + r;
            vy[r] = (col0 >= 0 && row < g.H) ? uint32_t(((nimg * g.cout + f) * g.H + row) * g.W + col0) * uint32_t(ESZ)
                                             : 0x80000000u;
        }
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            const int row = h0 - 1 + r;
            vx[r] = (col0 >= 0 && row >= 0 && row < g.H)
                        ? uint32_t((nimg * g.cin * g.H + row) * g.W + col0) * uint32_t(ESZ)
                        : 0x80000000u;
        }
        float dyr[R][4];
        load_row4<DT, R>(c.dys, vy, 0, dyr);
        float xk[kKC][R + 2][4];
#pragma unroll
        for (int j = 0; j < kKC; ++j)
            if (j < kc) load_row4<DT, R + 2>(c.xs, vx, ci[j] * c.chan_bytes, xk[j]);
        // the DPP sources (first and last column of every x row) as written
        // by an asm, then the wait states a DPP read needs after a VALU write
#pragma unroll
        for (int j = 0; j < kKC; ++j)
#pragma unroll
            for (int r = 0; r < R + 2; ++r) asm volatile("" : "+v"(xk[j][r][0]), "+v"(xk[j][r][3]));
        asm volatile("s_nop 1");
#pragma unroll
        for (int j = 0; j < kKC; ++j) {
            if (j < kc) {
                if constexpr (NT == 9) {
                    wtap4<0, R>(acc[j][0], xk[j], dyr);
                    wtap4<1, R>(acc[j][1], xk[j], dyr);
                    wtap4<2, R>(acc[j][2], xk[j], dyr);
                    wtap4<3, R>(acc[j][3], xk[j], dyr);
                    wtap4<4, R>(acc[j][4], xk[j], dyr);
                    wtap4<5, R>(acc[j][5], xk[j], dyr);
                    wtap4<6, R>(acc[j][6], xk[j], dyr);
                    wtap4<7, R>(acc[j][7], xk[j], dyr);
                    wtap4<8, R>(acc[j][8], xk[j], dyr);
                } else if constexpr (QD) {
                    wtap4_dyn<R>(q[0], acc[j][0], xk[j], dyr);
                    wtap4_dyn<R>(q[1], acc[j][1], xk[j], dyr);
                    wtap4_dyn<R>(q[2], acc[j][2], xk[j], dyr);
                    wtap4_dyn<R>(q[3], acc[j][3], xk[j], dyr);
                } else {
                    wtap4<Q0, R>(acc[j][0], xk[j], dyr);
                    wtap4<Q1, R>(acc[j][1], xk[j], dyr);
                    wtap4<Q2, R>(acc[j][2], xk[j], dyr);
                    wtap4<Q3, R>(acc[j][3], xk[j], dyr);
                }
            }
        }
    }
    if constexpr (NT == 4) {
        float a[kKC * 4];
#pragma unroll
        for (int j = 0; j < kKC; ++j)
#pragma unroll
            for (int t = 0; t < 4; ++t) a[j * 4 + t] = acc[j][t];
        const int v = wave_reduce_scatter<kKC * 4>(a, lane);
        // lanes with the same index hold the same sum: the lowest one writes it
        if ((lane & (64 / (kKC * 4) - 1)) == 0 && v / 4 < kc) out[int64_t(k0 + v / 4) * 4 + (v % 4)] = a[0];
    } else {
#pragma unroll
        for (int j = 0; j < kKC; ++j)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                float v = acc[j][t];
                for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
                acc[j][t] = v;
            }
        if (lane == 0)
#pragma unroll
            for (int j = 0; j < kKC; ++j)
                if (j < kc)
#pragma unroll
                    for (int t = 0; t < NT; ++t) out[int64_t(k0 + j) * NT + t] = acc[j][t];
    }
}

template <int DT, int R, int MASK>
__device__ __forceinline__ void run_chunk_wide_shape(const WGeo& g, const WCtx& c, const int32_t* cin_idx, int f,
                                                     int k0, int kc, const int (&q)[4], int sl0, int sl1, int lane,
                                                     float* out) {
    run_chunk_wide<DT, R, 4, false, NthBit<MASK, 0>::value(), NthBit<MASK, 1>::value(), NthBit<MASK, 2>::value(),
                   NthBit<MASK, 3>::value()>(g, c, cin_idx, f, k0, kc, 0, q, sl0, sl1, lane, out);
}

#define PSC_WW_CASE(I) \
    case I: run_chunk_wide_shape<DT, R, kCentre3.code[I]>(g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, out); return;
#define PSC_WW_CASE8(I)                                                                             \
    PSC_WW_CASE(I) PSC_WW_CASE(I + 1) PSC_WW_CASE(I + 2) PSC_WW_CASE(I + 3) PSC_WW_CASE(I + 4)      \
    PSC_WW_CASE(I + 5) PSC_WW_CASE(I + 6) PSC_WW_CASE(I + 7)
template <int DT, int R>
__device__ __forceinline__ void run_chunk_wide_pattern(int shape, const WGeo& g, const WCtx& c,
                                                       const int32_t* cin_idx, int f, int k0, int kc,
                                                       const int (&q)[4], int sl0, int sl1, int lane, float* out) {
    switch (shape) {
        PSC_WW_CASE8(0)
        PSC_WW_CASE8(8)
        PSC_WW_CASE8(16)
        PSC_WW_CASE8(24)
        PSC_WW_CASE8(32)
        PSC_WW_CASE8(40)
        PSC_WW_CASE8(48)
        default:
            run_chunk_wide<DT, R, 4, true, 0, 0, 0, 0>(g, c, cin_idx, f, k0, kc, 0, q, sl0, sl1, lane, out);
            return;
    }
}
#undef PSC_WW_CASE8
#undef PSC_WW_CASE

// ---- one image row per lane (small planes at large batch).  A wave holds S
// images, H row lanes each and a zero lane after each image; per image group
// a lane loads its dy row once (16-byte loads) and, for each kernel of the
// chunk, its x row; the rows above and below come from the neighbouring
// lanes by DPP inside the FMA, the left and right columns are other
// registers of the lane.
#define PSC_W_SHR "v_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
#define PSC_W_SHL "v_fmac_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
// acc += sum_c x(row r + ky - 1, column c + kx - 1) * dy[c] over the columns
// inside the row.
template <int W, int Q>
__device__ __forceinline__ void wtap_row(float& acc, const float (&x)[W], const float (&dyv)[W]) {
    constexpr int ky = Q / 3, kx = Q % 3;
    constexpr int c0 = kx == 0 ? 1 : 0, c1 = kx == 2 ? W - 1 : W;
#pragma unroll
    for (int c = c0; c < c1; ++c) {
        if constexpr (ky == 1)
            acc = __builtin_fmaf(x[c + kx - 1], dyv[c], acc);
        else if constexpr (ky == 0)
            asm volatile(PSC_W_SHR : "+v"(acc) : "v"(x[c + kx - 1]), "v"(dyv[c]));
        else
            asm volatile(PSC_W_SHL : "+v"(acc) : "v"(x[c + kx - 1]), "v"(dyv[c]));
    }
}
#undef PSC_W_SHL
#undef PSC_W_SHR

template <int W>
__device__ __forceinline__ void wtap_row_dyn(int q, float& acc, const float (&x)[W], const float (&dyv)[W]) {
    switch (q) {
        case 0: wtap_row<W, 0>(acc, x, dyv); break;
        case 1: wtap_row<W, 1>(acc, x, dyv); break;
        case 2: wtap_row<W, 2>(acc, x, dyv); break;
        case 3: wtap_row<W, 3>(acc, x, dyv); break;
        case 4: wtap_row<W, 4>(acc, x, dyv); break;
        case 5: wtap_row<W, 5>(acc, x, dyv); break;
        case 6: wtap_row<W, 6>(acc, x, dyv); break;
        case 7: wtap_row<W, 7>(acc, x, dyv); break;
        default: wtap_row<W, 8>(acc, x, dyv); break;
    }
}

template <int DT, int W, bool QD, int Q0, int Q1, int Q2, int Q3>
__device__ __forceinline__ void run_chunk_rows(const WGeo& g, const WCtx& c, const int32_t* __restrict__ cin_idx,
                                               int f, int k0, int kc, const int (&q)[4], int sl0, int sl1,
                                               int lane, float* __restrict__ out) {
    constexpr int ESZ = DT == DT_F32 ? 4 : 2;
    float acc[kKC][4];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[j][t] = 0.f;
    int soff[kKC];
#pragma unroll
    for (int j = 0; j < kKC; ++j) {
        const int cj = cin_idx[k0 + (j < kc ? j : 0)];
        // malformed channel indices read zeros (an offset past the range of x)
        soff[j] = __builtin_amdgcn_readfirstlane(unsigned(cj) < unsigned(g.cin) ? cj * c.chan_bytes : 0x7fffffff);
    }
    const int seg = lane / g.seg_len, r = lane - seg * g.seg_len;
    for (int sl = sl0; sl < sl1; ++sl) {
        const int img = sl * g.S + seg;
        const bool valid = seg < g.S && img < g.n && r < g.H;
        const uint32_t vx = valid ? uint32_t((img * g.cin * g.H + r) * g.W) * uint32_t(ESZ) : 0x80000000u;
        const uint32_t vy = valid ? uint32_t(((img * g.cout + f) * g.H + r) * g.W) * uint32_t(ESZ) : 0x80000000u;
        rw::RowWords<DT, W, 1> wy, wx[kKC];
        rw::load_words<DT, W, 1>(c.dys, vy, 0x80000000u, 0, g.dy_bytes, valid, wy);
#pragma unroll
        for (int j = 0; j < kKC; ++j)
            if (j < kc) rw::load_words<DT, W, 1>(c.xs, vx, 0x80000000u, soff[j], g.x_bytes, valid, wx[j]);
        rw::RowVals<W, 1> yv;
        rw::unpack_vals<DT, W, 1>(wy, yv);
#pragma unroll
        for (int j = 0; j < kKC; ++j) {
            if (j < kc) {
                rw::RowVals<W, 1> xv;
                rw::unpack_vals<DT, W, 1>(wx[j], xv);   // ends with the settle a DPP source needs
                if constexpr (QD) {
                    wtap_row_dyn<W>(q[0], acc[j][0], xv.e, yv.e);
                    wtap_row_dyn<W>(q[1], acc[j][1], xv.e, yv.e);
                    wtap_row_dyn<W>(q[2], acc[j][2], xv.e, yv.e);
                    wtap_row_dyn<W>(q[3], acc[j][3], xv.e, yv.e);
                } else {
                    wtap_row<W, Q0>(acc[j][0], xv.e, yv.e);
                    wtap_row<W, Q1>(acc[j][1], xv.e, yv.e);
                    wtap_row<W, Q2>(acc[j][2], xv.e, yv.e);
                    wtap_row<W, Q3>(acc[j][3], xv.e, yv.e);
                }
            }
        }
    }
    float a[kKC * 4];
#pragma unroll
    for (int j = 0; j < kKC; ++j)
#pragma unroll
        for (int t = 0; t < 4; ++t) a[j * 4 + t] = acc[j][t];
    const int v = wave_reduce_scatter<kKC * 4>(a, lane);
    if ((lane & (64 / (kKC * 4) - 1)) == 0 && v / 4 < kc) out[int64_t(k0 + v / 4) * 4 + (v % 4)] = a[0];
}

template <int DT, int W, int MASK>
__device__ __forceinline__ void run_chunk_rows_shape(const WGeo& g, const WCtx& c, const int32_t* cin_idx, int f,
                                                     int k0, int kc, const int (&q)[4], int sl0, int sl1, int lane,
                                                     float* out) {
    run_chunk_rows<DT, W, false, NthBit<MASK, 0>::value(), NthBit<MASK, 1>::value(), NthBit<MASK, 2>::value(),
                   NthBit<MASK, 3>::value()>(g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, out);
}

#define PSC_WR_CASE(I) \
    case I: run_chunk_rows_shape<DT, W, kCentre3.code[I]>(g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, out); return;
#define PSC_WR_CASE8(I)                                                                             \
    PSC_WR_CASE(I) PSC_WR_CASE(I + 1) PSC_WR_CASE(I + 2) PSC_WR_CASE(I + 3) PSC_WR_CASE(I + 4)      \
    PSC_WR_CASE(I + 5) PSC_WR_CASE(I + 6) PSC_WR_CASE(I + 7)
template <int DT, int W>
__device__ __forceinline__ void run_chunk_rows_pattern(int shape, const WGeo& g, const WCtx& c,
                                                       const int32_t* cin_idx, int f, int k0, int kc,
                                                       const int (&q)[4], int sl0, int sl1, int lane, float* out) {
    switch (shape) {
        PSC_WR_CASE8(0)
        PSC_WR_CASE8(8)
        PSC_WR_CASE8(16)
        PSC_WR_CASE8(24)
        PSC_WR_CASE8(32)
        PSC_WR_CASE8(40)
        PSC_WR_CASE8(48)
        default: run_chunk_rows<DT, W, true, 0, 0, 0, 0>(g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, out); return;
    }
}
#undef PSC_WR_CASE8
#undef PSC_WR_CASE

template <int DT, int R, int MASK>
__device__ __forceinline__ void run_chunk_shape(const WGeo& g, const WCtx& c, const int32_t* cin_idx, int f, int k0,
                                                int kc, const int (&q)[4], int sl0, int sl1, int lane, float* out) {
    run_chunk<DT, R, 4, false, NthBit<MASK, 0>::value(), NthBit<MASK, 1>::value(), NthBit<MASK, 2>::value(),
              NthBit<MASK, 3>::value()>(g, c, cin_idx, f, k0, kc, 0, q, sl0, sl1, lane, out);
}

#define PSC_WG_CASE(I) \
    case I: run_chunk_shape<DT, R, kCentre3.code[I]>(g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, out); return;
#define PSC_WG_CASE8(I)                                                                             \
    PSC_WG_CASE(I) PSC_WG_CASE(I + 1) PSC_WG_CASE(I + 2) PSC_WG_CASE(I + 3) PSC_WG_CASE(I + 4)      \
    PSC_WG_CASE(I + 5) PSC_WG_CASE(I + 6) PSC_WG_CASE(I + 7)
template <int DT, int R>
__device__ __forceinline__ void run_chunk_pattern(int shape, const WGeo& g, const WCtx& c, const int32_t* cin_idx,
                                                  int f, int k0, int kc, const int (&q)[4], int sl0, int sl1,
                                                  int lane, float* out) {
    switch (shape) {
        PSC_WG_CASE8(0)
        PSC_WG_CASE8(8)
        PSC_WG_CASE8(16)
        PSC_WG_CASE8(24)
        PSC_WG_CASE8(32)
        PSC_WG_CASE8(40)
        PSC_WG_CASE8(48)
        default: run_chunk<DT, R, 4, true, 0, 0, 0, 0>(g, c, cin_idx, f, k0, kc, 0, q, sl0, sl1, lane, out); return;
    }
}
#undef PSC_WG_CASE8
#undef PSC_WG_CASE

// One wave per (filter, chunk group, image share); chunk j of the filter
// (counted over its pattern segments in storage order) belongs to group
// j % G.
// W > 0: one image row per lane (masked gradients on planes of W columns);
// WIDE: 4 columns per lane; PIPE: one slot per wave, chunks pipelined.
template <int DT, int R, int NT, int W = 0, bool WIDE = false, bool PIPE = false>
__global__ __launch_bounds__(256) void k_wgrad(const typename Elt<DT>::T* __restrict__ x,
                                               const typename Elt<DT>::T* __restrict__ dy,
                                               const int32_t* __restrict__ perm, const int32_t* __restrict__ seg_ptr,
                                               const int32_t* __restrict__ cin_idx, WGeo g, float* __restrict__ out) {
    using E = Elt<DT>;
    constexpr int ESZ = int(sizeof(typename E::T));
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t per_filter = int64_t(g.G) * g.KS;
    const int i = __builtin_amdgcn_readfirstlane(int(wid / per_filter));
    if (i >= g.cout) return;                                 // whole waves leave together
    const int rem = int(wid - int64_t(i) * per_filter);
    const int grp = rem / g.KS, s = rem - grp * g.KS;
    const int sl0 = int(int64_t(g.slots) * s / g.KS), sl1 = int(int64_t(g.slots) * (s + 1) / g.KS);
    WCtx c;
    c.xs = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(x), int16_t(0), g.x_bytes, 0x00020000);
    c.dys = __builtin_amdgcn_make_buffer_rsrc(const_cast<typename E::T*>(dy), int16_t(0), g.dy_bytes, 0x00020000);
    c.chan_bytes = g.H * g.W * ESZ;
    float* o = out + int64_t(s) * g.nk * NT;
    const int q0[4] = {4, 4, 4, 4};
    if constexpr (NT == 9) {
        const int f = i;
        int j = 0;
        for (int c0 = 0; c0 < g.cin; c0 += kKC, ++j) {
            if (j % g.G != grp) continue;
            const int kc = g.cin - c0 < kKC ? g.cin - c0 : kKC;
            if constexpr (WIDE)
                run_chunk_wide<DT, R, 9, false, 0, 0, 0, 0>(g, c, nullptr, f, f * g.cin + c0, kc, c0, q0, sl0, sl1,
                                                            lane, o);
            else
                run_chunk<DT, R, 9, false, 0, 0, 0, 0>(g, c, nullptr, f, f * g.cin + c0, kc, c0, q0, sl0, sl1, lane,
                                                       o);
        }
    } else {
        const int f = perm[i];
        const int* segp = seg_ptr + int64_t(i) * (g.m + 1);
        if constexpr (PIPE) {
            run_filter_pipe<DT, R>(g, c, segp, cin_idx, f, grp, lane, o);
            return;
        }
        int j = 0;
        for (int p = 0; p < g.m; ++p) {
            const int k1 = segp[p + 1];
            int q[4] = {4, 4, 4, 4}, t = 0;
            const unsigned mk = g.mask[p];
            for (int u = 0; u < 9; ++u)
                if ((mk >> u) & 1u) {
                    if (t < 4) q[t] = u;
                    ++t;
                }
            for (int k0 = segp[p]; k0 < k1; k0 += kKC, ++j) {
                if (j % g.G != grp) continue;
                const int kc = k1 - k0 < kKC ? k1 - k0 : kKC;
                if constexpr (WIDE)
                    run_chunk_wide_pattern<DT, R>(g.shape[p], g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, o);
                else if constexpr (W > 0)
                    run_chunk_rows_pattern<DT, W>(g.shape[p], g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, o);
                else
                    run_chunk_pattern<DT, R>(g.shape[p], g, c, cin_idx, f, k0, kc, q, sl0, sl1, lane, o);
            }
        }
    }
}

// Launch of k_wgrad with these template arguments; each one is
// instantiated in one of the wgrad_*.hip translation units.
template <int DT, int R, int NT, int W, bool WIDE, bool PIPE>
hipError_t launch_wgrad(dim3 grid, const void* x, const void* dy, const int32_t* perm, const int32_t* seg_ptr,
                        const int32_t* cin_idx, const WGeo& g, float* dst, hipStream_t stream) {
    using T = typename Elt<DT>::T;
    hipLaunchKernelGGL((k_wgrad<DT, R, NT, W, WIDE, PIPE>), grid, dim3(256), 0, stream, static_cast<const T*>(x),
                       static_cast<const T*>(dy), perm, seg_ptr, cin_idx, g, dst);
    return hipGetLastError();
}

constexpr int kWideRows = 2;   // rows per lane of the 4-column layout

}  // namespace wg
}  // namespace psc
