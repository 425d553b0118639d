// Weight gradients of the 3x3 layer: the host side (work layout, launches,
// the share and bias reductions).  The kernels and their layouts are
// described in wgrad.h and instantiated in the wgrad_*.hip units.
#include "wgrad.h"

namespace psc {
namespace wg {
extern template hipError_t launch_wgrad<DT_F32, 8, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 8, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 8, 9, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 9, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, kWideRows, 4, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, kWideRows, 4, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, kWideRows, 9, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 4, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 7, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 8, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 14, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 16, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 4, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 7, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 8, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 14, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 16, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 8, 4, 0, false, true>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F32, 4, 4, 0, false, true>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 8, 4, 0, false, true>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
extern template hipError_t launch_wgrad<DT_F16, 4, 4, 0, false, true>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
}  // namespace wg

namespace {
using namespace wg;

// out[e] = sum over shares s (in order) of part[s][e]; the loads of four
// shares are issued together, the adds keep the share order.
__global__ __launch_bounds__(256) void k_wgrad_reduce(const float* __restrict__ part, int KS, int64_t n,
                                                      float* __restrict__ out) {
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256) {
        float v = part[e];
        int s = 1;
        for (; s + 4 <= KS; s += 4) {
            const float a = part[int64_t(s) * n + e], b = part[int64_t(s + 1) * n + e];
            const float c = part[int64_t(s + 2) * n + e], d = part[int64_t(s + 3) * n + e];
            v += a;
            v += b;
            v += c;
            v += d;
        }
        for (; s < KS; ++s) v += part[int64_t(s) * n + e];
        out[e] = v;
    }
}

// Bias gradient db[f] = sum over images and pixels of dy[n, f], in P parts
// per filter: part p of filter f sums elements [total p / P, total (p+1) / P)
// of its images x pixels (total = n * plane; element e is pixel e % plane of
// image e / plane), each thread with 4 independent accumulators; the parts
// go to out[p * cout + f] (P > 1; k_wgrad_reduce adds them in part order) or
// to db (P = 1).  Grid (cout, P), 256 threads.
constexpr int kBiasPartElems = 8192;

int bias_parts(int n, int plane) {
    const int64_t total = int64_t(n) * plane;
    int64_t P = (total + kBiasPartElems - 1) / kBiasPartElems;
    return int(P < 1 ? 1 : P > 1024 ? 1024 : P);
}

template <int DT>
__global__ __launch_bounds__(256) void k_bias_grad(const typename Elt<DT>::T* __restrict__ dy, int n, int cout,
                                                   int plane, int P, float* __restrict__ out) {
    using E = Elt<DT>;
    __shared__ float part[4];
    const int f = blockIdx.x, p = blockIdx.y;
    const int64_t total = int64_t(n) * plane;
    const int64_t e0 = total * p / P, e1 = total * (p + 1) / P;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    auto at = [&](int64_t e) -> float {
        const int64_t img = e / plane;
        return E::load(dy, (img * cout + f) * plane + (e - img * plane));
    };
    int64_t e = e0 + threadIdx.x;
    for (; e + 768 < e1; e += 1024) {
        const float v0 = at(e), v1 = at(e + 256), v2 = at(e + 512), v3 = at(e + 768);
        a0 += v0;
        a1 += v1;
        a2 += v2;
        a3 += v3;
    }
    for (; e < e1; e += 256) a0 += at(e);
    float acc = (a0 + a1) + (a2 + a3);
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) out[P > 1 ? int64_t(p) * cout + f : f] = (part[0] + part[1]) + (part[2] + part[3]);
}

constexpr int64_t kTargetWaves = 16384;   // 16 waves per SIMD
constexpr int64_t kPipeWaves = 3072;      // grid of the pipelined one-slot layout (3 waves per SIMD)
constexpr int kMaxShares = 64;

WGeo plan(int n, int cin, int cout, int h, int w, int64_t nk, bool dense, const PatTable* tab, int dtype) {
    WGeo g{};
    g.n = n;
    g.cin = cin;
    g.cout = cout;
    g.H = h;
    g.W = w;
    g.nk = nk;
    g.dense = dense ? 1 : 0;
    g.m = tab ? tab->m : 0;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.mask[p] = (tab && p < tab->m) ? tab->mask[p] : 0;
        g.shape[p] = -1;
        if (tab && p < tab->m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab->mask[p]) g.shape[p] = int8_t(t);
    }
    const int64_t esz = dtype == DT_F16 ? 2 : 4;
    const int64_t xb = int64_t(n) * cin * h * w * esz, yb = int64_t(n) * cout * h * w * esz;
    g.x_bytes = int(xb > 0x7fffffff ? 0x7fffffff : xb);
    g.dy_bytes = int(yb > 0x7fffffff ? 0x7fffffff : yb);
    // one image row per lane: masked gradients on compiled widths when the
    // batch fills a wave with whole images
    const bool wfit = w == 4 || w == 7 || w == 8 || w == 14 || w == 16;
    if (!dense && wfit && h <= 63 && n >= 64 / (h + 1)) {
        g.rows = 1;
        g.seg_len = h + 1;
        g.S = 64 / (h + 1);
        g.Wt = w;
        g.CT = 1;
        g.RB = 1;
        g.units = n;
        g.slots = (n + g.S - 1) / g.S;
    } else if (w % 4 == 0 && w / 4 + 1 <= 64) {
        // four columns per lane: full-row segments padded to a multiple of 4
        // lanes (at least one zero lane after each)
        g.wide = 1;
        g.cols_mode = 0;
        g.seg_len = (w / 4 + 1 + 3) / 4 * 4;
        g.S = 64 / g.seg_len;
        g.Wt = w;
        g.CT = 1;
    } else {
        // full-row segments if they use the lanes at least as well as
        // haloed column tiles (the forward's choice)
        const int S_rows = w <= 63 ? 65 / (w + 1) : 0;
        const int use_rows = S_rows * w;
        int ct = (w + 61) / 62, use_cols = 0;
        for (int t = ct; t <= w && t <= 64; ++t) {
            const int wt = (w + t - 1) / t;
            const int use = (64 / (wt + 2)) * w / t;
            if (use > use_cols) {
                use_cols = use;
                ct = t;
            }
        }
        if (S_rows > 0 && use_rows >= use_cols) {
            g.cols_mode = 0;
            g.seg_len = w + 1;
            g.S = S_rows;
            g.Wt = w;
            g.CT = 1;
        } else {
            g.cols_mode = 1;
            g.Wt = (w + ct - 1) / ct;
            g.seg_len = g.Wt + 2;
            g.S = 64 / g.seg_len;
            g.CT = ct;
        }
    }
    if (!g.rows) {
        const int R = g.wide ? kWideRows : h >= 8 ? 8 : 4;
        g.RB = (h + R - 1) / R;
        g.units = n * g.RB * g.CT;
        g.slots = (g.units + g.S - 1) / g.S;
    }
    // chunks of a filter: about its kernels / KC (the reordered filters run
    // from the most kept kernels down); spread them over G waves first, then
    // split the images into shares until the grid holds about kTargetWaves
    const int64_t per = cout > 0 ? (dense ? cin : (nk + cout - 1) / cout) : 0;
    const int64_t chunks = (per + kKC - 1) / kKC;
    if (!dense && !g.rows && !g.wide && g.slots == 1 && cout > 0) {
        // one slot: about kPipeWaves waves, each with at least 4 chunks to
        // pipeline where the filters have that many
        g.pipe = 1;
        int64_t G = kPipeWaves / cout;
        if (G > chunks / 4) G = chunks / 4;
        g.G = int(G < 1 ? 1 : G);
        g.KS = 1;
        return g;
    }
    int64_t G = cout > 0 ? kTargetWaves / cout : 1;
    if (G > chunks) G = chunks;
    g.G = int(G < 1 ? 1 : G);
    int64_t ks = cout > 0 ? kTargetWaves / (int64_t(cout) * g.G) : 1;
    if (ks > g.slots) ks = g.slots;
    if (ks > kMaxShares) ks = kMaxShares;
    g.KS = int(ks < 1 ? 1 : ks);
    return g;
}

template <int DT, int NT>
hipError_t run(const WGeo& g, const void* x, const void* dy, const int32_t* perm, const int32_t* seg_ptr,
               const int32_t* cin_idx, float* out, void* ws, hipStream_t stream) {
    if (g.nk == 0 || g.n == 0) return hipSuccess;
    float* dst = g.KS > 1 ? static_cast<float*>(ws) : out;
    const int64_t waves = int64_t(g.cout) * g.G * g.KS;
    const dim3 grid(unsigned((waves + 3) / 4));
    hipError_t e = hipSuccess;
    bool done = false;
    if constexpr (NT == 4) {
        if (g.rows) {
            switch (g.W) {
                case 4: e = launch_wgrad<DT, 4, NT, 4, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream); break;
                case 7: e = launch_wgrad<DT, 4, NT, 7, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream); break;
                case 8: e = launch_wgrad<DT, 4, NT, 8, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream); break;
                case 14: e = launch_wgrad<DT, 4, NT, 14, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream); break;
                default: e = launch_wgrad<DT, 4, NT, 16, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream); break;
            }
            done = true;
        } else if (g.pipe) {
            e = g.H >= 8 ? launch_wgrad<DT, 8, NT, 0, false, true>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream)
                         : launch_wgrad<DT, 4, NT, 0, false, true>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream);
            done = true;
        }
    }
    if (!done && g.wide) {
        e = launch_wgrad<DT, kWideRows, NT, 0, true, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream);
        done = true;
    }
    if (!done)
        e = g.H >= 8 ? launch_wgrad<DT, 8, NT, 0, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream)
                     : launch_wgrad<DT, 4, NT, 0, false, false>(grid, x, dy, perm, seg_ptr, cin_idx, g, dst, stream);
    if (e != hipSuccess || g.KS == 1) return e;
    const int64_t n = g.nk * NT;
    const int64_t gb = (n + 255) / 256;
    hipLaunchKernelGGL(k_wgrad_reduce, dim3(unsigned(gb > 8192 ? 8192 : gb)), dim3(256), 0, stream, dst, g.KS, n,
                       out);
    return hipGetLastError();
}

// db through P parts per filter (partials after the weight-gradient
// partials in the workspace when P > 1).
template <int DT>
hipError_t bias_grad(const void* dy, int n, int cout, int plane, float* db, float* part, hipStream_t stream) {
    const int P = bias_parts(n, plane);
    float* dst = P > 1 ? part : db;
    hipLaunchKernelGGL(k_bias_grad<DT>, dim3(unsigned(cout), unsigned(P)), dim3(256), 0, stream,
                       static_cast<const typename Elt<DT>::T*>(dy), n, cout, plane, P, dst);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || P == 1) return e;
    hipLaunchKernelGGL(k_wgrad_reduce, dim3(unsigned((cout + 255) / 256)), dim3(256), 0, stream, part, P,
                       int64_t(cout), db);
    return hipGetLastError();
}

}  // namespace

// Buffer descriptors address at most 2 GiB of x and of dy.
bool wgrad_fits(int n, int cin, int cout, int h, int w, int dtype) {
    const int64_t esz = dtype == DT_F16 ? 2 : 4;
    return int64_t(n) * cin * h * w * esz <= 0x7fffffff && int64_t(n) * cout * h * w * esz <= 0x7fffffff;
}

// Workspace: the image shares' weight-gradient sums (KS > 1), then the bias
// parts (P > 1).
static size_t wgrad_part_bytes(const WGeo& g, int64_t nk, bool dense) {
    return g.KS > 1 && g.n > 0 ? size_t(g.KS) * size_t(nk) * (dense ? 9 : 4) * sizeof(float) : 0;
}

// The masked gradient of a batch-1 layer of at least 16 input channels is
// taken from the dense one on the matrix cores: there the masked kernels are
// bound by load latency, and the dense GEMM over one image's pixels was
// measured faster on the VGG-16 and ResNet-50 layers although it does
// 9 / (4 keep) times the work.  Larger batches keep the masked kernels.
static bool masked_via_dense(int n, int cin, int cout, int h, int w, DenseWPlan* dp) {
    return n == 1 && dense_wgrad_mfma_plan(n, cin, cout, h, w, dp);
}

size_t wgrad_workspace_bytes(int n, int cin, int cout, int h, int w, int64_t nk, bool dense) {
    if (n <= 0) return 0;
    const int P = bias_parts(n, h * w);
    const size_t bias_bytes = P > 1 ? size_t(P) * size_t(cout) * sizeof(float) : 0;
    DenseWPlan dp;
    if (dense && dense_wgrad_mfma_plan(n, cin, cout, h, w, &dp)) return dense_wgrad_mfma_workspace(dp, cin, cout) + bias_bytes;
    // the masked route through the dense gradient needs the dense dW as well
    if (!dense && masked_via_dense(n, cin, cout, h, w, &dp)) {
        const WGeo g = plan(n, cin, cout, h, w, nk, false, nullptr, DT_F32);
        const size_t via = dense_wgrad_mfma_workspace(dp, cin, cout) + size_t(cout) * size_t(cin) * 9 * sizeof(float);
        const size_t direct = wgrad_part_bytes(g, nk, false);
        return (via > direct ? via : direct) + bias_bytes;
    }
    const WGeo g = plan(n, cin, cout, h, w, nk, dense, nullptr, DT_F32);
    return wgrad_part_bytes(g, nk, dense) + bias_bytes;
}

hipError_t launch_bwd_weight(const PatTable& tab, const PackedView& pk, int dtype, int n, int cin, int h, int w,
                             int cout, int64_t keep, const void* x, const void* dy, float* dv, float* db, void* ws,
                             hipStream_t stream) {
    const WGeo g = plan(n, cin, cout, h, w, keep, false, &tab, dtype);
    DenseWPlan dp;
    hipError_t e;
    size_t part_bytes = wgrad_part_bytes(g, keep, false);
    if (keep > 0 && masked_via_dense(n, cin, cout, h, w, &dp)) {
        // workspace: the matrix-core partial sums, then the dense dW, then
        // (after the larger of this and the masked kernels' partial sums,
        // as sized by wgrad_workspace_bytes) the bias parts
        const size_t slots = dense_wgrad_mfma_workspace(dp, cin, cout);
        float* dense_dw = reinterpret_cast<float*>(static_cast<char*>(ws) + slots);
        e = launch_dense_wgrad_mfma(dp, dtype, x, dy, n, cin, h, w, cout, dp.KS > 1 ? static_cast<float*>(ws) : dense_dw,
                                    stream);
        if (e == hipSuccess && dp.KS > 1) {
            const int64_t ne = int64_t(cout) * cin * 9;
            const int64_t gb = (ne + 255) / 256;
            hipLaunchKernelGGL(k_wgrad_reduce, dim3(unsigned(gb > 8192 ? 8192 : gb)), dim3(256), 0, stream,
                               static_cast<const float*>(ws), dp.KS, ne, dense_dw);
            e = hipGetLastError();
        }
        if (e == hipSuccess) e = launch_gather_masked(tab, pk, cout, cin, dense_dw, dv, stream);
        const size_t via = slots + size_t(cout) * size_t(cin) * 9 * sizeof(float);
        part_bytes = via > part_bytes ? via : part_bytes;
    } else {
        e = dtype == DT_F16 ? run<DT_F16, 4>(g, x, dy, pk.filter_perm, pk.seg_ptr, pk.cin_idx, dv, ws, stream)
                            : run<DT_F32, 4>(g, x, dy, pk.filter_perm, pk.seg_ptr, pk.cin_idx, dv, ws, stream);
    }
    if (e != hipSuccess || !db) return e;
    float* bpart = ws ? reinterpret_cast<float*>(static_cast<char*>(ws) + part_bytes) : nullptr;
    return dtype == DT_F16 ? bias_grad<DT_F16>(dy, n, cout, h * w, db, bpart, stream)
                           : bias_grad<DT_F32>(dy, n, cout, h * w, db, bpart, stream);
}

hipError_t launch_dense_wgrad(const float* x, const float* g_, int n, int cin, int h, int w, int cout, float* dw,
                              float* db, void* ws, hipStream_t stream) {
    hipError_t e;
    size_t part_bytes;
    DenseWPlan dp;
    if (dense_wgrad_mfma_plan(n, cin, cout, h, w, &dp)) {
        // matrix cores: KS slots of partial sums, added in slot order
        part_bytes = dense_wgrad_mfma_workspace(dp, cin, cout);
        e = launch_dense_wgrad_mfma(dp, DT_F32, x, g_, n, cin, h, w, cout, dp.KS > 1 ? static_cast<float*>(ws) : dw,
                                    stream);
        if (e == hipSuccess && dp.KS > 1) {
            const int64_t ne = int64_t(cout) * cin * 9;
            const int64_t gb = (ne + 255) / 256;
            hipLaunchKernelGGL(k_wgrad_reduce, dim3(unsigned(gb > 8192 ? 8192 : gb)), dim3(256), 0, stream,
                               static_cast<const float*>(ws), dp.KS, ne, dw);
            e = hipGetLastError();
        }
    } else {
        const WGeo g = plan(n, cin, cout, h, w, int64_t(cout) * cin, true, nullptr, DT_F32);
        part_bytes = wgrad_part_bytes(g, int64_t(cout) * cin, true);
        e = run<DT_F32, 9>(g, x, g_, nullptr, nullptr, nullptr, dw, ws, stream);
    }
    if (e != hipSuccess || !db) return e;
    float* bpart = ws ? reinterpret_cast<float*>(static_cast<char*>(ws) + part_bytes) : nullptr;
    return bias_grad<DT_F32>(g_, n, cout, h * w, db, bpart, stream);
}

}  // namespace psc
