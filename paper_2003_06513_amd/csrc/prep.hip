// Offline preparation kernels: pattern projection (Sec. 4.3, Eq. 6),
// connectivity pruning (Sec. 4.4), filter kernel reorder + compressed weight
// storage (Sec. 3.4) and the dense unpacker.  All results are integer or bit
// copies except the fp64 energies, which are sums of exact squares added in a
// fixed order, so every output is bit-exact and run-to-run deterministic.
#include <mutex>

#include "common.h"
#include "launch.h"

// Products of fp32 values are exact in fp64, so contraction could not change
// a result here; keep it off anyway so each add is a plain rounded add.
#pragma clang fp contract(off)

namespace psc {
namespace {

// ---------------------------------------------------------------- projection
constexpr int kProjBlock = 256;

template <int DT>
__global__ __launch_bounds__(kProjBlock) void k_project(const typename Elt<DT>::T* __restrict__ w,
                                                       int64_t n_kernels, PatTable tab,
                                                       uint8_t* __restrict__ pat,
                                                       double* __restrict__ energy) {
    __shared__ float tile[kProjBlock * 9];
    const int64_t k0 = int64_t(blockIdx.x) * kProjBlock;
    const int nk = int(min<int64_t>(kProjBlock, n_kernels - k0));
    // coalesced staging of the block's nk*9 contiguous weights
    for (int i = threadIdx.x; i < nk * 9; i += kProjBlock) tile[i] = Elt<DT>::load(w + k0 * 9, i);
    __syncthreads();
    const int t = threadIdx.x;
    if (t >= nk) return;
    double sq[9];
#pragma unroll
    for (int q = 0; q < 9; ++q) {
        const double v = double(tile[t * 9 + q]);  // stride 9: conflict-free
        sq[q] = v * v;
    }
    int best_p = 0;
    double best_e = 0.0;
    for (int p = 0; p < tab.m; ++p) {
        const unsigned mk = tab.mask[p];
        double e = 0.0;
#pragma unroll
        for (int q = 0; q < 9; ++q)
            if ((mk >> q) & 1u) e = e + sq[q];
        if (p == 0 || e > best_e) {
            best_e = e;
            best_p = p;
        }
    }
    pat[k0 + t] = uint8_t(best_p);
    energy[k0 + t] = best_e;
}

// ---------------------------------------------------------------- top-beta
// Radix select over the uint64 images of the non-negative fp64 energies
// (order-preserving), 8 bits per pass from the top, then an index-ordered
// rank of the keys equal to the threshold.
struct SelState {
    uint64_t prefix;     // digits of the threshold found so far
    uint64_t mask;       // which bits of prefix are decided
    int64_t remaining;   // kernels still to keep among keys matching prefix
    int64_t pad;
};
constexpr int kSelChunk = 1024;     // keys per block in count/mark
constexpr size_t kSelHistOff = 0;   // 256 x u32
constexpr size_t kSelStateOff = 1024;
constexpr size_t kSelCountOff = 1280;

// The digit of one radix pass, by threads 0..255 of the block (every thread
// of the block calls it): with S(d) the number of candidate keys whose digit
// is d or more, the digit is the largest d >= 1 with S(d) >= r (r = kernels
// still to keep), else 0 -- the first digit from the top at which the
// running count reaches r -- and S(d + 1) keys rank above it.  Suffix sums
// in LDS instead of a serial walk over the 256 bins.  Returns the digit and
// sets *above (both valid in every thread).
__device__ __forceinline__ int sel_digit(const uint32_t* hist, int64_t r, uint64_t* sfx, int* s_d, int64_t* above) {
    const int t = threadIdx.x;
    if (t < 256) sfx[t] = hist[t];
    if (t == 0) {
        sfx[256] = 0;
        *s_d = 0;
    }
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint64_t v = t < 256 && t + off < 256 ? sfx[t + off] : 0u;
        __syncthreads();
        if (t < 256) sfx[t] += v;
        __syncthreads();
    }
    if (t >= 1 && t < 256 && int64_t(sfx[t]) >= r) atomicMax(s_d, t);
    __syncthreads();
    const int d = *s_d;
    *above = int64_t(sfx[d + 1]);
    return d;
}

__global__ __launch_bounds__(256) void k_sel_init(uint32_t* __restrict__ hist, SelState* __restrict__ st,
                                                  int64_t keep) {
    hist[threadIdx.x] = 0;
    if (threadIdx.x == 0) {
        st->prefix = 0;
        st->mask = 0;
        st->remaining = keep;
        st->pad = 0;
    }
}

__global__ __launch_bounds__(256) void k_sel_hist(const uint64_t* __restrict__ keys, int64_t n,
                                                  int shift, const SelState* __restrict__ st,
                                                  uint32_t* __restrict__ hist) {
    __shared__ uint32_t lh[256];
    lh[threadIdx.x] = 0;
    __syncthreads();
    const uint64_t prefix = st->prefix, mask = st->mask;
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
        const uint64_t key = keys[i];
        if ((key & mask) == prefix) atomicAdd(&lh[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    const uint32_t c = lh[threadIdx.x];
    if (c) atomicAdd(&hist[threadIdx.x], c);
}

__global__ __launch_bounds__(256) void k_sel_pick(uint32_t* __restrict__ hist, SelState* __restrict__ st,
                                                  int shift) {
    __shared__ uint64_t sfx[257];
    __shared__ int s_d;
    const int64_t r = st->remaining;
    int64_t above;
    const int d = sel_digit(hist, r, sfx, &s_d, &above);
    if (threadIdx.x == 0) {
        st->remaining = r - above;
        st->prefix |= uint64_t(d) << shift;
        st->mask |= uint64_t(255) << shift;
    }
    hist[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void k_sel_count(const uint64_t* __restrict__ keys, int64_t n,
                                                   const SelState* __restrict__ st,
                                                   uint32_t* __restrict__ blk) {
    __shared__ uint32_t red[256];
    const uint64_t T = st->prefix;
    const int64_t base = int64_t(blockIdx.x) * kSelChunk + threadIdx.x * 4;
    uint32_t c = 0;
    for (int j = 0; j < 4; ++j) {
        const int64_t i = base + j;
        if (i < n && keys[i] == T) ++c;
    }
    red[threadIdx.x] = c;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) blk[blockIdx.x] = red[0];
}

// In-place exclusive scan of n u32 values with one block of 1024 threads,
// each owning a contiguous run (so the result is in index order).
__global__ __launch_bounds__(1024) void k_scan_excl_u32(uint32_t* __restrict__ a, int64_t n) {
    __shared__ uint32_t part[1024];
    const int t = threadIdx.x;
    const int64_t per = (n + 1023) / 1024;
    const int64_t beg = min<int64_t>(n, t * per), end = min<int64_t>(n, beg + per);
    uint32_t s = 0;
    for (int64_t i = beg; i < end; ++i) s += a[i];
    part[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const uint32_t v = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    uint32_t run = part[t] - s;
    for (int64_t i = beg; i < end; ++i) {
        const uint32_t v = a[i];
        a[i] = run;
        run += v;
    }
}

__global__ __launch_bounds__(256) void k_sel_mark(const uint64_t* __restrict__ keys, int64_t n,
                                                  const SelState* __restrict__ st,
                                                  const uint32_t* __restrict__ blk_off,
                                                  uint8_t* __restrict__ keep) {
    __shared__ uint32_t part[256];
    const uint64_t T = st->prefix;
    const int64_t r = st->remaining;
    const int t = threadIdx.x;
    const int64_t base = int64_t(blockIdx.x) * kSelChunk + t * 4;
    uint64_t kv[4];
    uint32_t c = 0;
    for (int j = 0; j < 4; ++j) {
        const int64_t i = base + j;
        kv[j] = i < n ? keys[i] : 0;
        if (i < n && kv[j] == T) ++c;
    }
    part[t] = c;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint32_t v = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    int64_t rank = int64_t(blk_off[blockIdx.x]) + (part[t] - c);
    for (int j = 0; j < 4; ++j) {
        const int64_t i = base + j;
        if (i >= n) break;
        uint8_t v = 0;
        if (kv[j] > T) {
            v = 1;
        } else if (kv[j] == T) {
            v = rank < r ? 1 : 0;
            ++rank;
        }
        keep[i] = v;
    }
}

// The whole selection in one workgroup of 1024 threads, for layers of at
// most kSelOneBlockMax kernels, where the passes above would be bound by
// their 19 launches: the same 8 radix passes (histogram of the keys that
// match the digits found so far, then the same digit), then the same
// index-ordered rank of the keys equal to the threshold
// -- each thread owns a contiguous run of indices -- so the keep mask is the
// same bit for bit.
constexpr int64_t kSelOneBlockMax = 65536;

__global__ __launch_bounds__(1024) void k_sel_one(const uint64_t* __restrict__ keys, int64_t n, int64_t keep,
                                                  uint8_t* __restrict__ out) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t part[1024];
    __shared__ uint64_t sfx[257];
    __shared__ uint64_t s_prefix, s_mask;
    __shared__ int64_t s_rem;
    __shared__ int s_d;
    const int t = threadIdx.x;
    if (t == 0) {
        s_prefix = 0;
        s_mask = 0;
        s_rem = keep;
    }
    for (int shift = 56; shift >= 0; shift -= 8) {
        if (t < 256) hist[t] = 0;
        __syncthreads();
        const uint64_t prefix = s_prefix, mask = s_mask;
        for (int64_t i = t; i < n; i += 1024) {
            const uint64_t key = keys[i];
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        const int64_t r = s_rem;
        int64_t above;
        const int d = sel_digit(hist, r, sfx, &s_d, &above);
        __syncthreads();   // every thread has read s_rem, s_d and sfx
        if (t == 0) {
            s_rem = r - above;
            s_prefix = prefix | (uint64_t(d) << shift);
            s_mask = mask | (uint64_t(255) << shift);
        }
        __syncthreads();
    }
    const uint64_t T = s_prefix;
    const int64_t r = s_rem;
    const int64_t per = (n + 1023) / 1024;
    const int64_t beg = min<int64_t>(n, t * per), end = min<int64_t>(n, beg + per);
    uint32_t c = 0;
    for (int64_t i = beg; i < end; ++i) c += keys[i] == T ? 1u : 0u;
    part[t] = c;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const uint32_t v = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    int64_t rank = int64_t(part[t] - c);
    for (int64_t i = beg; i < end; ++i) {
        const uint64_t key = keys[i];
        uint8_t v = 0;
        if (key > T) {
            v = 1;
        } else if (key == T) {
            v = rank < r ? 1 : 0;
            ++rank;
        }
        out[i] = v;
    }
}

__global__ __launch_bounds__(256) void k_fill_u8(uint8_t* __restrict__ p, int64_t n, uint8_t v) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) p[i] = v;
}

// ---------------------------------------------------------------- packing
// Per filter: kept count and per-pattern counts.  One wave per filter.
__global__ __launch_bounds__(64) void k_pack_count(const uint8_t* __restrict__ pat,
                                                   const uint8_t* __restrict__ keep, int cin, int m,
                                                   int32_t* __restrict__ cnt, int32_t* __restrict__ nf) {
    __shared__ int32_t c_s[kMaxPatterns];
    const int f = blockIdx.x, lane = threadIdx.x;
    for (int p = lane; p < m; p += 64) c_s[p] = 0;
    __syncthreads();
    int n = 0;
    for (int c0 = 0; c0 < cin; c0 += 64) {
        const int ci = c0 + lane;
        bool kept = false;
        int pp = 0;
        if (ci < cin) {
            const int64_t k = int64_t(f) * cin + ci;
            kept = keep[k] != 0;
            pp = pat[k];
        }
        n += __popcll(__ballot(kept));
        if (kept && pp < m) atomicAdd(&c_s[pp], 1);
    }
    __syncthreads();
    for (int p = lane; p < m; p += 64) cnt[int64_t(f) * m + p] = c_s[p];
    if (lane == 0) nf[f] = n;
}

// Rank of each filter under (count desc, per-pattern counts lexicographically
// desc, index asc); the key is a total order, so ranks form a permutation.
// One block per filter f: its threads compare f with every other filter g
// (g = t, t + 256, ...) and the block adds up how many come first.
__global__ __launch_bounds__(256) void k_pack_rank(const int32_t* __restrict__ cnt,
                                                   const int32_t* __restrict__ nf, int cout, int m,
                                                   int32_t* __restrict__ perm,
                                                   int32_t* __restrict__ nf_sorted) {
    __shared__ int part[4];
    const int f = blockIdx.x;
    const int nff = nf[f];
    const int32_t* cf = cnt + int64_t(f) * m;
    int rank = 0;
    for (int g = threadIdx.x; g < cout; g += 256) {
        if (g == f) continue;
        const int ng = nf[g];
        bool before;
        if (ng != nff) {
            before = ng > nff;
        } else {
            before = g < f;
            const int32_t* cg = cnt + int64_t(g) * m;
            for (int p = 0; p < m; ++p) {
                if (cg[p] != cf[p]) {
                    before = cg[p] > cf[p];
                    break;
                }
            }
        }
        rank += before ? 1 : 0;
    }
    for (int off = 32; off > 0; off >>= 1) rank += __shfl_xor(rank, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = rank;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int r = part[0] + part[1] + part[2] + part[3];
        perm[r] = f;
        nf_sorted[r] = nff;
    }
}

// out[0..n] = exclusive prefix sums of in[0..n-1], out[n] = total.
__global__ __launch_bounds__(1024) void k_scan_excl_i32(const int32_t* __restrict__ in,
                                                        int32_t* __restrict__ out, int n) {
    __shared__ int32_t part[1024];
    const int t = threadIdx.x;
    const int per = (n + 1023) / 1024;
    const int beg = min(n, t * per), end = min(n, beg + per);
    int32_t s = 0;
    for (int i = beg; i < end; ++i) s += in[i];
    part[t] = s;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int32_t v = t >= off ? part[t - off] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    int32_t run = part[t] - s;
    for (int i = beg; i < end; ++i) {
        out[i] = run;
        run += in[i];
    }
    if (t == 1023) out[n] = part[1023];
}

__global__ __launch_bounds__(256) void k_pack_seg(const int32_t* __restrict__ cnt,
                                                  const int32_t* __restrict__ perm,
                                                  const int32_t* __restrict__ fptr, int cout, int m,
                                                  int32_t* __restrict__ seg) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= cout) return;
    const int f = perm[i];
    int32_t s = fptr[i];
    for (int p = 0; p < m; ++p) {
        seg[int64_t(i) * (m + 1) + p] = s;
        s += cnt[int64_t(f) * m + p];
    }
    seg[int64_t(i) * (m + 1) + m] = fptr[i + 1];
}

// Scatter of one reordered filter per wave: a kernel's slot is the start of
// its pattern's segment + kept kernels of that pattern at lower ci.
template <typename B>
__global__ __launch_bounds__(64) void k_pack_scatter(const B* __restrict__ w,
                                                     const uint8_t* __restrict__ pat,
                                                     const uint8_t* __restrict__ keep, int cin,
                                                     int64_t n_keep, PatTable tab, const int32_t* __restrict__ perm,
                                                     const int32_t* __restrict__ seg,
                                                     int32_t* __restrict__ cin_idx,
                                                     uint8_t* __restrict__ pat_id,
                                                     B* __restrict__ values) {
    __shared__ int32_t cur[kMaxPatterns];
    __shared__ uint16_t msk[kMaxPatterns];
    const int i = blockIdx.x, lane = threadIdx.x, m = tab.m;
    const int f = perm[i];
    for (int p = lane; p < m; p += 64) {
        cur[p] = seg[int64_t(i) * (m + 1) + p];
        msk[p] = tab.mask[p];
    }
    __syncthreads();
    for (int c0 = 0; c0 < cin; c0 += 64) {
        const int ci = c0 + lane;
        bool kept = false;
        int pp = 0;
        const int64_t k = int64_t(f) * cin + ci;
        if (ci < cin) {
            kept = keep[k] != 0;
            pp = pat[k];
        }
        int pos = -1;
        for (int p = 0; p < m; ++p) {
            const bool mine = kept && pp == p;
            const uint64_t b = __ballot(mine);
            if (b == 0) continue;
            if (mine) pos = cur[p] + __popcll(b & ((uint64_t(1) << lane) - 1));
            __syncthreads();
            if (lane == 0) cur[p] += __popcll(b);
            __syncthreads();
        }
        if (kept && pos >= 0 && pos < n_keep) {   // a keep mask with too many ones writes nothing past the arrays
            cin_idx[pos] = ci;
            pat_id[pos] = uint8_t(pp);
            const unsigned mk = msk[pp];
            int j = 0;
            for (int q = 0; q < 9; ++q)
                if ((mk >> q) & 1u) values[int64_t(pos) * 4 + j++] = w[k * 9 + q];
        }
    }
}

template <typename B>
__global__ __launch_bounds__(256) void k_fill_zero(B* __restrict__ p, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) p[i] = 0;
}

template <typename B>
__global__ __launch_bounds__(256) void k_unpack(const int32_t* __restrict__ perm,
                                                const int32_t* __restrict__ fptr,
                                                const int32_t* __restrict__ cin_idx,
                                                const uint8_t* __restrict__ pat_id,
                                                const B* __restrict__ values, int cin, PatTable tab,
                                                B* __restrict__ dense) {
    __shared__ uint16_t msk[kMaxPatterns];
    for (int p = threadIdx.x; p < tab.m; p += 256) msk[p] = tab.mask[p];
    __syncthreads();
    const int i = blockIdx.x;
    const int f = perm[i];
    for (int k = fptr[i] + threadIdx.x; k < fptr[i + 1]; k += 256) {
        const int ci = cin_idx[k];
        const int p = pat_id[k];
        if (unsigned(ci) >= unsigned(cin) || p >= tab.m) continue;   // malformed storage
        const unsigned mk = msk[p];
        int j = 0;
        for (int q = 0; q < 9; ++q)
            if ((mk >> q) & 1u) dense[(int64_t(f) * cin + ci) * 9 + q] = values[int64_t(k) * 4 + j++];
    }
}

int grid_for(int64_t n, int per_block, int cap) {
    const int64_t g = (n + per_block - 1) / per_block;
    return int(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_project(const PatTable& tab, int dtype, const void* w, int64_t n_kernels,
                          uint8_t* pat, double* energy, hipStream_t stream) {
    if (n_kernels == 0) return hipSuccess;
    const dim3 grid(unsigned((n_kernels + kProjBlock - 1) / kProjBlock));
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_project<DT_F16>, grid, dim3(kProjBlock), 0, stream,
                           static_cast<const uint16_t*>(w), n_kernels, tab, pat, energy);
    else
        hipLaunchKernelGGL(k_project<DT_F32>, grid, dim3(kProjBlock), 0, stream,
                           static_cast<const float*>(w), n_kernels, tab, pat, energy);
    return hipGetLastError();
}

size_t select_workspace_bytes(int64_t n_kernels) {
    const int64_t nblk = (n_kernels + kSelChunk - 1) / kSelChunk;
    const size_t b = kSelCountOff + size_t(nblk) * 4;
    return (b + 255) / 256 * 256;
}

hipError_t launch_select(int64_t n, int64_t keep, const double* energy, uint8_t* keep_out, void* ws,
                         hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (keep == 0 || keep == n) {
        hipLaunchKernelGGL(k_fill_u8, dim3(grid_for(n, 256, 4096)), dim3(256), 0, stream, keep_out, n,
                           uint8_t(keep == n ? 1 : 0));
        return hipGetLastError();
    }
    if (n <= kSelOneBlockMax) {
        hipLaunchKernelGGL(k_sel_one, dim3(1), dim3(1024), 0, stream, reinterpret_cast<const uint64_t*>(energy), n,
                           keep, keep_out);
        return hipGetLastError();
    }
    char* base = static_cast<char*>(ws);
    uint32_t* hist = reinterpret_cast<uint32_t*>(base + kSelHistOff);
    SelState* st = reinterpret_cast<SelState*>(base + kSelStateOff);
    uint32_t* blk = reinterpret_cast<uint32_t*>(base + kSelCountOff);
    const uint64_t* keys = reinterpret_cast<const uint64_t*>(energy);
    const int nblk = int((n + kSelChunk - 1) / kSelChunk);
    hipLaunchKernelGGL(k_sel_init, dim3(1), dim3(256), 0, stream, hist, st, keep);
    const int hg = grid_for(n, 256, 2048);
    for (int pass = 7; pass >= 0; --pass) {
        hipLaunchKernelGGL(k_sel_hist, dim3(hg), dim3(256), 0, stream, keys, n, pass * 8, st, hist);
        hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(256), 0, stream, hist, st, pass * 8);
    }
    hipLaunchKernelGGL(k_sel_count, dim3(nblk), dim3(256), 0, stream, keys, n, st, blk);
    hipLaunchKernelGGL(k_scan_excl_u32, dim3(1), dim3(1024), 0, stream, blk, int64_t(nblk));
    hipLaunchKernelGGL(k_sel_mark, dim3(nblk), dim3(256), 0, stream, keys, n, st, blk, keep_out);
    return hipGetLastError();
}

// ---------------------------------------------------------------- static scratch
// The select workspace of the entry point that allocates nothing: one array
// in the library's device code.  Each GPU holds its own copy at its own
// address; in host code the array's name is only a stand-in, so kernels get
// the address hipGetSymbolAddress reports for the current device.
constexpr size_t kSelScratchBytes = 64 * 1024;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint8_t scratch[kSelScratchBytes];

size_t select_scratch_bytes() { return kSelScratchBytes; }

hipError_t select_scratch(void** out) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // with this device current
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

// Pack workspace: cnt[cout*m] | nf[cout] | nf_sorted[cout], each 256-aligned.
size_t pack_workspace_bytes(int cout, int m) {
    auto al = [](size_t b) { return (b + 255) / 256 * 256; };
    return al(size_t(cout) * m * 4) + al(size_t(cout) * 4) + al(size_t(cout) * 4);
}

hipError_t launch_pack(const PatTable& tab, int dtype, int cout, int cin, int64_t n_keep, const void* w,
                       const uint8_t* pat, const uint8_t* keep, const PackedOut& out, void* ws,
                       hipStream_t stream) {
    auto al = [](size_t b) { return (b + 255) / 256 * 256; };
    char* base = static_cast<char*>(ws);
    int32_t* cnt = reinterpret_cast<int32_t*>(base);
    int32_t* nf = reinterpret_cast<int32_t*>(base + al(size_t(cout) * tab.m * 4));
    int32_t* nfs = reinterpret_cast<int32_t*>(base + al(size_t(cout) * tab.m * 4) + al(size_t(cout) * 4));
    const int m = tab.m;
    const unsigned g256 = unsigned((cout + 255) / 256);
    hipLaunchKernelGGL(k_pack_count, dim3(cout), dim3(64), 0, stream, pat, keep, cin, m, cnt, nf);
    hipLaunchKernelGGL(k_pack_rank, dim3(unsigned(cout)), dim3(256), 0, stream, cnt, nf, cout, m,
                       out.filter_perm, nfs);
    hipLaunchKernelGGL(k_scan_excl_i32, dim3(1), dim3(1024), 0, stream, nfs, out.filter_ptr, cout);
    hipLaunchKernelGGL(k_pack_seg, dim3(g256), dim3(256), 0, stream, cnt, out.filter_perm,
                       out.filter_ptr, cout, m, out.seg_ptr);
    if (dtype == DT_F16)
        hipLaunchKernelGGL(k_pack_scatter<uint16_t>, dim3(cout), dim3(64), 0, stream,
                           static_cast<const uint16_t*>(w), pat, keep, cin, n_keep, tab, out.filter_perm,
                           out.seg_ptr, out.cin_idx, out.pat_id, static_cast<uint16_t*>(out.values));
    else
        hipLaunchKernelGGL(k_pack_scatter<uint32_t>, dim3(cout), dim3(64), 0, stream,
                           static_cast<const uint32_t*>(w), pat, keep, cin, n_keep, tab, out.filter_perm,
                           out.seg_ptr, out.cin_idx, out.pat_id, static_cast<uint32_t*>(out.values));
    return hipGetLastError();
}

hipError_t launch_unpack(const PatTable& tab, int dtype, int cout, int cin, int64_t keep,
                         const PackedView& pk, void* dense, hipStream_t stream) {
    const int64_t total = int64_t(cout) * cin * 9;
    if (dtype == DT_F16) {
        hipLaunchKernelGGL(k_fill_zero<uint16_t>, dim3(grid_for(total, 256, 4096)), dim3(256), 0, stream,
                           static_cast<uint16_t*>(dense), total);
        if (keep > 0)
            hipLaunchKernelGGL(k_unpack<uint16_t>, dim3(cout), dim3(256), 0, stream, pk.filter_perm,
                               pk.filter_ptr, pk.cin_idx, pk.pat_id,
                               static_cast<const uint16_t*>(pk.values), cin, tab,
                               static_cast<uint16_t*>(dense));
    } else {
        hipLaunchKernelGGL(k_fill_zero<uint32_t>, dim3(grid_for(total, 256, 4096)), dim3(256), 0, stream,
                           static_cast<uint32_t*>(dense), total);
        if (keep > 0)
            hipLaunchKernelGGL(k_unpack<uint32_t>, dim3(cout), dim3(256), 0, stream, pk.filter_perm,
                               pk.filter_ptr, pk.cin_idx, pk.pat_id,
                               static_cast<const uint32_t*>(pk.values), cin, tab,
                               static_cast<uint32_t*>(dense));
    }
    return hipGetLastError();
}

}  // namespace psc
