// C ABI of the pattern-sparse 3x3 convolution library: argument validation,
// error reporting, the host-side pattern-library heuristic and dispatch to
// the HIP launchers.  Every check runs before the first HIP call.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "../../include/psc.h"
#include "common.h"
#include "launch.h"

namespace {

thread_local std::string g_last_error;

psc_status fail(psc_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

psc_status ok() {
    g_last_error.clear();
    return PSC_OK;
}

psc_status device_status(hipError_t e, const char* what) {
    if (e != hipSuccess)
        return fail(PSC_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

int popcount9(unsigned v) {
    int c = 0;
    for (int b = 0; b < 9; ++b) c += (v >> b) & 1u;
    return c;
}

size_t elt_size(int dtype) { return dtype == PSC_F16 ? 2 : 4; }

bool dtype_ok(int32_t d) { return d == PSC_F32 || d == PSC_F16; }

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

// Layer checks shared by every entry point that takes a psc_layer.
psc_status check_layer(const psc_layer* L, bool need_keep) {
    if (!L) return fail(PSC_ERR_ARG, "layer is NULL");
    if (L->cout < 1 || L->cout > 65535)
        return fail(PSC_ERR_ARG, "cout=%d outside 1..65535", L->cout);
    if (L->cin < 1 || L->cin > (1 << 24))
        return fail(PSC_ERR_ARG, "cin=%d outside 1..2^24", L->cin);
    const int64_t K = int64_t(L->cout) * L->cin;
    if (K * 9 > kMaxElems)
        return fail(PSC_ERR_ARG, "cout*cin*9=%lld exceeds 2^31-1", (long long)(K * 9));
    if (L->m < 1 || L->m > PSC_MAX_PATTERNS)
        return fail(PSC_ERR_ARG, "m=%d outside 1..%d", L->m, PSC_MAX_PATTERNS);
    if (!dtype_ok(L->wdtype)) return fail(PSC_ERR_ARG, "wdtype=%d is not a psc_dtype", L->wdtype);
    for (int p = 0; p < L->m; ++p) {
        const unsigned c = L->masks[p];
        if (c >= 512 || popcount9(c) != 4)
            return fail(PSC_ERR_ARG, "masks[%d]=0x%x is not a 9-bit code with 4 bits set", p, c);
        for (int q = 0; q < p; ++q)
            if (L->masks[q] == c)
                return fail(PSC_ERR_ARG, "masks[%d] duplicates masks[%d] (0x%x)", p, q, c);
    }
    if (need_keep && (L->keep < 0 || L->keep > K))
        return fail(PSC_ERR_ARG, "keep=%lld outside 0..cout*cin=%lld", (long long)L->keep,
                    (long long)K);
    return PSC_OK;
}

psc::PatTable table_of(const psc_layer* L) {
    psc::PatTable t;
    std::memset(&t, 0, sizeof t);
    t.m = L->m;
    for (int p = 0; p < L->m; ++p) t.mask[p] = L->masks[p];
    return t;
}

psc_status check_packed(const psc_layer* L, const psc_packed* pk) {
    if (!pk) return fail(PSC_ERR_ARG, "packed is NULL");
    if (!pk->filter_perm || !pk->filter_ptr || !pk->seg_ptr)
        return fail(PSC_ERR_ARG, "packed filter_perm/filter_ptr/seg_ptr must be non-NULL");
    if (L->keep > 0 && (!pk->cin_idx || !pk->pat_id || !pk->values))
        return fail(PSC_ERR_ARG, "packed cin_idx/pat_id/values must be non-NULL when keep > 0");
    if (pk->values && (reinterpret_cast<uintptr_t>(pk->values) & 15u))
        return fail(PSC_ERR_ARG, "packed values must be 16-byte aligned");
    return PSC_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return na && nb && pa < pb + nb && pb < pa + na;
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

const char* psc_last_error(void) { return g_last_error.c_str(); }

const char* psc_status_string(psc_status s) {
    // a C caller may pass any int: read the bits as one, not as the enum
    // (whose value range ends at 7)
    int32_t v;
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
        case PSC_OK: return "PSC_OK";
        case PSC_ERR_ARG: return "PSC_ERR_ARG";
        case PSC_ERR_UNSUPPORTED: return "PSC_ERR_UNSUPPORTED";
        case PSC_ERR_WORKSPACE: return "PSC_ERR_WORKSPACE";
        case PSC_ERR_DEVICE: return "PSC_ERR_DEVICE";
        case PSC_ERR_INTERNAL: return "PSC_ERR_INTERNAL";
    }
    return "PSC_UNKNOWN_STATUS";
}

int32_t psc_abi_version(void) { return 1; }

// Sec. 4.2.  Host only.  Magnitudes are compared as floats (fp16 widens
// exactly), so fp16 and fp32 copies of the same values give the same library.
psc_status psc_select_library(const void* h_w, int32_t dtype, int64_t n_kernels, int32_t m,
                              uint16_t* h_masks_out) {
    if (!dtype_ok(dtype)) return fail(PSC_ERR_ARG, "dtype=%d is not a psc_dtype", dtype);
    if (m < 1 || m > PSC_MAX_LIBRARY_HEURISTIC)
        return fail(PSC_ERR_ARG, "m=%d outside 1..%d", m, PSC_MAX_LIBRARY_HEURISTIC);
    if (n_kernels < 0) return fail(PSC_ERR_ARG, "n_kernels=%lld < 0", (long long)n_kernels);
    if (n_kernels > 0 && !h_w) return fail(PSC_ERR_ARG, "h_w is NULL");
    if (!h_masks_out) return fail(PSC_ERR_ARG, "h_masks_out is NULL");

    int64_t hist[512];
    std::memset(hist, 0, sizeof hist);
    const float* wf = static_cast<const float*>(h_w);
    const uint16_t* wh = static_cast<const uint16_t*>(h_w);
    for (int64_t k = 0; k < n_kernels; ++k) {
        float a[9];
        for (int q = 0; q < 9; ++q) {
            float v;
            if (dtype == PSC_F16) {
                // binary16 -> binary32 by exponent rebias (exact)
                const uint32_t h = wh[k * 9 + q];
                const uint32_t s = (h & 0x8000u) << 16, e = (h >> 10) & 0x1f, f = h & 0x3ff;
                uint32_t bits;
                if (e == 0) {
                    if (f == 0) {
                        bits = s;
                    } else {  // subnormal: normalise
                        int sh = 0;
                        uint32_t ff = f;
                        while (!(ff & 0x400)) { ff <<= 1; ++sh; }
                        bits = s | uint32_t(127 - 15 + 1 - sh) << 23 | (ff & 0x3ff) << 13;
                    }
                } else if (e == 31) {
                    bits = s | 0x7f800000u | f << 13;
                } else {
                    bits = s | (e + 112) << 23 | f << 13;
                }
                std::memcpy(&v, &bits, 4);
            } else {
                v = wf[k * 9 + q];
            }
            a[q] = v < 0 ? -v : v;
        }
        // three passes of "largest remaining neighbour", first index on ties
        unsigned taken = 1u << 4;
        for (int t = 0; t < 3; ++t) {
            int arg = -1;
            for (int q = 0; q < 9; ++q) {
                if (taken >> q & 1u) continue;
                if (arg < 0 || a[q] > a[arg]) arg = q;
            }
            taken |= 1u << arg;
        }
        ++hist[taken];
    }
    // rank all 56 centre+3 codes by (count desc, code asc): insertion sort
    int codes[56];
    int nc = 0;
    for (int c = 0; c < 512; ++c)
        if ((c >> 4 & 1) && popcount9(unsigned(c)) == 4) {
            int j = nc++;
            while (j > 0 && (hist[codes[j - 1]] < hist[c])) {
                codes[j] = codes[j - 1];
                --j;
            }
            codes[j] = c;
        }
    for (int i = 0; i < m; ++i) h_masks_out[i] = uint16_t(codes[i]);
    return ok();
}

psc_status psc_workspace_size(const psc_layer* L, int32_t op, size_t* bytes) {
    if (psc_status s = check_layer(L, false)) return s;
    if (!bytes) return fail(PSC_ERR_ARG, "bytes is NULL");
    switch (op) {
        case PSC_OP_SELECT: *bytes = psc::select_workspace_bytes(int64_t(L->cout) * L->cin); break;
        case PSC_OP_PACK: *bytes = psc::pack_workspace_bytes(L->cout, L->m); break;
        default: return fail(PSC_ERR_ARG, "op=%d is not a psc_op", op);
    }
    return ok();
}

psc_status psc_project(const psc_layer* L, const void* d_w, uint8_t* d_pat, double* d_energy,
                       void* stream) {
    if (psc_status s = check_layer(L, false)) return s;
    if (!d_w || !d_pat || !d_energy) return fail(PSC_ERR_ARG, "d_w, d_pat and d_energy must be non-NULL");
    const psc::PatTable t = table_of(L);
    return device_status(psc::launch_project(t, L->wdtype, d_w, int64_t(L->cout) * L->cin, d_pat,
                                             d_energy, as_stream(stream)),
                         "psc_project launch");
}

psc_status psc_select(const psc_layer* L, const double* d_energy, uint8_t* d_keep, void* d_ws,
                      size_t ws_bytes, void* stream) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!d_energy || !d_keep) return fail(PSC_ERR_ARG, "d_energy and d_keep must be non-NULL");
    const int64_t K = int64_t(L->cout) * L->cin;
    const size_t need = psc::select_workspace_bytes(K);
    if (need && (!d_ws || ws_bytes < need))
        return fail(PSC_ERR_WORKSPACE, "select needs %zu workspace bytes, got %zu%s", need, ws_bytes,
                    d_ws ? "" : " (NULL)");
    if (d_ws && (reinterpret_cast<uintptr_t>(d_ws) & 255u))
        return fail(PSC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    return device_status(psc::launch_select(K, L->keep, d_energy, d_keep, d_ws, as_stream(stream)),
                         "psc_select launch");
}

psc_status psc_select_noalloc(const psc_layer* L, const double* d_energy, uint8_t* d_keep, void* stream) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!d_energy || !d_keep) return fail(PSC_ERR_ARG, "d_energy and d_keep must be non-NULL");
    const int64_t K = int64_t(L->cout) * L->cin;
    if (K > PSC_SELECT_NOALLOC_MAX_KERNELS)
        return fail(PSC_ERR_UNSUPPORTED, "psc_select_noalloc handles at most %d kernels (cout*cin=%lld); "
                    "use psc_select with a workspace", PSC_SELECT_NOALLOC_MAX_KERNELS, (long long)K);
    const size_t need = psc::select_workspace_bytes(K);
    if (need > psc::select_scratch_bytes())
        return fail(PSC_ERR_INTERNAL, "select scratch of %zu bytes is smaller than the %zu needed",
                    psc::select_scratch_bytes(), need);
    void* ws = nullptr;
    if (psc_status s = device_status(psc::select_scratch(&ws), "psc_select_noalloc scratch address")) return s;
    return device_status(psc::launch_select(K, L->keep, d_energy, d_keep, ws, as_stream(stream)),
                         "psc_select_noalloc launch");
}

psc_status psc_pack(const psc_layer* L, const void* d_w, const uint8_t* d_pat,
                    const uint8_t* d_keep, const psc_packed* out, void* d_ws, size_t ws_bytes,
                    void* stream) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!d_w || !d_pat || !d_keep) return fail(PSC_ERR_ARG, "d_w, d_pat and d_keep must be non-NULL");
    if (psc_status s = check_packed(L, out)) return s;
    const size_t need = psc::pack_workspace_bytes(L->cout, L->m);
    if (!d_ws || ws_bytes < need)
        return fail(PSC_ERR_WORKSPACE, "pack needs %zu workspace bytes, got %zu%s", need, ws_bytes,
                    d_ws ? "" : " (NULL)");
    if (reinterpret_cast<uintptr_t>(d_ws) & 255u)
        return fail(PSC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    const psc::PatTable t = table_of(L);
    const psc::PackedOut o{out->filter_perm, out->filter_ptr, out->seg_ptr,
                           out->cin_idx,     out->pat_id,     out->values};
    return device_status(psc::launch_pack(t, L->wdtype, L->cout, L->cin, L->keep, d_w, d_pat, d_keep, o,
                                          d_ws, as_stream(stream)),
                         "psc_pack launch");
}

psc_status psc_unpack_dense(const psc_layer* L, const psc_packed* pk, void* d_w_dense,
                            void* stream) {
    if (psc_status s = check_layer(L, true)) return s;
    if (psc_status s = check_packed(L, pk)) return s;
    if (!d_w_dense) return fail(PSC_ERR_ARG, "d_w_dense is NULL");
    const psc::PatTable t = table_of(L);
    const psc::PackedView v{pk->filter_perm, pk->filter_ptr, pk->seg_ptr,
                            pk->cin_idx,     pk->pat_id,     pk->values};
    return device_status(psc::launch_unpack(t, L->wdtype, L->cout, L->cin, L->keep, v, d_w_dense,
                                            as_stream(stream)),
                         "psc_unpack_dense launch");
}

// Shape checks of every conv entry point (no pointers involved).
static psc_status check_conv_shape(const psc_layer* L, int32_t act_dtype, int32_t n, int32_t h, int32_t w,
                                   int32_t algo, int pool, int32_t stride) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!dtype_ok(act_dtype)) return fail(PSC_ERR_ARG, "act_dtype=%d is not a psc_dtype", act_dtype);
    if (act_dtype != L->wdtype)
        return fail(PSC_ERR_UNSUPPORTED, "act_dtype=%d differs from wdtype=%d", act_dtype, L->wdtype);
    if (n < 0 || n > 65535) return fail(PSC_ERR_ARG, "n=%d outside 0..65535", n);
    if (h < 1 || w < 1 || h > 32768 || w > 32768)
        return fail(PSC_ERR_ARG, "h=%d, w=%d outside 1..32768", h, w);
    if (algo < 0 || algo > 3) return fail(PSC_ERR_ARG, "algo=%d is not 0, 1, 2 or 3", algo);
    if (pool && ((h & 1) || (w & 1))) return fail(PSC_ERR_ARG, "h=%d, w=%d must be even for the 2x2 pool", h, w);
    if (stride != 1 && stride != 2) return fail(PSC_ERR_ARG, "stride=%d is not 1 or 2", stride);
    const int64_t plane = int64_t(h) * w;
    const int64_t oplane = pool ? plane / 4 : int64_t((h - 1) / stride + 1) * ((w - 1) / stride + 1);
    const int64_t xe = int64_t(n) * L->cin * plane, ye = int64_t(n) * L->cout * oplane;
    if (xe > kMaxElems || ye > kMaxElems)
        return fail(PSC_ERR_ARG, "x or y holds more than 2^31-1 elements");
    if (pool && stride != 1) return fail(PSC_ERR_ARG, "the fused 2x2 pool needs stride 1");
    if (algo == 2) {
        const psc::ConvArgs a{act_dtype, n, L->cin, h, w, L->cout, L->keep, nullptr, nullptr, 0, nullptr, pool, stride};
        if (!psc::conv_rows_takes(table_of(L), a))
            return fail(PSC_ERR_UNSUPPORTED,
                        "algo 2 (one row per lane) needs no pool, at most 63 output rows and, with stride 1, "
                        "w in {4, 7, 8, 14, 16, 28} (fp16: w even or 7), with stride 2, w in {8, 16, 32}; "
                        "got h=%d, w=%d, stride=%d, pool=%d",
                        h, w, stride, pool);
    }
    return PSC_OK;
}

static psc::ConvArgs conv_args(const psc_layer* L, int32_t act_dtype, const void* d_x, int32_t n, int32_t h,
                               int32_t w, const void* d_bias, int32_t relu, void* d_y, int pool, int32_t stride) {
    return psc::ConvArgs{act_dtype, n, L->cin, h, w, L->cout, L->keep, d_x, d_bias, relu != 0, d_y, pool, stride};
}

static psc_status conv_common(const psc_layer* L, const psc_packed* pk, int32_t act_dtype, const void* d_x,
                              int32_t n, int32_t h, int32_t w, const void* d_bias, int32_t relu, void* d_y,
                              int32_t algo, int pool, int32_t stride, void* stream) {
    if (psc_status s = check_conv_shape(L, act_dtype, n, h, w, algo, pool, stride)) return s;
    if (psc_status s = check_packed(L, pk)) return s;
    const int64_t plane = int64_t(h) * w;
    const int64_t oplane = pool ? plane / 4 : int64_t((h - 1) / stride + 1) * ((w - 1) / stride + 1);
    const int64_t xe = int64_t(n) * L->cin * plane, ye = int64_t(n) * L->cout * oplane;
    if (n == 0) return ok();
    if (!d_x || !d_y) return fail(PSC_ERR_ARG, "d_x and d_y must be non-NULL");
    const size_t es = elt_size(act_dtype);
    if (overlaps(d_x, size_t(xe) * es, d_y, size_t(ye) * es))
        return fail(PSC_ERR_ARG, "d_y overlaps d_x");
    if ((reinterpret_cast<uintptr_t>(d_x) | reinterpret_cast<uintptr_t>(d_y)) & (es - 1))
        return fail(PSC_ERR_ARG, "d_x and d_y must be aligned to the element size");
    const psc::PatTable t = table_of(L);
    const psc::PackedView v{pk->filter_perm, pk->filter_ptr, pk->seg_ptr,
                            pk->cin_idx,     pk->pat_id,     pk->values};
    const psc::ConvArgs a = conv_args(L, act_dtype, d_x, n, h, w, d_bias, relu, d_y, pool, stride);
    return device_status(psc::launch_conv(t, v, a, algo, as_stream(stream)), "psc_conv3x3_fwd launch");
}

psc_status psc_conv3x3_config(const psc_layer* L, int32_t act_dtype, int32_t n, int32_t h, int32_t w,
                              int32_t pool, int32_t stride, int32_t algo, psc_conv_config* out) {
    if (psc_status s = check_conv_shape(L, act_dtype, n, h, w, algo, pool != 0, stride)) return s;
    if (!out) return fail(PSC_ERR_ARG, "out is NULL");
    const psc::PatTable t = table_of(L);
    const psc::ConvArgs a = conv_args(L, act_dtype, nullptr, n, h, w, nullptr, 0, nullptr, pool != 0, stride);
    psc::ConvForm f{};
    psc::describe_conv(t, a, algo, f);
    *out = psc_conv_config{f.kernel, f.staged, f.rows_per_lane, f.cols_per_lane, f.segments_per_wave,
                           f.column_tiles, f.shares, f.filters_per_block, f.blocks, f.threads_per_block};
    return ok();
}

psc_status psc_conv3x3_fwd_algo(const psc_layer* L, const psc_packed* pk, int32_t act_dtype,
                                const void* d_x, int32_t n, int32_t h, int32_t w,
                                const void* d_bias, int32_t relu, void* d_y, int32_t algo,
                                void* stream) {
    return conv_common(L, pk, act_dtype, d_x, n, h, w, d_bias, relu, d_y, algo, 0, 1, stream);
}

psc_status psc_conv3x3_fwd(const psc_layer* L, const psc_packed* pk, int32_t act_dtype,
                           const void* d_x, int32_t n, int32_t h, int32_t w, const void* d_bias,
                           int32_t relu, void* d_y, void* stream) {
    return conv_common(L, pk, act_dtype, d_x, n, h, w, d_bias, relu, d_y, 0, 0, 1, stream);
}

psc_status psc_conv3x3_fwd_pool2(const psc_layer* L, const psc_packed* pk, int32_t act_dtype,
                                 const void* d_x, int32_t n, int32_t h, int32_t w, const void* d_bias,
                                 int32_t relu, void* d_y, int32_t algo, void* stream) {
    return conv_common(L, pk, act_dtype, d_x, n, h, w, d_bias, relu, d_y, algo, 1, 1, stream);
}

psc_status psc_conv3x3_fwd_strided(const psc_layer* L, const psc_packed* pk, int32_t act_dtype,
                                   const void* d_x, int32_t n, int32_t h, int32_t w, const void* d_bias,
                                   int32_t relu, void* d_y, int32_t stride, int32_t algo, void* stream) {
    return conv_common(L, pk, act_dtype, d_x, n, h, w, d_bias, relu, d_y, algo, 0, stride, stream);
}

psc_status psc_transpose_layer(const psc_layer* L, psc_layer* out) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!out) return fail(PSC_ERR_ARG, "out is NULL");
    psc_layer t;
    std::memset(&t, 0, sizeof t);
    t.cout = L->cin;
    t.cin = L->cout;
    t.m = L->m;
    t.wdtype = L->wdtype;
    t.keep = L->keep;
    for (int p = 0; p < L->m; ++p) {
        unsigned r = 0;
        for (int q = 0; q < 9; ++q)
            if ((L->masks[p] >> q) & 1u) r |= 1u << (8 - q);   // rotated by 180 degrees
        t.masks[p] = uint16_t(r);
    }
    if (t.cout > 65535) return fail(PSC_ERR_UNSUPPORTED, "cin=%d: the transposed layer needs cin <= 65535", L->cin);
    *out = t;
    return ok();
}

psc_status psc_transpose_prep(const psc_layer* L, const void* d_w, const uint8_t* d_pat, const uint8_t* d_keep,
                              void* d_w_t, uint8_t* d_pat_t, uint8_t* d_keep_t, void* stream) {
    if (psc_status s = check_layer(L, true)) return s;
    if (!d_w || !d_pat || !d_keep || !d_w_t || !d_pat_t || !d_keep_t)
        return fail(PSC_ERR_ARG, "every pointer must be non-NULL");
    const size_t K = size_t(L->cout) * L->cin;
    if (overlaps(d_w, K * 9 * elt_size(L->wdtype), d_w_t, K * 9 * elt_size(L->wdtype)) ||
        overlaps(d_pat, K, d_pat_t, K) || overlaps(d_keep, K, d_keep_t, K))
        return fail(PSC_ERR_ARG, "outputs must not overlap inputs");
    return device_status(psc::launch_transpose_prep(L->wdtype, L->cout, L->cin, d_w, d_pat, d_keep, d_w_t, d_pat_t,
                                                    d_keep_t, as_stream(stream)),
                         "psc_transpose_prep launch");
}

psc_status psc_conv3x3_bwd_weight_workspace(const psc_layer* L, int32_t act_dtype, int32_t n, int32_t h, int32_t w,
                                            size_t* bytes) {
    if (psc_status s = check_conv_shape(L, act_dtype, n, h, w, 0, 0, 1)) return s;
    if (!bytes) return fail(PSC_ERR_ARG, "bytes is NULL");
    *bytes = psc::wgrad_workspace_bytes(n, L->cin, L->cout, h, w, L->keep, false);
    return ok();
}

psc_status psc_conv3x3_bwd_weight(const psc_layer* L, const psc_packed* pk, int32_t act_dtype, const void* d_x,
                                  const void* d_dy, int32_t n, int32_t h, int32_t w, float* d_dvalues,
                                  float* d_dbias, void* d_ws, size_t ws_bytes, void* stream) {
    if (psc_status s = check_conv_shape(L, act_dtype, n, h, w, 0, 0, 1)) return s;
    if (psc_status s = check_packed(L, pk)) return s;
    const size_t need = psc::wgrad_workspace_bytes(n, L->cin, L->cout, h, w, L->keep, false);
    if (need && (!d_ws || ws_bytes < need))
        return fail(PSC_ERR_WORKSPACE, "bwd weight needs %zu workspace bytes, got %zu", need, ws_bytes);
    if (n == 0) return ok();
    if (!psc::wgrad_fits(n, L->cin, L->cout, h, w, act_dtype))
        return fail(PSC_ERR_UNSUPPORTED, "bwd weight: x and dy must each fit in 2 GiB");
    if (!d_x || !d_dy) return fail(PSC_ERR_ARG, "d_x and d_dy must be non-NULL");
    if (L->keep > 0 && !d_dvalues) return fail(PSC_ERR_ARG, "d_dvalues must be non-NULL when keep > 0");
    if (reinterpret_cast<uintptr_t>(d_dvalues) & 15u) return fail(PSC_ERR_ARG, "d_dvalues must be 16-byte aligned");
    const psc::PatTable t = table_of(L);
    const psc::PackedView v{pk->filter_perm, pk->filter_ptr, pk->seg_ptr, pk->cin_idx, pk->pat_id, pk->values};
    return device_status(psc::launch_bwd_weight(t, v, act_dtype, n, L->cin, h, w, L->cout, L->keep, d_x, d_dy,
                                                d_dvalues, d_dbias, d_ws, as_stream(stream)),
                         "psc_conv3x3_bwd_weight launch");
}

psc_status psc_admm_residual(const float* d_z, const float* d_target, int64_t numel, float scale, float* d_g,
                             double* d_loss, void* d_ws, size_t ws_bytes, void* stream) {
    if (numel < 0 || numel > kMaxElems) return fail(PSC_ERR_ARG, "numel=%lld outside 0..2^31-1", (long long)numel);
    if (!(scale > 0.f) || !std::isfinite(scale)) return fail(PSC_ERR_ARG, "scale must be positive and finite");
    if (!d_loss || (numel > 0 && (!d_z || !d_target || !d_g)))
        return fail(PSC_ERR_ARG, "d_z, d_target, d_g and d_loss must be non-NULL");
    if (!d_ws || ws_bytes < psc::admm_residual_workspace_bytes())
        return fail(PSC_ERR_WORKSPACE, "psc_admm_residual needs %zu workspace bytes, got %zu",
                    psc::admm_residual_workspace_bytes(), ws_bytes);
    if (reinterpret_cast<uintptr_t>(d_ws) & 255u) return fail(PSC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    return device_status(psc::launch_admm_residual(d_z, d_target, numel, scale, d_g, d_loss, d_ws, as_stream(stream)),
                         "psc_admm_residual launch");
}

static psc_status check_dense_wgrad_shape(int32_t n, int32_t cin, int32_t h, int32_t w, int32_t cout) {
    if (n < 0 || n > 65535 || cin < 1 || cout < 1 || cout > 65535 || h < 1 || w < 1 || h > 32768 || w > 32768)
        return fail(PSC_ERR_ARG, "bad shape n=%d cin=%d cout=%d h=%d w=%d", n, cin, cout, h, w);
    const int64_t plane = int64_t(h) * w;
    if (int64_t(n) * cin * plane > kMaxElems || int64_t(n) * cout * plane > kMaxElems ||
        int64_t(cout) * cin * 9 > kMaxElems)
        return fail(PSC_ERR_ARG, "a tensor holds more than 2^31-1 elements");
    return PSC_OK;
}

psc_status psc_dense3x3_bwd_weight_workspace(int32_t n, int32_t cin, int32_t h, int32_t w, int32_t cout,
                                             size_t* bytes) {
    if (psc_status s = check_dense_wgrad_shape(n, cin, h, w, cout)) return s;
    if (!bytes) return fail(PSC_ERR_ARG, "bytes is NULL");
    *bytes = psc::wgrad_workspace_bytes(n, cin, cout, h, w, int64_t(cout) * cin, true);
    return ok();
}

psc_status psc_dense3x3_bwd_weight(const float* d_x, const float* d_g, int32_t n, int32_t cin, int32_t h,
                                   int32_t w, int32_t cout, float* d_dw, float* d_db, void* d_ws, size_t ws_bytes,
                                   void* stream) {
    if (psc_status s = check_dense_wgrad_shape(n, cin, h, w, cout)) return s;
    if (!d_dw) return fail(PSC_ERR_ARG, "d_dw must be non-NULL");
    if (n > 0 && (!d_x || !d_g)) return fail(PSC_ERR_ARG, "d_x and d_g must be non-NULL");
    const size_t need = psc::wgrad_workspace_bytes(n, cin, cout, h, w, int64_t(cout) * cin, true);
    if (need && (!d_ws || ws_bytes < need))
        return fail(PSC_ERR_WORKSPACE, "dense bwd weight needs %zu workspace bytes, got %zu", need, ws_bytes);
    if (n == 0) return ok();
    if (!psc::wgrad_fits(n, cin, cout, h, w, PSC_F32))
        return fail(PSC_ERR_UNSUPPORTED, "dense bwd weight: x and g must each fit in 2 GiB");
    return device_status(psc::launch_dense_wgrad(d_x, d_g, n, cin, h, w, cout, d_dw, d_db, d_ws, as_stream(stream)),
                         "psc_dense3x3_bwd_weight launch");
}

psc_status psc_admm_primal(int64_t n_weights, float* d_w, const float* d_dw, const float* d_a, const float* d_d,
                           int32_t cout, float* d_b, const float* d_db, float lr, float rho, float* d_v,
                           void* stream) {
    if (n_weights < 0 || n_weights > kMaxElems) return fail(PSC_ERR_ARG, "n_weights outside 0..2^31-1");
    if (cout < 0) return fail(PSC_ERR_ARG, "cout < 0");
    if (!std::isfinite(lr) || !std::isfinite(rho) || rho < 0.f) return fail(PSC_ERR_ARG, "lr and rho must be finite, rho >= 0");
    if (n_weights > 0 && (!d_w || !d_dw || !d_a || !d_d || !d_v))
        return fail(PSC_ERR_ARG, "d_w, d_dw, d_a, d_d and d_v must be non-NULL");
    if (d_b && cout > 0 && !d_db) return fail(PSC_ERR_ARG, "d_db must be non-NULL with d_b");
    return device_status(psc::launch_admm_primal(d_w, d_dw, d_a, d_d, n_weights, d_b, d_db, cout, lr, rho, d_v,
                                                 as_stream(stream)),
                         "psc_admm_primal launch");
}

psc_status psc_admm_dual(const psc_layer* L, const float* d_v, const uint8_t* d_pat, const uint8_t* d_keep,
                         float* d_a, float* d_d, void* stream) {
    if (psc_status s = check_layer(L, false)) return s;
    if (L->wdtype != PSC_F32) return fail(PSC_ERR_UNSUPPORTED, "the ADMM steps run in fp32");
    if (!d_v || !d_pat || !d_keep || !d_a || !d_d) return fail(PSC_ERR_ARG, "every pointer must be non-NULL");
    const psc::PatTable t = table_of(L);
    return device_status(psc::launch_admm_dual(t, d_v, d_pat, d_keep, int64_t(L->cout) * L->cin, d_a, d_d,
                                               as_stream(stream)),
                         "psc_admm_dual launch");
}

psc_status psc_dense3x3_fwd(int32_t dtype, const void* d_x, int32_t n, int32_t cin, int32_t h,
                            int32_t w, const void* d_w, int32_t cout, const void* d_bias,
                            int32_t relu, void* d_y, void* stream) {
    if (!dtype_ok(dtype)) return fail(PSC_ERR_ARG, "dtype=%d is not a psc_dtype", dtype);
    if (n < 0 || n > 65535 || cin < 1 || cout < 1 || cout > 65535 || h < 1 || w < 1 ||
        h > 32768 || w > 32768)
        return fail(PSC_ERR_ARG, "bad shape n=%d cin=%d cout=%d h=%d w=%d", n, cin, cout, h, w);
    const int64_t plane = int64_t(h) * w;
    if (int64_t(n) * cin * plane > kMaxElems || int64_t(n) * cout * plane > kMaxElems ||
        int64_t(cout) * cin * 9 > kMaxElems)
        return fail(PSC_ERR_ARG, "a tensor holds more than 2^31-1 elements");
    if (n == 0) return ok();
    if (!d_x || !d_w || !d_y) return fail(PSC_ERR_ARG, "d_x, d_w and d_y must be non-NULL");
    const size_t es = elt_size(dtype);
    if (overlaps(d_x, size_t(int64_t(n) * cin * plane) * es, d_y, size_t(int64_t(n) * cout * plane) * es))
        return fail(PSC_ERR_ARG, "d_y overlaps d_x");
    return device_status(psc::launch_dense(dtype, d_x, n, cin, h, w, d_w, cout, d_bias, relu != 0,
                                           d_y, as_stream(stream)),
                         "psc_dense3x3_fwd launch");
}

psc_status psc_maxpool2x2(int32_t dtype, const void* d_x, int32_t n, int32_t c, int32_t h, int32_t w,
                          void* d_y, void* stream) {
    if (!dtype_ok(dtype)) return fail(PSC_ERR_ARG, "dtype=%d is not a psc_dtype", dtype);
    if (n < 0 || c < 1 || h < 2 || w < 2 || (h & 1) || (w & 1))
        return fail(PSC_ERR_ARG, "bad shape n=%d c=%d h=%d w=%d (h, w even and >= 2)", n, c, h, w);
    if (int64_t(n) * c * h * w > kMaxElems) return fail(PSC_ERR_ARG, "x holds more than 2^31-1 elements");
    if (n == 0) return ok();
    if (!d_x || !d_y) return fail(PSC_ERR_ARG, "d_x and d_y must be non-NULL");
    return device_status(psc::launch_maxpool(dtype, d_x, n, c, h, w, d_y, as_stream(stream)),
                         "psc_maxpool2x2 launch");
}

psc_status psc_probe_fma(int32_t blocks, int32_t iters, float* d_out, void* stream) {
    if (blocks < 1 || blocks > (1 << 20) || iters < 0) return fail(PSC_ERR_ARG, "blocks=%d iters=%d", blocks, iters);
    if (!d_out) return fail(PSC_ERR_ARG, "d_out is NULL");
    return device_status(psc::launch_probe_fma(blocks, iters, d_out, as_stream(stream)), "psc_probe_fma launch");
}

psc_status psc_probe_mfma(int32_t blocks, int32_t iters, float* d_out, void* stream) {
    if (blocks < 1 || blocks > (1 << 20) || iters < 0) return fail(PSC_ERR_ARG, "blocks=%d iters=%d", blocks, iters);
    if (!d_out) return fail(PSC_ERR_ARG, "d_out is NULL");
    return device_status(psc::launch_probe_mfma(blocks, iters, d_out, as_stream(stream)), "psc_probe_mfma launch");
}

}  // extern "C"
