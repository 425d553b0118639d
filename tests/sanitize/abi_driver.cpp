// Host-side driver of libpsc's C ABI for the CPU sanitizer test: every call
// here either runs on the host only (library selection, configuration and
// workspace queries, transposed-layer description) or fails argument
// validation before any HIP call.  Built from host-only objects with
// AddressSanitizer and UndefinedBehaviorSanitizer; exits non-zero on the
// first unexpected status.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "psc.h"

static int g_fail = 0;
#define EXPECT(cond)                                                        \
    do {                                                                    \
        if (!(cond)) {                                                      \
            std::fprintf(stderr, "FAIL %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, psc_last_error()); \
            ++g_fail;                                                       \
        }                                                                   \
    } while (0)

static uint16_t f16_bits(float f) {
    // round-to-nearest-even fp32 -> fp16 for finite values in range, enough
    // for test data
    uint32_t x;
    std::memcpy(&x, &f, 4);
    const uint32_t sign = (x >> 16) & 0x8000u;
    const int exp = int((x >> 23) & 0xff) - 127 + 15;
    uint32_t mant = x & 0x7fffffu;
    if (exp <= 0) return uint16_t(sign);
    if (exp >= 31) return uint16_t(sign | 0x7c00u);
    uint32_t h = sign | (uint32_t(exp) << 10) | (mant >> 13);
    const uint32_t rest = mant & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h;
    return uint16_t(h);
}

static void library_selection() {
    std::mt19937 rng(7);
    std::normal_distribution<float> nd;
    for (int64_t nk : {int64_t(0), int64_t(1), int64_t(5), int64_t(1000)}) {
        std::vector<float> w(size_t(nk) * 9 + 1);
        for (auto& v : w) v = nd(rng);
        if (nk >= 5) {
            w[0] = 0.f, w[1] = -0.f, w[2] = INFINITY, w[3] = -INFINITY, w[5] = NAN;   // edge values
            for (int q = 9; q < 18; ++q) w[q] = 1.f;                                   // all ties
        }
        std::vector<uint16_t> h(w.size());
        for (size_t i = 0; i < w.size(); ++i) h[i] = f16_bits(w[i]);
        for (int m : {1, 8, 56}) {
            std::vector<uint16_t> masks(size_t(m) + 1, 0xffff);
            EXPECT(psc_select_library(w.data(), PSC_F32, nk, m, masks.data()) == PSC_OK);
            EXPECT(masks[size_t(m)] == 0xffff);                       // nothing written past m
            for (int p = 0; p < m; ++p) EXPECT(masks[size_t(p)] < 512 && ((masks[size_t(p)] >> 4) & 1));
            EXPECT(psc_select_library(h.data(), PSC_F16, nk, m, masks.data()) == PSC_OK);
        }
        uint16_t one[1];
        EXPECT(psc_select_library(w.data(), PSC_F32, nk, 0, one) == PSC_ERR_ARG);
        EXPECT(psc_select_library(w.data(), PSC_F32, nk, 57, one) == PSC_ERR_ARG);
        EXPECT(psc_select_library(w.data(), 7, nk, 8, one) == PSC_ERR_ARG);
        EXPECT(psc_select_library(w.data(), PSC_F32, nk, 8, nullptr) == PSC_ERR_ARG);
    }
    EXPECT(psc_select_library(nullptr, PSC_F32, 3, 8, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_select_library(nullptr, PSC_F32, -1, 8, nullptr) == PSC_ERR_ARG);
}

static psc_layer make_layer(int cout, int cin, int m, int64_t keep, int dt) {
    psc_layer L;
    std::memset(&L, 0, sizeof L);
    L.cout = cout, L.cin = cin, L.m = m, L.wdtype = dt, L.keep = keep;
    int n = 0;
    for (int c = 0; c < 512 && n < m; ++c)
        if (__builtin_popcount(unsigned(c)) == 4) L.masks[n++] = uint16_t(c);
    return L;
}

static void queries() {
    const int shapes[][2] = {{1, 1}, {2, 7}, {4, 4}, {8, 8}, {7, 7}, {13, 14}, {14, 14}, {16, 16}, {28, 28},
                             {32, 32}, {56, 56}, {63, 64}, {64, 64}, {112, 112}, {224, 224}, {17, 130}, {5, 253}};
    int n_ok = 0;
    for (int dt : {PSC_F32, PSC_F16})
        for (int m : {1, 6, 126}) {
            const psc_layer L = make_layer(24, 40, m, 24 * 40 / 3, dt);
            for (auto& hw : shapes)
                for (int n : {0, 1, 3, 8, 32, 300})
                    for (int algo = 0; algo <= 3; ++algo)
                        for (int stride = 1; stride <= 2; ++stride)
                            for (int pool = 0; pool <= 1; ++pool) {
                                psc_conv_config c;
                                const psc_status s = psc_conv3x3_config(&L, dt, n, hw[0], hw[1], pool, stride, algo, &c);
                                if (s == PSC_OK) {
                                    ++n_ok;
                                    EXPECT(c.kernel >= 0 && c.kernel <= 4 && c.blocks >= 0 && c.threads_per_block > 0 &&
                                           c.threads_per_block <= 1024 && c.shares >= 1 && c.shares <= 8);
                                } else {
                                    EXPECT(s == PSC_ERR_ARG || s == PSC_ERR_UNSUPPORTED);
                                }
                            }
            size_t b = 0;
            EXPECT(psc_workspace_size(&L, PSC_OP_SELECT, &b) == PSC_OK);
            EXPECT(psc_workspace_size(&L, PSC_OP_PACK, &b) == PSC_OK);
            EXPECT(psc_workspace_size(&L, 9, &b) == PSC_ERR_ARG);
            psc_layer T;
            EXPECT(psc_transpose_layer(&L, &T) == PSC_OK);
            EXPECT(T.cout == L.cin && T.cin == L.cout && T.m == L.m && T.keep == L.keep);
            EXPECT(psc_conv3x3_bwd_weight_workspace(&L, dt, 4, 9, 11, &b) == PSC_OK);
            EXPECT(psc_conv3x3_bwd_weight_workspace(&L, dt, -1, 9, 11, &b) == PSC_ERR_ARG);
        }
    EXPECT(n_ok > 1000);
    size_t b = 0;
    EXPECT(psc_dense3x3_bwd_weight_workspace(32, 3, 224, 224, 64, &b) == PSC_OK);
    EXPECT(psc_dense3x3_bwd_weight_workspace(0, 3, 224, 224, 64, &b) == PSC_OK);
    EXPECT(psc_dense3x3_bwd_weight_workspace(1, 0, 4, 4, 4, &b) == PSC_ERR_ARG);
}

static void validation() {
    // malformed layers: every entry point rejects them before touching a pointer
    psc_layer bad = make_layer(4, 4, 2, 3, PSC_F32);
    bad.masks[1] = bad.masks[0];                                   // duplicate mask
    size_t b;
    EXPECT(psc_workspace_size(&bad, PSC_OP_PACK, &b) == PSC_ERR_ARG);
    bad = make_layer(4, 4, 2, 17, PSC_F32);                        // keep > cout*cin
    EXPECT(psc_workspace_size(&bad, PSC_OP_PACK, &b) == PSC_OK);  // sizes do not depend on keep
    psc_conv_config cfg;
    EXPECT(psc_conv3x3_config(&bad, PSC_F32, 1, 8, 8, 0, 1, 0, &cfg) == PSC_ERR_ARG);
    bad = make_layer(4, 4, 0, 3, PSC_F32);                         // empty library
    EXPECT(psc_project(&bad, nullptr, nullptr, nullptr, nullptr) == PSC_ERR_ARG);
    bad = make_layer(4, 4, 2, 3, PSC_F32);
    bad.masks[0] = 0x1ff;                                          // 9 bits set
    EXPECT(psc_project(&bad, nullptr, nullptr, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_project(nullptr, nullptr, nullptr, nullptr, nullptr) == PSC_ERR_ARG);
    const psc_layer L = make_layer(4, 4, 2, 3, PSC_F32);
    EXPECT(psc_project(&L, nullptr, nullptr, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_select(&L, nullptr, nullptr, nullptr, 0, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_pack(&L, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr) == PSC_ERR_ARG);
    psc_packed pk;
    std::memset(&pk, 0, sizeof pk);
    EXPECT(psc_conv3x3_fwd(&L, &pk, PSC_F32, nullptr, 1, 4, 4, nullptr, 0, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_conv3x3_fwd(&L, nullptr, PSC_F32, nullptr, 1, 4, 4, nullptr, 0, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_conv3x3_fwd_algo(&L, &pk, PSC_F32, nullptr, 1, 4, 4, nullptr, 0, nullptr, 9, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_conv3x3_fwd_strided(&L, &pk, PSC_F32, nullptr, 1, 4, 4, nullptr, 0, nullptr, 3, 0, nullptr) ==
           PSC_ERR_ARG);
    EXPECT(psc_conv3x3_fwd_pool2(&L, &pk, PSC_F32, nullptr, 1, 5, 4, nullptr, 0, nullptr, 0, nullptr) ==
           PSC_ERR_ARG);
    EXPECT(psc_conv3x3_fwd(&L, &pk, PSC_F16, nullptr, 1, 4, 4, nullptr, 0, nullptr, nullptr) ==
           PSC_ERR_UNSUPPORTED);                                  // activations differ from the weights
    EXPECT(psc_conv3x3_fwd(&L, &pk, PSC_F32, nullptr, 1, 1 << 20, 1 << 20, nullptr, 0, nullptr, nullptr) ==
           PSC_ERR_ARG);                                          // beyond 2^31 elements
    EXPECT(psc_maxpool2x2(PSC_F32, nullptr, 1, 1, 3, 4, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_dense3x3_fwd(5, nullptr, 1, 1, 4, 4, nullptr, 1, nullptr, 0, nullptr, nullptr) == PSC_ERR_ARG);
    EXPECT(psc_admm_primal(-1, nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, 0.1f, 0.1f, nullptr,
                           nullptr) == PSC_ERR_ARG);
    EXPECT(std::strlen(psc_status_string(PSC_ERR_DEVICE)) > 0);
    EXPECT(std::strlen(psc_status_string(psc_status(99))) > 0);
    EXPECT(psc_abi_version() >= 1);
}

int main() {
    library_selection();
    queries();
    validation();
    if (g_fail) {
        std::fprintf(stderr, "%d failures\n", g_fail);
        return 1;
    }
    std::printf("abi driver ok\n");
    return 0;
}
