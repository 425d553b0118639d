/* Driver of the oracle (oracle/pso.c) for the CPU sanitizer test: the whole
 * pipeline -- library selection, projection, selection, packing, unpacking,
 * masking, the sparse conv at stride 1 and 2 (fp64 and fp32 accumulation),
 * the dense witness, the pool and both backward passes -- on small seeded
 * shapes including single rows and columns, odd sizes, keep = 0 and keep =
 * all.  Built with AddressSanitizer and UndefinedBehaviorSanitizer; exits
 * non-zero if a call fails. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int pso_select_library(const void *w, int dtype, int64_t n_kernels, int m, uint16_t *masks_out);
int pso_project(const void *w, int dtype, int64_t n_kernels, const uint16_t *masks, int m, uint8_t *pat,
                double *energy);
int pso_select(const double *energy, int64_t n_kernels, int64_t keep, uint8_t *keep_out);
int pso_pack(const void *w, int dtype, int cout, int cin, int m, const uint16_t *masks, const uint8_t *pat,
             const uint8_t *keep, int32_t *filter_perm, int32_t *filter_ptr, int32_t *seg_ptr, int32_t *cin_idx,
             uint8_t *pat_id, void *values);
int pso_mask_weights(const void *w, int dtype, int64_t n_kernels, const uint16_t *masks, int m, const uint8_t *pat,
                     const uint8_t *keep, void *w_masked);
int pso_unpack(int dtype, int cout, int cin, int m, const uint16_t *masks, const int32_t *filter_perm,
               const int32_t *filter_ptr, const int32_t *cin_idx, const uint8_t *pat_id, const void *values,
               void *w_dense);
int pso_conv_sparse_st(const double *x, int n, int cin, int h, int w, int cout, int m, const uint16_t *masks,
                       const int32_t *filter_perm, const int32_t *filter_ptr, const int32_t *cin_idx,
                       const uint8_t *pat_id, const void *values, int vdtype, const double *bias, int relu, int st,
                       double *y, double *s);
int pso_conv_sparse_f32acc(const float *x, int n, int cin, int h, int w, int cout, int m, const uint16_t *masks,
                           const int32_t *filter_perm, const int32_t *filter_ptr, const int32_t *cin_idx,
                           const uint8_t *pat_id, const void *values, int vdtype, const float *bias, int relu,
                           int st, float *y);
int pso_conv_sparse_bwd_data(const double *dy, int n, int cin, int h, int w, int cout, int m,
                             const uint16_t *masks, const int32_t *filter_perm, const int32_t *filter_ptr,
                             const int32_t *cin_idx, const uint8_t *pat_id, const void *values, int vdtype,
                             double *dx, double *s);
int pso_conv_sparse_bwd_weight(const double *x, const double *dy, int n, int cin, int h, int w, int cout, int m,
                               const uint16_t *masks, const int32_t *filter_perm, const int32_t *filter_ptr,
                               const int32_t *cin_idx, const uint8_t *pat_id, double *dv, double *s_dv,
                               double *db);
int pso_conv_dense(const void *x, int dtype, int n, int cin, int h, int w, const void *wdense, int cout,
                   const void *bias, int relu, double *y);
int pso_maxpool2x2(const double *x, int64_t nc, int h, int w, double *y);

static uint64_t g_state = 88172645463325252ull;
static double urand(void) {   /* xorshift64, uniform in [-1, 1) */
    g_state ^= g_state << 13;
    g_state ^= g_state >> 7;
    g_state ^= g_state << 17;
    return (double)(g_state >> 11) / 4503599627370496.0 - 1.0;
}

static int fails = 0;
#define CHECK(e)                                                            \
    do {                                                                    \
        if ((e) != 0) {                                                     \
            fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #e);            \
            ++fails;                                                        \
        }                                                                   \
    } while (0)

static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    if (!p) abort();
    memset(p, 0, n ? n : 1);
    return p;
}

static void run_case(int n, int cin, int cout, int h, int w, int m, int keep_mode) {
    const int64_t nk = (int64_t)cout * cin;
    float *wt = xmalloc(sizeof(float) * (size_t)nk * 9);
    for (int64_t i = 0; i < nk * 9; ++i) wt[i] = (float)urand();
    uint16_t masks[56];
    CHECK(pso_select_library(wt, 0, nk, m, masks));
    uint8_t *pat = xmalloc((size_t)nk);
    double *energy = xmalloc(sizeof(double) * (size_t)nk);
    CHECK(pso_project(wt, 0, nk, masks, m, pat, energy));
    const int64_t keep = keep_mode == 0 ? 0 : (keep_mode == 1 ? nk : nk / 3);
    uint8_t *kp = xmalloc((size_t)nk);
    CHECK(pso_select(energy, nk, keep, kp));
    int32_t *perm = xmalloc(sizeof(int32_t) * (size_t)cout), *fptr = xmalloc(sizeof(int32_t) * (size_t)(cout + 1));
    int32_t *seg = xmalloc(sizeof(int32_t) * (size_t)cout * (size_t)(m + 1));
    int32_t *ci = xmalloc(sizeof(int32_t) * (size_t)keep);
    uint8_t *pid = xmalloc((size_t)keep);
    float *vals = xmalloc(sizeof(float) * (size_t)keep * 4);
    CHECK(pso_pack(wt, 0, cout, cin, m, masks, pat, kp, perm, fptr, seg, ci, pid, vals));
    float *wd = xmalloc(sizeof(float) * (size_t)nk * 9), *wm = xmalloc(sizeof(float) * (size_t)nk * 9);
    CHECK(pso_unpack(0, cout, cin, m, masks, perm, fptr, ci, pid, vals, wd));
    CHECK(pso_mask_weights(wt, 0, nk, masks, m, pat, kp, wm));
    CHECK(memcmp(wd, wm, sizeof(float) * (size_t)nk * 9) != 0);
    const size_t xe = (size_t)n * cin * h * w, ye = (size_t)n * cout * h * w;
    double *x = xmalloc(sizeof(double) * xe), *y = xmalloc(sizeof(double) * ye), *s = xmalloc(sizeof(double) * ye);
    float *xf = xmalloc(sizeof(float) * xe), *yf = xmalloc(sizeof(float) * ye), *bf = xmalloc(sizeof(float) * cout);
    double *b = xmalloc(sizeof(double) * (size_t)cout);
    for (size_t i = 0; i < xe; ++i) xf[i] = (float)urand(), x[i] = xf[i];
    for (int i = 0; i < cout; ++i) bf[i] = (float)urand(), b[i] = bf[i];
    for (int st = 1; st <= 2; ++st)
        CHECK(pso_conv_sparse_st(x, n, cin, h, w, cout, m, masks, perm, fptr, ci, pid, vals, 0, b, st - 1, st, y, s));
    for (int st = 1; st <= 2; ++st)
        CHECK(pso_conv_sparse_f32acc(xf, n, cin, h, w, cout, m, masks, perm, fptr, ci, pid, vals, 0, bf, 1, st, yf));
    CHECK(pso_conv_dense(xf, 0, n, cin, h, w, wd, cout, bf, 0, y));
    double *dx = xmalloc(sizeof(double) * xe), *sx = xmalloc(sizeof(double) * xe);
    double *dv = xmalloc(sizeof(double) * (size_t)keep * 4);
    double *sdv = xmalloc(sizeof(double) * (size_t)keep * 4), *db = xmalloc(sizeof(double) * (size_t)cout);
    CHECK(pso_conv_sparse_bwd_data(y, n, cin, h, w, cout, m, masks, perm, fptr, ci, pid, vals, 0, dx, sx));
    CHECK(pso_conv_sparse_bwd_weight(x, y, n, cin, h, w, cout, m, masks, perm, fptr, ci, pid, dv, sdv, db));
    if (h % 2 == 0 && w % 2 == 0) {
        double *p = xmalloc(sizeof(double) * ye / 4);
        CHECK(pso_maxpool2x2(y, (int64_t)n * cout, h, w, p));
        free(p);
    }
    free(wt), free(pat), free(energy), free(kp), free(perm), free(fptr), free(seg), free(ci), free(pid);
    free(vals), free(wd), free(wm), free(x), free(y), free(s), free(xf), free(yf), free(bf), free(b);
    free(dx), free(sx), free(dv), free(sdv), free(db);
}

int main(void) {
    const int shapes[][5] = {{1, 1, 1, 1, 1}, {2, 3, 5, 1, 9}, {1, 4, 2, 9, 1}, {3, 5, 7, 6, 8},
                             {2, 8, 3, 13, 17}, {1, 2, 9, 32, 4}};
    for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i)
        for (int km = 0; km < 3; ++km)
            for (int m = 1; m <= 56; m += 55 - 47 * (m == 1))   /* m = 1, 8, 56 */
                run_case(shapes[i][0], shapes[i][1], shapes[i][2], shapes[i][3], shapes[i][4], m, km);
    /* argument checks */
    uint16_t masks[8];
    CHECK(pso_select_library(NULL, 0, 5, 8, masks) != -1);
    CHECK(pso_select(NULL, 4, 5, NULL) != -1);
    if (fails) {
        fprintf(stderr, "%d failures\n", fails);
        return 1;
    }
    printf("pso driver ok\n");
    return 0;
}
