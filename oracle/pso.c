/*
 * pso.c -- CPU oracle for pattern-sparse 3x3 convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no source with the HIP library.
 *
 * Every function is the plain definition of one step of the method of
 * "A Privacy-Preserving-Oriented DNN Pruning and Mobile Acceleration
 * Framework" (Gong et al., GLSVLSI'20), written for obviousness, not speed:
 *
 *   pso_select_library  pattern-library heuristic            (Sec. 4.2)
 *   pso_project         Euclidean projection onto C_n        (Sec. 4.3, Eq. 6)
 *   pso_select          connectivity pruning, C'_n           (Sec. 4.4)
 *   pso_pack            filter kernel reorder + compressed
 *                       weight storage                       (Sec. 3.4)
 *   pso_mask_weights    M o W with dropped kernels zeroed    (Sec. 3.2)
 *   pso_unpack          compressed storage -> dense OIHW     (Sec. 3.4)
 *   pso_conv_sparse_st  X_n = sigma(W_n X_{n-1} + b_n) from
 *                       the compressed storage, stride 1 or 2
 *                       (stride 2: stage-entry convs of the
 *                       pruned ResNets)                      (Sec. 4.1, Eq. 1)
 *   pso_conv_sparse_f32acc  the same loop accumulating in fp32
 *                       (timed CPU baseline only)
 *   pso_conv_sparse_bwd_data    dx: adjoint of Eq. 1 (retraining)   (Sec. 3.3)
 *   pso_conv_sparse_bwd_weight  masked gradient of the stored values
 *                       and of the bias (retraining)         (Sec. 3.3)
 *   pso_conv_dense      textbook dense direct convolution of
 *                       zero-masked OIHW weights (witness)   (Sec. 4.1, Eq. 1)
 *   pso_maxpool2x2      2x2/2 max-pool between VGG-16 layers
 *
 * Arithmetic is fp64 throughout.  fp16 (IEEE binary16) and fp32 inputs are
 * converted to double exactly.
 *
 * Readings of points the paper leaves open:
 *  - "3 largest weights" means largest magnitude; ties go to the lower
 *    position index 3r+s.
 *  - library order: code frequency descending, then code ascending; when
 *    fewer than m codes occur, unseen centre+3 codes follow in ascending order.
 *  - "largest Frobenius norm": the energy of a pattern is the fp64 sum of the
 *    squares of the kept entries, added in ascending position order; ties go
 *    to the lowest library index.
 *  - connectivity pruning keeps exactly beta kernels: the beta largest
 *    post-projection energies, ties to the lower flat index co*Cin+ci.
 *  - compressed storage order: filters sorted by (kept count descending,
 *    per-pattern counts lexicographically descending, filter ascending);
 *    inside a filter, kernels sorted by (pattern ascending, ci ascending).
 *  - convolution is cross-correlation, stride 1, zero padding 1, optional
 *    bias, optional ReLU as sigma.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define PSO_F32 0
#define PSO_F16 1
#define PSO_F64 2   /* activations widened to double before the call */

/* IEEE 754 binary16 -> double, from the format's definition (exact). */
static double half_bits_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0)
        v = ldexp((double)frac, -24);                 /* subnormal or zero */
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(frac | 0x400), expo - 25); /* (1.f) * 2^(e-15) */
    return sign ? -v : v;
}

static double elem(const void *p, int dtype, size_t i)
{
    if (dtype == PSO_F16)
        return half_bits_to_double(((const uint16_t *)p)[i]);
    if (dtype == PSO_F64)
        return ((const double *)p)[i];
    return (double)((const float *)p)[i];
}

static size_t elem_size(int dtype) { return dtype == PSO_F16 ? 2 : (dtype == PSO_F64 ? 8 : 4); }

static int popcount9(unsigned v)
{
    int c = 0;
    for (int b = 0; b < 9; ++b)
        c += (v >> b) & 1;
    return c;
}

int pso_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for the following parallel loops (the benchmark times the
 * baseline on all cores and on one). */
void pso_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Sec. 4.2: for every kernel, the positions of its 3 largest non-centre
 * weights plus the centre form a 4-entry pattern; the m patterns that occur
 * most often form the library.  Only centre+3 codes can be produced, so m is
 * at most C(8,3) = 56.  Returns 0 on success, -1 on bad arguments. */
int pso_select_library(const void *w, int dtype, int64_t n_kernels, int m,
                       uint16_t *masks_out)
{
    if (m < 1 || m > 56 || n_kernels < 0 || (n_kernels > 0 && !w) || !masks_out)
        return -1;
    int64_t count[512];
    for (int c = 0; c < 512; ++c)
        count[c] = 0;
    for (int64_t k = 0; k < n_kernels; ++k) {
        double mag[9];
        for (int pos = 0; pos < 9; ++pos)
            mag[pos] = fabs(elem(w, dtype, (size_t)k * 9 + pos));
        unsigned code = 1u << 4;                  /* the centre is always kept */
        for (int t = 0; t < 3; ++t) {
            int best = -1;
            for (int pos = 0; pos < 9; ++pos) {
                if (pos == 4 || (code >> pos) & 1)
                    continue;
                if (best < 0 || mag[pos] > mag[best]) /* strict: lower pos wins ties */
                    best = pos;
            }
            code |= 1u << best;
        }
        count[code] += 1;
    }
    /* Candidates: every centre+3 code, ordered by (count desc, code asc).
     * Unseen codes have count 0 and so follow the seen ones in code order. */
    int cand[56];
    int nc = 0;
    for (unsigned c = 0; c < 512; ++c)
        if (((c >> 4) & 1) && popcount9(c) == 4)
            cand[nc++] = (int)c;
    /* selection sort: obviously correct, 56 entries */
    for (int i = 0; i < nc; ++i) {
        int best = i;
        for (int j = i + 1; j < nc; ++j) {
            int64_t cj = count[cand[j]], cb = count[cand[best]];
            if (cj > cb || (cj == cb && cand[j] < cand[best]))
                best = j;
        }
        int tmp = cand[i];
        cand[i] = cand[best];
        cand[best] = tmp;
    }
    for (int i = 0; i < m; ++i)
        masks_out[i] = (uint16_t)cand[i];
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 4.3, Eq. 6: the Euclidean projection onto C_n keeps, per kernel, the
 * library pattern whose pruned kernel has the largest Frobenius norm.  The
 * energy e[k,p] is the squared norm of the kept entries.  Returns -1 on bad
 * arguments (mask not a 4-of-9 code). */
int pso_project(const void *w, int dtype, int64_t n_kernels,
                const uint16_t *masks, int m, uint8_t *pat, double *energy)
{
    if (m < 1 || m > 126 || n_kernels < 0 || !masks)
        return -1;
    for (int p = 0; p < m; ++p)
        if (masks[p] >= 512 || popcount9(masks[p]) != 4)
            return -1;
    for (int64_t k = 0; k < n_kernels; ++k) {
        int best_p = 0;
        double best_e = 0.0;
        for (int p = 0; p < m; ++p) {
            double e = 0.0;
            for (int pos = 0; pos < 9; ++pos) {
                if ((masks[p] >> pos) & 1) {
                    double v = elem(w, dtype, (size_t)k * 9 + pos);
                    e = e + v * v;
                }
            }
            if (p == 0 || e > best_e) {     /* strict: first maximum wins */
                best_e = e;
                best_p = p;
            }
        }
        pat[k] = (uint8_t)best_p;
        energy[k] = best_e;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 4.4: at most beta_n kernels may be nonzero.  The projection keeps the
 * kernels with the largest retained energy.  Exactly `keep` are kept; equal
 * energies are broken by the lower flat index. */
typedef struct {
    double e;
    int64_t idx;
} pso_ekey;

static int cmp_ekey(const void *a, const void *b)
{
    const pso_ekey *x = (const pso_ekey *)a, *y = (const pso_ekey *)b;
    if (x->e > y->e) return -1;
    if (x->e < y->e) return 1;
    if (x->idx < y->idx) return -1;
    if (x->idx > y->idx) return 1;
    return 0;
}

int pso_select(const double *energy, int64_t n_kernels, int64_t keep,
               uint8_t *keep_out)
{
    if (n_kernels < 0 || keep < 0 || keep > n_kernels)
        return -1;
    pso_ekey *keys = (pso_ekey *)malloc(sizeof(pso_ekey) * (size_t)(n_kernels > 0 ? n_kernels : 1));
    if (!keys)
        return -1;
    for (int64_t k = 0; k < n_kernels; ++k) {
        keys[k].e = energy[k];
        keys[k].idx = k;
        keep_out[k] = 0;
    }
    qsort(keys, (size_t)n_kernels, sizeof(pso_ekey), cmp_ekey);
    for (int64_t r = 0; r < keep; ++r)
        keep_out[keys[r].idx] = 1;
    free(keys);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.4: filter kernel reorder groups filters of similar length and
 * pattern make-up; the compressed storage then holds, per reordered filter,
 * the kept kernels' input-channel index, pattern id and 4 values. */
typedef struct {
    int f;
    int n;
    const int32_t *cnt; /* m counts */
    int m;
} pso_fkey;

static int cmp_fkey(const void *a, const void *b)
{
    const pso_fkey *x = (const pso_fkey *)a, *y = (const pso_fkey *)b;
    if (x->n != y->n)
        return x->n > y->n ? -1 : 1;
    for (int p = 0; p < x->m; ++p)
        if (x->cnt[p] != y->cnt[p])
            return x->cnt[p] > y->cnt[p] ? -1 : 1;
    return x->f < y->f ? -1 : (x->f > y->f ? 1 : 0);
}

int pso_pack(const void *w, int dtype, int cout, int cin, int m,
             const uint16_t *masks, const uint8_t *pat, const uint8_t *keep,
             int32_t *filter_perm, int32_t *filter_ptr, int32_t *seg_ptr,
             int32_t *cin_idx, uint8_t *pat_id, void *values)
{
    if (cout < 0 || cin < 0 || m < 1 || m > 126)
        return -1;
    size_t es = elem_size(dtype);
    int32_t *cnt = (int32_t *)calloc((size_t)(cout > 0 ? cout : 1) * (size_t)m, sizeof(int32_t));
    pso_fkey *fk = (pso_fkey *)malloc(sizeof(pso_fkey) * (size_t)(cout > 0 ? cout : 1));
    if (!cnt || !fk) {
        free(cnt);
        free(fk);
        return -1;
    }
    for (int f = 0; f < cout; ++f) {
        int n = 0;
        for (int ci = 0; ci < cin; ++ci) {
            size_t k = (size_t)f * cin + ci;
            if (keep[k]) {
                if (pat[k] >= m) {
                    free(cnt);
                    free(fk);
                    return -1;
                }
                n += 1;
                cnt[(size_t)f * m + pat[k]] += 1;
            }
        }
        fk[f].f = f;
        fk[f].n = n;
        fk[f].cnt = cnt + (size_t)f * m;
        fk[f].m = m;
    }
    qsort(fk, (size_t)cout, sizeof(pso_fkey), cmp_fkey);
    filter_ptr[0] = 0;
    for (int i = 0; i < cout; ++i) {
        filter_perm[i] = fk[i].f;
        filter_ptr[i + 1] = filter_ptr[i] + fk[i].n;
    }
    for (int i = 0; i < cout; ++i) {
        int f = fk[i].f;
        int32_t start = filter_ptr[i];
        for (int p = 0; p < m; ++p) {
            seg_ptr[(size_t)i * (m + 1) + p] = start;
            start += cnt[(size_t)f * m + p];
        }
        seg_ptr[(size_t)i * (m + 1) + m] = filter_ptr[i + 1];
        int32_t pos = filter_ptr[i];
        for (int p = 0; p < m; ++p) {
            for (int ci = 0; ci < cin; ++ci) {
                size_t k = (size_t)f * cin + ci;
                if (!keep[k] || pat[k] != p)
                    continue;
                cin_idx[pos] = ci;
                pat_id[pos] = (uint8_t)p;
                int j = 0;
                for (int q = 0; q < 9; ++q) {
                    if ((masks[p] >> q) & 1) {
                        memcpy((char *)values + ((size_t)pos * 4 + j) * es,
                               (const char *)w + (k * 9 + q) * es, es);
                        j += 1;
                    }
                }
                pos += 1;
            }
        }
    }
    free(cnt);
    free(fk);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2: pattern pruning is the element-wise product M o W; connectivity
 * pruning removes whole kernels.  Kept entries are bit copies of W, every
 * other entry is +0. */
int pso_mask_weights(const void *w, int dtype, int64_t n_kernels,
                     const uint16_t *masks, int m, const uint8_t *pat,
                     const uint8_t *keep, void *w_masked)
{
    size_t es = elem_size(dtype);
    memset(w_masked, 0, (size_t)n_kernels * 9 * es);
    for (int64_t k = 0; k < n_kernels; ++k) {
        if (!keep[k])
            continue;
        if (pat[k] >= m)
            return -1;
        for (int q = 0; q < 9; ++q)
            if ((masks[pat[k]] >> q) & 1)
                memcpy((char *)w_masked + ((size_t)k * 9 + q) * es,
                       (const char *)w + ((size_t)k * 9 + q) * es, es);
    }
    return 0;
}

/* Compressed storage back to dense OIHW (original filter order). */
int pso_unpack(int dtype, int cout, int cin, int m, const uint16_t *masks,
               const int32_t *filter_perm, const int32_t *filter_ptr,
               const int32_t *cin_idx, const uint8_t *pat_id,
               const void *values, void *w_dense)
{
    size_t es = elem_size(dtype);
    memset(w_dense, 0, (size_t)cout * cin * 9 * es);
    for (int i = 0; i < cout; ++i) {
        int f = filter_perm[i];
        for (int32_t k = filter_ptr[i]; k < filter_ptr[i + 1]; ++k) {
            if (pat_id[k] >= m || cin_idx[k] < 0 || cin_idx[k] >= cin)
                return -1;
            int j = 0;
            for (int q = 0; q < 9; ++q) {
                if ((masks[pat_id[k]] >> q) & 1) {
                    memcpy((char *)w_dense + (((size_t)f * cin + cin_idx[k]) * 9 + q) * es,
                           (const char *)values + ((size_t)k * 4 + j) * es, es);
                    j += 1;
                }
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 4.1, Eq. 1: a layer computes X_n = sigma(W_n X_{n-1} + b_n).  For a
 * 3x3 convolution with zero padding 1, read from the compressed storage:
 *   y[n,f,i,j] = sigma(b[f] + sum over the kept kernels (ci, p) of f of
 *                sum_t v_t * x[n, ci, st*i + r_t - 1, st*j + s_t - 1]),
 * where (r_t, s_t) is the t-th set position of pattern p in ascending 3r+s
 * order, st the stride (1, or 2 for the stage-entry convolutions of the
 * ResNets the paper prunes) and taps outside the image read zero.  The
 * output is [n][cout][OH][OW], OH = (h-1)/st + 1, OW = (w-1)/st + 1.
 *
 * Every output starts at +0 and receives its products in storage order
 * (kernels in order, the 4 taps in ascending position), then the bias; each
 * tap is applied to the rows and columns whose input lies inside the image
 * (the range is computed instead of testing every pixel; the adds are the
 * same).  x is double [n][cin][h][w] (fp32 and fp16 activations widen to
 * double exactly); values are in vdtype; bias is double [cout] or NULL.
 * If s is non-null it receives the sum of |v*x| over the same terms plus |b|,
 * the scale of an element-wise rounding-error bound. */
static void out_range(int st, int off, int in_size, int out_size, int *lo, int *hi)
{
    /* outputs o in [0, out_size) with 0 <= st*o + off - 1 < in_size */
    int a = 0, b = out_size;
    while (a < b && st * a + off - 1 < 0)
        ++a;
    while (b > a && st * (b - 1) + off - 1 >= in_size)
        --b;
    *lo = a;
    *hi = b;
}

/* One output row of one tap: y[o] += v * x[st*o], and s[o] += |v * x[st*o]|
 * when s is non-null, for o in [o0, o1).  st is a compile-time 1 or 2 at
 * each call, so the unit-stride loop vectorises. */
static inline void tap_row(double *restrict y, double *restrict s, const double *restrict x,
                           const int st, double v, int o0, int o1)
{
    if (s) {
        for (int o = o0; o < o1; ++o) {
            double prod = v * x[(size_t)st * o];
            y[o] += prod;
            s[o] += fabs(prod);
        }
    } else {
        for (int o = o0; o < o1; ++o)
            y[o] += v * x[(size_t)st * o];
    }
}

int pso_conv_sparse_st(const double *x, int n, int cin, int h, int w,
                       int cout, int m, const uint16_t *masks,
                       const int32_t *filter_perm, const int32_t *filter_ptr,
                       const int32_t *cin_idx, const uint8_t *pat_id,
                       const void *values, int vdtype, const double *bias, int relu,
                       int st, double *y, double *s)
{
    if (n < 0 || cin < 0 || h < 1 || w < 1 || cout < 0 || m < 1 || m > 126 || st < 1 || st > 2)
        return -1;
    const int OH = (h - 1) / st + 1, OW = (w - 1) / st + 1;
    const size_t plane = (size_t)h * w, oplane = (size_t)OH * OW;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < (int64_t)n * cout; ++t) {
        int nn = (int)(t / cout);
        int i = (int)(t % cout);
        int f = filter_perm[i];
        double *yp = y + ((size_t)nn * cout + f) * oplane;
        double *sp = s ? s + ((size_t)nn * cout + f) * oplane : NULL;
        for (size_t q = 0; q < oplane; ++q) {
            yp[q] = 0.0;
            if (sp)
                sp[q] = 0.0;
        }
        for (int32_t k = filter_ptr[i]; k < filter_ptr[i + 1]; ++k) {
            int ci = cin_idx[k];
            int p = pat_id[k];
            if (p >= m || ci < 0 || ci >= cin) {
                bad = 1;
                continue;
            }
            const double *xc = x + ((size_t)nn * cin + ci) * plane;
            int j = 0;
            for (int q = 0; q < 9; ++q) {
                if (!((masks[p] >> q) & 1))
                    continue;
                int r = q / 3, c = q % 3;
                double v = elem(values, vdtype, (size_t)k * 4 + j);
                j += 1;
                int oh0, oh1, ow0, ow1;
                out_range(st, r, h, OH, &oh0, &oh1);
                out_range(st, c, w, OW, &ow0, &ow1);
                for (int oh = oh0; oh < oh1; ++oh) {
                    const double *xr = xc + (size_t)(st * oh + r - 1) * w + (c - 1);
                    double *yr = yp + (size_t)oh * OW;
                    double *sr = sp ? sp + (size_t)oh * OW : NULL;
                    if (st == 1)
                        tap_row(yr, sr, xr, 1, v, ow0, ow1);
                    else
                        tap_row(yr, sr, xr, 2, v, ow0, ow1);
                }
            }
        }
        double b = bias ? bias[f] : 0.0;
        for (size_t q = 0; q < oplane; ++q) {
            double v = yp[q] + b;
            yp[q] = (relu && v < 0.0) ? 0.0 : v;
            if (sp)
                sp[q] += fabs(b);
        }
    }
    return bad ? -1 : 0;
}

/* The same loop with fp32 accumulation (float activations, outputs and
 * bias): the CPU baseline the benchmark times.  Never used for parity. */
int pso_conv_sparse_f32acc(const float *x, int n, int cin, int h, int w,
                           int cout, int m, const uint16_t *masks,
                           const int32_t *filter_perm, const int32_t *filter_ptr,
                           const int32_t *cin_idx, const uint8_t *pat_id,
                           const void *values, int vdtype, const float *bias, int relu,
                           int st, float *y)
{
    if (n < 0 || cin < 0 || h < 1 || w < 1 || cout < 0 || m < 1 || m > 126 || st < 1 || st > 2)
        return -1;
    const int OH = (h - 1) / st + 1, OW = (w - 1) / st + 1;
    const size_t plane = (size_t)h * w, oplane = (size_t)OH * OW;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < (int64_t)n * cout; ++t) {
        int nn = (int)(t / cout);
        int i = (int)(t % cout);
        int f = filter_perm[i];
        float *yp = y + ((size_t)nn * cout + f) * oplane;
        for (size_t q = 0; q < oplane; ++q)
            yp[q] = 0.0f;
        for (int32_t k = filter_ptr[i]; k < filter_ptr[i + 1]; ++k) {
            int ci = cin_idx[k];
            int p = pat_id[k];
            if (p >= m || ci < 0 || ci >= cin) {
                bad = 1;
                continue;
            }
            const float *xc = x + ((size_t)nn * cin + ci) * plane;
            int j = 0;
            for (int q = 0; q < 9; ++q) {
                if (!((masks[p] >> q) & 1))
                    continue;
                int r = q / 3, c = q % 3;
                float v = (float)elem(values, vdtype, (size_t)k * 4 + j);
                j += 1;
                int oh0, oh1, ow0, ow1;
                out_range(st, r, h, OH, &oh0, &oh1);
                out_range(st, c, w, OW, &ow0, &ow1);
                for (int oh = oh0; oh < oh1; ++oh) {
                    const float *xr = xc + (size_t)(st * oh + r - 1) * w + (c - 1);
                    float *yr = yp + (size_t)oh * OW;
                    for (int ow = ow0; ow < ow1; ++ow)
                        yr[ow] += v * xr[(size_t)st * ow];
                }
            }
        }
        float b = bias ? bias[f] : 0.0f;
        for (size_t q = 0; q < oplane; ++q) {
            float v = yp[q] + b;
            yp[q] = (relu && v < 0.0f) ? 0.0f : v;
        }
    }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Retraining (Sec. 3.3): the user retrains the pruned model with the pruned
 * weights' gradients set to zero.  For the layer of Eq. 1 (stride 1, zero
 * padding 1) with loss gradient dy = dL/dy (taken after sigma), these are
 * the two products of backpropagation through the linear part:
 *
 *   dx[n,ci,i,j] = sum over kept kernels (f, ci, p) of sum_t v_t *
 *                  dy[n, f, i - r_t + 1, j - s_t + 1]          (adjoint of Eq. 1)
 *   dv[k,t]      = sum over n, i, j of dy[n, f, i, j] * x[n, ci, i + r_t - 1, j + s_t - 1]
 *   db[f]        = sum over n, i, j of dy[n, f, i, j]
 *
 * dv holds the gradient of the 4 stored values of every kept kernel k (in
 * storage order): the masked gradient, nothing for pruned weights.  Terms
 * outside the image are absent.  Inputs are double (widened exactly).  dx
 * is summed per (image, input channel) over the kernels in storage order;
 * s, if non-null, receives the sum of the absolute terms. */
int pso_conv_sparse_bwd_data(const double *dy, int n, int cin, int h, int w,
                             int cout, int m, const uint16_t *masks,
                             const int32_t *filter_perm, const int32_t *filter_ptr,
                             const int32_t *cin_idx, const uint8_t *pat_id,
                             const void *values, int vdtype, double *dx, double *s)
{
    if (n < 0 || cin < 0 || h < 1 || w < 1 || cout < 0 || m < 1 || m > 126)
        return -1;
    const size_t plane = (size_t)h * w;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < (int64_t)n * cin; ++t) {
        int nn = (int)(t / cin);
        int ci = (int)(t % cin);
        double *xp = dx + ((size_t)nn * cin + ci) * plane;
        double *sp = s ? s + ((size_t)nn * cin + ci) * plane : NULL;
        for (size_t q = 0; q < plane; ++q) {
            xp[q] = 0.0;
            if (sp)
                sp[q] = 0.0;
        }
        for (int i = 0; i < cout; ++i) {
            int f = filter_perm[i];
            const double *yp = dy + ((size_t)nn * cout + f) * plane;
            for (int32_t k = filter_ptr[i]; k < filter_ptr[i + 1]; ++k) {
                if (cin_idx[k] != ci)
                    continue;
                int p = pat_id[k];
                if (p >= m) {
                    bad = 1;
                    continue;
                }
                int j = 0;
                for (int q = 0; q < 9; ++q) {
                    if (!((masks[p] >> q) & 1))
                        continue;
                    int r = q / 3, c = q % 3;
                    double v = elem(values, vdtype, (size_t)k * 4 + j);
                    j += 1;
                    /* dx[i0, j0] += v * dy[i0 - r + 1, j0 - c + 1] */
                    for (int i0 = 0; i0 < h; ++i0) {
                        int oi = i0 - r + 1;
                        if (oi < 0 || oi >= h)
                            continue;
                        for (int j0 = 0; j0 < w; ++j0) {
                            int oj = j0 - c + 1;
                            if (oj < 0 || oj >= w)
                                continue;
                            double prod = v * yp[(size_t)oi * w + oj];
                            xp[(size_t)i0 * w + j0] += prod;
                            if (sp)
                                sp[(size_t)i0 * w + j0] += fabs(prod);
                        }
                    }
                }
            }
        }
    }
    return bad ? -1 : 0;
}

/* dv (keep*4 doubles, storage order) and, if non-null, db (cout doubles,
 * original filter order); s_dv, if non-null, receives the sum of the
 * absolute terms of each dv entry.  Each entry is summed over images, then
 * rows, then columns. */
int pso_conv_sparse_bwd_weight(const double *x, const double *dy, int n, int cin, int h, int w,
                               int cout, int m, const uint16_t *masks,
                               const int32_t *filter_perm, const int32_t *filter_ptr,
                               const int32_t *cin_idx, const uint8_t *pat_id,
                               double *dv, double *s_dv, double *db)
{
    if (n < 0 || cin < 0 || h < 1 || w < 1 || cout < 0 || m < 1 || m > 126)
        return -1;
    const size_t plane = (size_t)h * w;
    int bad = 0;
    for (int i = 0; i < cout; ++i) {
        int f = filter_perm[i];
#pragma omp parallel for schedule(dynamic, 1)
        for (int32_t k = filter_ptr[i]; k < filter_ptr[i + 1]; ++k) {
            int ci = cin_idx[k];
            int p = pat_id[k];
            if (p >= m || ci < 0 || ci >= cin) {
                bad = 1;
                continue;
            }
            int j = 0;
            for (int q = 0; q < 9; ++q) {
                if (!((masks[p] >> q) & 1))
                    continue;
                int r = q / 3, c = q % 3;
                double acc = 0.0, sacc = 0.0;
                for (int nn = 0; nn < n; ++nn) {
                    const double *yp = dy + ((size_t)nn * cout + f) * plane;
                    const double *xc = x + ((size_t)nn * cin + ci) * plane;
                    for (int oi = 0; oi < h; ++oi) {
                        int ii = oi + r - 1;
                        if (ii < 0 || ii >= h)
                            continue;
                        for (int oj = 0; oj < w; ++oj) {
                            int ij = oj + c - 1;
                            if (ij < 0 || ij >= w)
                                continue;
                            double prod = yp[(size_t)oi * w + oj] * xc[(size_t)ii * w + ij];
                            acc += prod;
                            sacc += fabs(prod);
                        }
                    }
                }
                dv[(size_t)k * 4 + j] = acc;
                if (s_dv)
                    s_dv[(size_t)k * 4 + j] = sacc;
                j += 1;
            }
        }
    }
    if (db) {
        for (int f = 0; f < cout; ++f) {
            double acc = 0.0;
            for (int nn = 0; nn < n; ++nn)
                for (size_t q = 0; q < plane; ++q)
                    acc += dy[((size_t)nn * cout + f) * plane + q];
            db[f] = acc;
        }
    }
    return bad ? -1 : 0;
}

/* Witness: a textbook dense direct convolution (cross-correlation, stride 1,
 * zero padding 1) over dense OIHW weights, written independently of the
 * sparse loop above.  y is [n][cout][h][w] doubles. */
int pso_conv_dense(const void *x, int dtype, int n, int cin, int h, int w,
                   const void *wdense, int cout, const void *bias, int relu,
                   double *y)
{
    if (n < 0 || cin < 0 || h < 0 || w < 0 || cout < 0)
        return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < (int64_t)n * cout; ++t) {
        int nn = (int)(t / cout);
        int co = (int)(t % cout);
        for (int oh = 0; oh < h; ++oh) {
            for (int ow = 0; ow < w; ++ow) {
                double acc = bias ? elem(bias, dtype, (size_t)co) : 0.0;
                for (int ci = 0; ci < cin; ++ci) {
                    for (int r = 0; r < 3; ++r) {
                        for (int c = 0; c < 3; ++c) {
                            int ih = oh - 1 + r, iw = ow - 1 + c;
                            if (ih < 0 || ih >= h || iw < 0 || iw >= w)
                                continue;
                            double wv = elem(wdense, dtype, (((size_t)co * cin + ci) * 3 + r) * 3 + c);
                            double xv = elem(x, dtype, (((size_t)nn * cin + ci) * h + ih) * (size_t)w + iw);
                            acc += wv * xv;
                        }
                    }
                }
                if (relu && acc < 0.0)
                    acc = 0.0;
                y[(((size_t)nn * cout + co) * h + oh) * (size_t)w + ow] = acc;
            }
        }
    }
    return 0;
}

/* 2x2 max-pool with stride 2 on fp64 planes (the pooling between the VGG-16
 * layers).  x is [nc][h][w], y is [nc][h/2][w/2]; h and w must be even. */
int pso_maxpool2x2(const double *x, int64_t nc, int h, int w, double *y)
{
    if (nc < 0 || h < 2 || w < 2 || (h & 1) || (w & 1))
        return -1;
    for (int64_t c = 0; c < nc; ++c)
        for (int oh = 0; oh < h / 2; ++oh)
            for (int ow = 0; ow < w / 2; ++ow) {
                const double *p = x + ((size_t)c * h + 2 * oh) * (size_t)w + 2 * ow;
                double v = p[0];
                if (p[1] > v) v = p[1];
                if (p[w] > v) v = p[w];
                if (p[w + 1] > v) v = p[w + 1];
                y[((size_t)c * (h / 2) + oh) * (size_t)(w / 2) + ow] = v;
            }
    return 0;
}
