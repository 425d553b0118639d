/*
 * psc.h -- pattern-sparse 3x3 convolution for AMD MI355X (gfx950).
 *
 * A C ABI over hand-written HIP kernels implementing the inference path of
 * Gong et al., "A Privacy-Preserving-Oriented DNN Pruning and Mobile
 * Acceleration Framework" (GLSVLSI'20):
 *
 *   psc_select_library  pattern-library heuristic                 Sec. 4.2
 *   psc_project         projection of each kernel onto the
 *                       pattern set C_n                           Sec. 4.3, Eq. 6
 *   psc_select          connectivity pruning (constraint C'_n)    Sec. 4.4
 *   psc_pack            filter kernel reorder + compressed
 *                       weight storage                            Sec. 3.4
 *   psc_conv3x3_fwd     the pruned layer X_n = sigma(W_n X + b_n) Sec. 4.1, Eq. 1
 *
 * plus a dense comparator, a dense unpacker and the 2x2 max-pool of the
 * VGG-16 stack.
 *
 * Conventions for every entry point:
 *  - "d_" pointers are device memory, "h_" pointers host memory; all of it is
 *    owned and allocated by the caller.  The library never allocates or frees
 *    device memory and never synchronises a stream: work is enqueued on
 *    `stream` (a hipStream_t, NULL = the null stream) and the caller keeps
 *    every buffer alive until that stream has drained it.
 *  - Weights are contiguous OIHW [cout][cin][3][3]; activations contiguous
 *    NCHW.  Masks are 9-bit codes, bit 3r+s for kernel row r, column s.
 *  - Arguments are validated synchronously, before any HIP call, so errors
 *    are reported the same way with or without a device.  A failed launch is
 *    returned as PSC_ERR_DEVICE.  No C++ exception crosses the ABI.
 *  - On any status other than PSC_OK, psc_last_error() returns a message for
 *    the calling thread.  The library keeps no other global mutable state.
 */
#ifndef PSC_H
#define PSC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PSC_MAX_PATTERNS 126      /* C(9,4): every distinct 4-of-9 mask */
#define PSC_MAX_LIBRARY_HEURISTIC 56 /* C(8,3): centre + 3 neighbours */

typedef enum {
    PSC_OK = 0,
    PSC_ERR_ARG = 1,          /* a null pointer, bad size, bad mask, ... */
    PSC_ERR_UNSUPPORTED = 2,  /* a valid request the library does not run */
    PSC_ERR_WORKSPACE = 3,    /* workspace pointer missing or too small */
    PSC_ERR_DEVICE = 4,       /* a HIP call or kernel launch failed */
    PSC_ERR_INTERNAL = 5
} psc_status;

typedef enum { PSC_F32 = 0, PSC_F16 = 1 } psc_dtype;

/* Operations that take a workspace (psc_workspace_size). */
typedef enum { PSC_OP_SELECT = 0, PSC_OP_PACK = 1 } psc_op;

/* The per-layer representation the compiler optimisations work on (Sec. 3.4:
 * layer shape, pattern style, connectivity).  Plain data, host memory. */
typedef struct psc_layer {
    int32_t cout;       /* output channels (filters), >= 1 */
    int32_t cin;        /* input channels, >= 1 */
    int32_t m;          /* pattern-library size, 1..PSC_MAX_PATTERNS (Sec. 3.2) */
    int32_t wdtype;     /* psc_dtype of weights (and of activations) */
    int64_t keep;       /* beta_n (Sec. 4.4): exact number of kernels kept,
                           0..cout*cin */
    uint16_t masks[PSC_MAX_PATTERNS]; /* masks[0..m-1]: pairwise distinct
                           9-bit codes with exactly 4 bits set (Sec. 3.2) */
} psc_layer;

/* Compressed weight storage (Sec. 3.4), device pointers, caller-owned.
 * Filters appear in reordered position i = 0..cout-1; inside a filter, kept
 * kernels are sorted by (pattern id ascending, input channel ascending).
 * Sizes follow from (cout, m, keep) alone. */
typedef struct psc_packed {
    int32_t *filter_perm; /* [cout]          reordered position -> original filter */
    int32_t *filter_ptr;  /* [cout+1]        first kernel of position i; [cout] = keep */
    int32_t *seg_ptr;     /* [cout*(m+1)]    seg_ptr[i*(m+1)+p]: first kernel of
                                              pattern p in position i;
                                              seg_ptr[i*(m+1)+m] = filter_ptr[i+1] */
    int32_t *cin_idx;     /* [keep]          input channel of each kept kernel */
    uint8_t *pat_id;      /* [keep]          library index of each kept kernel */
    void *values;         /* [keep*4]        the 4 kept weights in ascending
                                              3r+s order, wdtype; 16-byte aligned */
} psc_packed;

/* Message for the last failure on the calling thread ("" if none). */
const char *psc_last_error(void);
/* Constant name of a status code. */
const char *psc_status_string(psc_status s);
/* ABI version; bumped on any incompatible change. */
int32_t psc_abi_version(void);

/* Sec. 4.2: for each of the n_kernels 3x3 kernels in h_w (host, dtype),
 * take the positions of its 3 largest-magnitude non-centre weights (ties to
 * the lower position) plus the centre; the library is the m codes that occur
 * most often, ordered by count descending then code ascending, filled with
 * unseen centre+3 codes in ascending order.  Host only, no device work.
 * m must be 1..PSC_MAX_LIBRARY_HEURISTIC.  h_masks_out receives m codes. */
psc_status psc_select_library(const void *h_w, int32_t dtype, int64_t n_kernels,
                              int32_t m, uint16_t *h_masks_out);

/* Bytes of device workspace `op` needs for `layer` (0 is a valid answer).
 * The workspace must be 256-byte aligned. */
psc_status psc_workspace_size(const psc_layer *layer, int32_t op, size_t *bytes);

/* Sec. 4.3, Eq. 6: projection of every kernel of d_w (cout*cin kernels) onto
 * the pattern set.  For kernel k and library pattern p the energy is the fp64
 * sum of the squares of the 4 kept weights, added in ascending position
 * order; d_pat[k] is the first p of largest energy and d_energy[k] that
 * energy.  Bit-exact and deterministic.  layer->keep is not read. */
psc_status psc_project(const psc_layer *layer, const void *d_w, uint8_t *d_pat,
                       double *d_energy, void *stream);

/* Sec. 4.4: connectivity pruning.  d_keep[k] = 1 for exactly layer->keep
 * kernels -- the largest energies, equal energies broken by the lower flat
 * index k = co*cin+ci -- and 0 otherwise.  Energies must be non-negative
 * (as psc_project writes them).  Needs PSC_OP_SELECT workspace. */
psc_status psc_select(const psc_layer *layer, const double *d_energy,
                      uint8_t *d_keep, void *d_ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: psc_select
 * without a workspace argument, with the same results.  Its scratch is a
 * 64 KiB array in the library's device code, one per GPU, held until the
 * process ends; the call allocates nothing.  Layers of more than
 * PSC_SELECT_NOALLOC_MAX_KERNELS kernels (cout*cin) return
 * PSC_ERR_UNSUPPORTED before any HIP call.  Every call on a GPU uses that
 * GPU's one array: calls whose work may overlap on one GPU (on different
 * streams, or from concurrent host threads) race, and the caller must order
 * them.  stream must belong to the current device. */
#define PSC_SELECT_NOALLOC_MAX_KERNELS 16449536   /* (64 KiB - 1280 B) / 4 B x 1024 */
psc_status psc_select_noalloc(const psc_layer *layer, const double *d_energy,
                              uint8_t *d_keep, void *stream);

/* Sec. 3.4: filter kernel reorder + compressed weight storage.  Filters are
 * ordered by (kept-kernel count descending, per-pattern counts
 * lexicographically descending, filter index ascending); values are bit
 * copies of d_w.  d_keep must hold exactly layer->keep ones, d_pat entries
 * must be < m (else the result is undefined).  Needs PSC_OP_PACK workspace.
 * Every array of *out is written. */
psc_status psc_pack(const psc_layer *layer, const void *d_w, const uint8_t *d_pat,
                    const uint8_t *d_keep, const psc_packed *out, void *d_ws,
                    size_t ws_bytes, void *stream);

/* Compressed storage -> dense OIHW weights in the original filter order,
 * zeros outside the kept patterns (bit copies of the stored values). */
psc_status psc_unpack_dense(const psc_layer *layer, const psc_packed *packed,
                            void *d_w_dense, void *stream);

/* Sec. 4.1, Eq. 1: y = sigma(W x + b) for the pruned 3x3 layer, stride 1,
 * zero padding 1, cross-correlation:
 *   y[n,f,h,w] = b[f] + sum over kept kernels (ci, p) of filter f of
 *                sum_j v_j * x[n, ci, h + r_j - 1, w + s_j - 1]
 * with sigma = ReLU when relu != 0.  d_x is [n][cin][h][w], d_y is
 * [n][cout][h][w] in the original filter order, both of dtype act_dtype,
 * which must equal layer->wdtype.  fp16 data is accumulated in fp32 and the
 * result rounded to nearest-even once.  d_bias ([cout], same dtype) may be
 * NULL.  d_y must not overlap d_x.  n == 0 is a no-op. */
psc_status psc_conv3x3_fwd(const psc_layer *layer, const psc_packed *packed,
                           int32_t act_dtype, const void *d_x, int32_t n,
                           int32_t h, int32_t w, const void *d_bias,
                           int32_t relu, void *d_y, void *stream);

/* Same as psc_conv3x3_fwd with an explicit kernel choice: algo 0 = the
 * default tuned kernels (chosen from the shape), 1 = the simple
 * one-output-per-lane kernel (kept as a second implementation for testing),
 * 2 = the one-row-per-lane kernel, which algo 0 picks for batches that fill
 * a wave with whole images on planes of at most 16 columns, 3 = the
 * column-per-lane tuned kernels (algo 0 without that choice).  Algo 2 needs
 * no pool, at most 63 output rows and w in {4, 7, 8, 14, 16, 28} (fp16: w
 * even, or 7); with stride 2 (psc_conv3x3_fwd_strided) w in {8, 16, 32};
 * else PSC_ERR_UNSUPPORTED. */
psc_status psc_conv3x3_fwd_algo(const psc_layer *layer, const psc_packed *packed,
                                int32_t act_dtype, const void *d_x, int32_t n,
                                int32_t h, int32_t w, const void *d_bias,
                                int32_t relu, void *d_y, int32_t algo, void *stream);

/* Sec. 4.1, Eq. 1 followed by the 2x2/2 max-pool of the VGG-16 stack, in
 * one pass: d_y [n][cout][h/2][w/2] (original filter order) receives
 *   y[n,f,i,j] = max over a,b in {0,1} of sigma(conv(x)[n,f,2i+a,2j+b] + b[f])
 * with conv and sigma as in psc_conv3x3_fwd; the un-pooled output is never
 * written.  h and w must be even.  algo as in psc_conv3x3_fwd_algo.  d_y must
 * not overlap d_x. */
psc_status psc_conv3x3_fwd_pool2(const psc_layer *layer, const psc_packed *packed,
                                 int32_t act_dtype, const void *d_x, int32_t n,
                                 int32_t h, int32_t w, const void *d_bias,
                                 int32_t relu, void *d_y, int32_t algo, void *stream);

/* Sec. 4.1, Eq. 1 with a stride, for the stage-entry convolutions of the
 * ResNets the paper prunes: 3x3, zero padding 1, stride 1 or 2.  d_y is
 * [n][cout][OH][OW] (original filter order), OH = (h-1)/stride + 1,
 * OW = (w-1)/stride + 1, and
 *   y[n,f,i,j] = sigma(b[f] + sum over kept (ci, p) of f of
 *                sum_{(r,s) in p} v * x[n, ci, stride*i + r - 1, stride*j + s - 1])
 * with out-of-image taps reading zero.  stride 1 is psc_conv3x3_fwd_algo.
 * Stride 2 with algo 0 runs the one-row-per-lane kernel when the batch
 * fills a wave with whole images of 8 columns, or of 16 x 16 in fp32;
 * otherwise, and always with algo 3, the tuned stride-2 kernel for even
 * widths of at most 126 columns (the one-output-per-lane kernel otherwise,
 * and always with algo 1); algo 2 the one-row-per-lane kernel.  Other
 * conventions and errors as in psc_conv3x3_fwd_algo; a stride other than 1
 * or 2 returns PSC_ERR_ARG. */
psc_status psc_conv3x3_fwd_strided(const psc_layer *layer, const psc_packed *packed,
                                   int32_t act_dtype, const void *d_x, int32_t n,
                                   int32_t h, int32_t w, const void *d_bias,
                                   int32_t relu, void *d_y, int32_t stride, int32_t algo,
                                   void *stream);

/* ---- Retraining (Sec. 3.3): the user retrains the pruned model like a
 * dense one, except that the gradients of pruned weights are zero.  For the
 * layer y = W x of psc_conv3x3_fwd (before sigma; dy is the gradient at
 * that point):
 *
 *   dx = W^T dy  is a pattern-sparse 3x3 convolution of dy by the transposed
 *                layer: filter ci, input channel f, every kernel rotated by
 *                180 degrees.  psc_transpose_layer describes that layer (a
 *                rotated 4-of-9 mask is a 4-of-9 mask, library order kept),
 *                psc_transpose_prep writes its dense weights, pattern ids
 *                and keep mask, psc_pack packs it, and psc_conv3x3_fwd (or
 *                _algo) on dy gives dx;
 *   dv, db       are the masked gradient: psc_conv3x3_bwd_weight. */

/* Host only: *out = the transposed layer of *layer (cout and cin swapped,
 * masks[p] rotated: bit q -> bit 8-q, same keep and dtype). */
psc_status psc_transpose_layer(const psc_layer *layer, psc_layer *out);

/* The transposed layer's dense inputs to psc_pack: for kernel k = f*cin+ci
 * of layer, kt = ci*cout+f, d_w_t[kt][q] = d_w[k][8-q] (bit copies, OIHW of
 * the transposed layer), d_pat_t[kt] = d_pat[k], d_keep_t[kt] = d_keep[k].
 * Outputs must not overlap inputs. */
psc_status psc_transpose_prep(const psc_layer *layer, const void *d_w, const uint8_t *d_pat,
                              const uint8_t *d_keep, void *d_w_t, uint8_t *d_pat_t,
                              uint8_t *d_keep_t, void *stream);

/* The masked weight gradient of the layer for output gradient d_dy
 * ([n][cout][h][w], act_dtype; d_x [n][cin][h][w] the layer's input):
 *   d_dvalues[4k+t] = sum over images and pixels (i, j) of
 *                     dy[n, f, i, j] * x[n, ci, i + r_t - 1, j + s_t - 1]
 * for every kept kernel k of the storage (filter f, channel ci, t-th kept
 * position (r_t, s_t)), and, if d_dbias is non-NULL,
 *   d_dbias[f] = sum over images and pixels of dy[n, f].
 * Outputs are fp32 (fp32 accumulation for both activation dtypes), written
 * in full; d_dvalues [keep*4] must be 16-byte aligned, d_dbias is [cout] in
 * the original filter order.  Stride 1, zero padding 1.  The batch and the
 * image may be split over several waves per kernel; their sums meet in the
 * caller's workspace (psc_conv3x3_bwd_weight_workspace bytes, may be 0) and
 * are added in a fixed order, so results are reproducible bit for bit.
 * x and dy of more than 2 GiB each return PSC_ERR_UNSUPPORTED. */
psc_status psc_conv3x3_bwd_weight_workspace(const psc_layer *layer, int32_t act_dtype, int32_t n,
                                            int32_t h, int32_t w, size_t *bytes);
psc_status psc_conv3x3_bwd_weight(const psc_layer *layer, const psc_packed *packed,
                                  int32_t act_dtype, const void *d_x, const void *d_dy,
                                  int32_t n, int32_t h, int32_t w, float *d_dvalues,
                                  float *d_dbias, void *d_ws, size_t ws_bytes, void *stream);

/* ---- Data-free ADMM pattern pruning of one layer (Sec. 4.3, Eq. 4-7;
 * Algorithm 1).  With input X (synthetic data), pre-trained W0, b0 and
 * target X' = relu(W0 X + b0) (psc_dense3x3_fwd with relu), an iteration is
 *   Z = W X + b                           psc_dense3x3_fwd, relu off
 *   G, loss = c ||relu(Z) - X'||^2        psc_admm_residual
 *   dW, db                                psc_dense3x3_bwd_weight
 *   W -= lr (dW + rho (W - A + D)),
 *   b -= lr db, V = W + D                 psc_admm_primal            (Eq. 4)
 *   pattern ids + energies of V           psc_project                (Eq. 6)
 *   keep mask (beta kernels)              psc_select or _noalloc     (Sec. 4.4)
 *   A = V on the kept pattern positions,
 *   0 elsewhere; D = V - A                psc_admm_dual        (Eq. 6, Eq. 7)
 * starting from A = W0, D = 0.  All tensors fp32, weights OIHW, activations
 * NCHW, each rounding as written (the loss sums in fp64). */

/* G[i] = 2 scale (relu(z[i]) - t[i]) if z[i] > 0, else 0; *d_loss (device
 * double) = scale * sum (relu(z) - t)^2, summed in fp64 in a fixed order.
 * d_ws: PSC_ADMM_RESIDUAL_WS_BYTES bytes, 256-byte aligned, caller-owned. */
#define PSC_ADMM_RESIDUAL_WS_BYTES 8192
psc_status psc_admm_residual(const float *d_z, const float *d_target, int64_t numel, float scale,
                             float *d_g, double *d_loss, void *d_ws, size_t ws_bytes, void *stream);

/* The dense weight gradient of the 3x3 layer (stride 1, zero padding 1):
 *   d_dw[o][i][r][s] = sum over images and pixels of
 *                      g[n, o, h, w] * x[n, i, h + r - 1, w + s - 1]
 * and, if d_db is non-NULL, d_db[o] = sum of g[n, o, :, :]; fp32.  Layers of
 * at least 16 input channels run on the matrix cores (fp32 MFMA), the others
 * on the vector ALUs; partial sums are added in a fixed order, so results
 * are deterministic.  Workspace as for psc_conv3x3_bwd_weight
 * (psc_dense3x3_bwd_weight_workspace bytes); x and g of more than 2 GiB
 * each return PSC_ERR_UNSUPPORTED. */
psc_status psc_dense3x3_bwd_weight_workspace(int32_t n, int32_t cin, int32_t h, int32_t w,
                                             int32_t cout, size_t *bytes);
psc_status psc_dense3x3_bwd_weight(const float *d_x, const float *d_g, int32_t n, int32_t cin,
                                   int32_t h, int32_t w, int32_t cout, float *d_dw, float *d_db,
                                   void *d_ws, size_t ws_bytes, void *stream);

/* Eq. 4, one SGD step, in place: for each of the n_weights entries
 *   W = W - lr * (dW + rho * ((W - A) + D)),   V = W + D;
 * and, if d_b is non-NULL, b[o] = b[o] - lr * db[o] for o < cout. */
psc_status psc_admm_primal(int64_t n_weights, float *d_w, const float *d_dw, const float *d_a,
                           const float *d_d, int32_t cout, float *d_b, const float *d_db,
                           float lr, float rho, float *d_v, void *stream);

/* Eq. 6-7 given the projection's choices for V (d_pat from psc_project on
 * V, d_keep from psc_select): A = V at the positions of kept kernels' chosen
 * patterns, +0 elsewhere; D = V - A.  layer->wdtype must be PSC_F32. */
psc_status psc_admm_dual(const psc_layer *layer, const float *d_v, const uint8_t *d_pat,
                         const uint8_t *d_keep, float *d_a, float *d_d, void *stream);

/* The launch configuration the conv entry points would use for a call with
 * these arguments: which kernel runs and how work maps onto it.  Host only,
 * no device work; arguments are validated as by psc_conv3x3_fwd_strided
 * (pool != 0 as by psc_conv3x3_fwd_pool2, which needs stride 1), except that
 * no pointer is needed.  Meant for tests and benchmark reports. */
typedef struct psc_conv_config {
    int32_t kernel;            /* 0: tuned kernel, one output column per lane
                                  1: tuned kernel, 4 output columns per lane
                                  2: one-output-per-lane kernel
                                  3: stride-2 kernel, 1 output column per lane
                                     (2 when w is a multiple of 4)
                                  4: one output row per lane (all w columns) */
    int32_t staged;            /* 0: input rows loaded straight into registers,
                                  1: staged through LDS, one run per wave
                                     (kernel 4: the wave's whole planes),
                                  2: staged through LDS, several runs per wave */
    int32_t rows_per_lane;     /* output rows per lane */
    int32_t cols_per_lane;     /* output columns per lane */
    int32_t segments_per_wave; /* row bands (or column tiles, or images) per wave */
    int32_t column_tiles;      /* column tiles per image row (1: full rows) */
    int32_t shares;            /* waves that split one filter's kernels */
    int32_t filters_per_block;
    int32_t blocks;
    int32_t threads_per_block;
} psc_conv_config;

psc_status psc_conv3x3_config(const psc_layer *layer, int32_t act_dtype, int32_t n,
                              int32_t h, int32_t w, int32_t pool, int32_t stride,
                              int32_t algo, psc_conv_config *out);

/* Comparator, and the dense layer of the ADMM loop: the dense 3x3
 * convolution (stride 1, pad 1) of dense OIHW weights d_w [cout][cin][3][3],
 * same conventions as psc_conv3x3_fwd, fp32 accumulation (fp16 inputs
 * widened exactly).  Layers of more than 8 input channels run on the matrix
 * cores (fp32 MFMA), the others on the vector ALUs. */
psc_status psc_dense3x3_fwd(int32_t dtype, const void *d_x, int32_t n, int32_t cin,
                            int32_t h, int32_t w, const void *d_w, int32_t cout,
                            const void *d_bias, int32_t relu, void *d_y, void *stream);

/* 2x2 max-pool, stride 2 (the pooling of the VGG-16 stack): d_x
 * [n][c][h][w] -> d_y [n][c][h/2][w/2]; h and w must be even. */
psc_status psc_maxpool2x2(int32_t dtype, const void *d_x, int32_t n, int32_t c,
                          int32_t h, int32_t w, void *d_y, void *stream);

/* Measurement probe, not part of the method: blocks x 256 lanes each run 8
 * independent chains of iters fp32 FMAs (v_fmac_f32; the library is compiled
 * with packed fp32 disabled) and store one sum to d_out [blocks*256] (fp32, device).
 * Timing it gives the vector-ALU FMA rate the conv kernels can reach:
 * 2 * 8 * iters * blocks * 256 flops.  blocks in 1..2^20, iters >= 0. */
psc_status psc_probe_fma(int32_t blocks, int32_t iters, float *d_out, void *stream);

/* Measurement probe, not part of the method: blocks x 4 waves each run 4
 * independent chains of iters fp32 MFMA 16x16x4 (the instruction of the
 * dense conv and dense weight gradient), with A all 1 and B all 1/4, so each
 * MFMA adds exactly 1 to each result; d_out [blocks*256] (fp32, device)
 * receives per lane the sum of its 16 results, 16 * iters.  Timing it gives
 * the matrix-core rate those kernels can reach: 32768 * iters * blocks
 * flops.  blocks in 1..2^20, iters >= 0. */
psc_status psc_probe_mfma(int32_t blocks, int32_t iters, float *d_out, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* PSC_H */
