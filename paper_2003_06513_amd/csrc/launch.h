// Internal launcher interface between the C ABI (psc_api.cpp) and the HIP
// kernels.  Arguments arrive here already validated; launchers only enqueue
// work on `stream` and return the launch status.
#pragma once
#include <hip/hip_runtime_api.h>
#include <cstddef>
#include <cstdint>

namespace psc {

struct PatTable;

struct PackedView {
    const int32_t* filter_perm;
    const int32_t* filter_ptr;
    const int32_t* seg_ptr;
    const int32_t* cin_idx;
    const uint8_t* pat_id;
    const void* values;
};

struct PackedOut {
    int32_t* filter_perm;
    int32_t* filter_ptr;
    int32_t* seg_ptr;
    int32_t* cin_idx;
    uint8_t* pat_id;
    void* values;
};

// Sec. 4.3 Eq. 6
hipError_t launch_project(const PatTable& tab, int dtype, const void* w, int64_t n_kernels,
                          uint8_t* pat, double* energy, hipStream_t stream);

// Sec. 4.4
size_t select_workspace_bytes(int64_t n_kernels);
hipError_t launch_select(int64_t n_kernels, int64_t keep, const double* energy, uint8_t* keep_out,
                         void* ws, hipStream_t stream);

// The select workspace kept in the library's device code (allocates nothing):
// its size, and its address on the current device.
size_t select_scratch_bytes();
hipError_t select_scratch(void** out);

// Sec. 3.4
size_t pack_workspace_bytes(int cout, int m);
hipError_t launch_pack(const PatTable& tab, int dtype, int cout, int cin, int64_t n_keep, const void* w,
                       const uint8_t* pat, const uint8_t* keep, const PackedOut& out, void* ws,
                       hipStream_t stream);
hipError_t launch_unpack(const PatTable& tab, int dtype, int cout, int cin, int64_t keep,
                         const PackedView& pk, void* dense, hipStream_t stream);

// Sec. 4.1 Eq. 1
struct ConvArgs {
    int dtype;
    int n, cin, h, w, cout;
    int64_t keep;
    const void* x;
    const void* bias;
    int relu;
    void* y;
    int pool;       // 1: y is the 2x2/2 max-pool of sigma(conv), [n][cout][h/2][w/2]
    int stride = 1; // 1 or 2 (zero padding 1): y is [n][cout][(h-1)/stride+1][(w-1)/stride+1]
};
hipError_t launch_conv(const PatTable& tab, const PackedView& pk, const ConvArgs& a, int algo,
                       hipStream_t stream);

// The launch configuration launch_conv would use (host only, no device work).
struct ConvForm {
    int kernel;             // 0 k_conv_stream, 1 k_conv_wide, 2 k_conv_simple, 3 k_conv_stride2, 4 k_conv_rows
    int staged;             // 0 direct loads, 1 rows staged through LDS, 2 staged, several runs per wave
    int rows_per_lane, cols_per_lane, segments_per_wave, column_tiles;
    int shares, filters_per_block, blocks, threads_per_block;
};
void describe_conv(const PatTable& tab, const ConvArgs& a, int algo, ConvForm& out);
// Whether the one-row-per-lane kernel (algo 2) takes the call (host only).
bool conv_rows_takes(const PatTable& tab, const ConvArgs& a);
// Sec. 3.3 retraining: the transposed, rotated layer (for dx) and the masked
// weight gradient.
hipError_t launch_transpose_prep(int dtype, int cout, int cin, const void* w, const uint8_t* pat,
                                 const uint8_t* keep, void* wt, uint8_t* pat_t, uint8_t* keep_t,
                                 hipStream_t stream);
size_t wgrad_workspace_bytes(int n, int cin, int cout, int h, int w, int64_t nk, bool dense);
// Measurement probe: blocks x 256 lanes, each 8 x iters fp32 FMAs; out [blocks*256].
hipError_t launch_probe_fma(int blocks, int iters, float* out, hipStream_t stream);
// Measurement probe: blocks x 4 waves, each 4 chains of iters fp32 MFMA 16x16x4; out [blocks*256].
hipError_t launch_probe_mfma(int blocks, int iters, float* out, hipStream_t stream);
// Whether x and dy fit the 2 GiB a buffer descriptor addresses.
bool wgrad_fits(int n, int cin, int cout, int h, int w, int dtype);
hipError_t launch_bwd_weight(const PatTable& tab, const PackedView& pk, int dtype, int n, int cin, int h, int w,
                             int cout, int64_t keep, const void* x, const void* dy, float* dv, float* db, void* ws,
                             hipStream_t stream);

// Sec. 4.3 Eq. 4-7: the data-free ADMM pruning of one layer (fp32).
size_t admm_residual_workspace_bytes();
hipError_t launch_admm_residual(const float* z, const float* t, int64_t numel, float scale, float* g,
                                double* loss, void* ws, hipStream_t stream);
hipError_t launch_dense_wgrad(const float* x, const float* g, int n, int cin, int h, int w, int cout, float* dw,
                              float* db, void* ws, hipStream_t stream);
// The dense weight gradient on the matrix cores (layers of at least 16 input
// channels): blocks of 64 filters x 16 channels, the 4x16 pixel tiles split
// over KS blocks with KS partial-sum slots in the workspace.
struct DenseWPlan {
    int fb, cb;             // filter and channel blocks
    int tiles_w, tiles_img; // pixel tiles per image row of tiles, per image
    int64_t tiles;          // pixel tiles in all
    int KS;                 // blocks the tiles are split over
};
bool dense_wgrad_mfma_plan(int n, int cin, int cout, int h, int w, DenseWPlan* p);
size_t dense_wgrad_mfma_workspace(const DenseWPlan& p, int cin, int cout);
hipError_t launch_dense_wgrad_mfma(const DenseWPlan& p, int dtype, const void* x, const void* g, int n, int cin,
                                   int h, int w, int cout, float* dst, hipStream_t stream);
// The masked gradient of the stored kernels taken from a dense dw [cout][cin][9].
hipError_t launch_gather_masked(const PatTable& tab, const PackedView& pk, int cout, int cin, const float* dw,
                                float* dv, hipStream_t stream);
hipError_t launch_admm_primal(float* w, const float* dw, const float* a, const float* d, int64_t nw, float* b,
                              const float* db, int cout, float lr, float rho, float* v, hipStream_t stream);
hipError_t launch_admm_dual(const PatTable& tab, const float* v, const uint8_t* pat, const uint8_t* keep, int64_t nk,
                            float* a, float* d, hipStream_t stream);

hipError_t launch_dense(int dtype, const void* x, int n, int cin, int h, int w, const void* wd,
                        int cout, const void* bias, int relu, void* y, hipStream_t stream);
hipError_t launch_maxpool(int dtype, const void* x, int n, int c, int h, int w, void* y,
                          hipStream_t stream);

}  // namespace psc
