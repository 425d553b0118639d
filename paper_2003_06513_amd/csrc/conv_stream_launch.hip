// Launch configuration of the tuned pattern-sparse 3x3 convolution (Sec. 4.1
// Eq. 1): lane layout, rows per lane, filter shares and load form are chosen
// here on the host; the kernels are the templates of conv_stream.h, each
// instantiation set compiled in its own translation unit (conv_stream_*.hip).
#include <cstring>

#include "conv_stream.h"

namespace psc {
using namespace cs;

#define PSC_EXTERN_R(DT, R) \
    extern template hipError_t cs::launch_r<DT, R>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
PSC_EXTERN_R(DT_F32, 2)
PSC_EXTERN_R(DT_F32, 4)
PSC_EXTERN_R(DT_F32, 7)
PSC_EXTERN_R(DT_F32, 8)
PSC_EXTERN_R(DT_F16, 2)
PSC_EXTERN_R(DT_F16, 4)
PSC_EXTERN_R(DT_F16, 7)
PSC_EXTERN_R(DT_F16, 8)
#undef PSC_EXTERN_R
extern template hipError_t cs::launch_wide<DT_F32, 4>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
extern template hipError_t cs::launch_wide<DT_F16, 4>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);

// Grids of at least this many waves are throughput-bound (16 waves per SIMD).
constexpr int64_t kManyWaves = 16384;
// Filters are split into more shares while the grid holds fewer waves.
constexpr int64_t kSplitWaves = 4096;

// Note on R = 8 with several segments per wave: launches of the direct form
// with R = 8 and 3 or 7 full-row segments per wave (the batch-256 CIFAR
// layers 128@16 and 256@8) once faulted the device.  Every load of x and
// the metadata in that form is range-checked by its buffer descriptor and
// every store index was checked on the host for those launches, so the cause
// is not known; the launcher never picks R = 8 when a wave holds more than
// one segment.
//
// Launch configuration.  Rows per lane R minimise the lane-rows loaded
// (ceil(units / S) * (R + 2)) in throughput-bound grids, the lane-rows
// issued (ceil(units / S) * R) otherwise, larger R on ties (7 over 8 for
// staged single-segment grids of long kernel chains); even R when
// pooling; R = 8 only with one segment per wave.  A workgroup holds 4
// filters, or fewer filters split into KS shares (KS doubles up to 8) while
// the grid holds under 4 waves per SIMD.  Returns false when the tuned kernels do not
// take the call: x beyond the 2 GiB a buffer descriptor addresses here, or a
// pooled output of haloed column tiles.  Host only.
bool plan_conv_stream(const PatTable& tab, const ConvArgs& a, Geo& g) {
    const int64_t x_bytes = int64_t(a.n) * a.cin * a.h * a.w * (a.dtype == DT_F16 ? 2 : 4);
    // buffer descriptors address at most 2 GiB (x) and the packed weights
    if (x_bytes >= (int64_t(1) << 31) || a.keep * 4 * (a.dtype == DT_F16 ? 2 : 4) > 0x7fffffff)
        return false;
    std::memset(&g, 0, sizeof g);
    g.n = a.n;
    g.cin = a.cin;
    g.H = a.h;
    g.W = a.w;
    g.cout = a.cout;
    g.m = tab.m;
    g.relu = a.relu;
    g.x_bytes = int(x_bytes);
    g.keep = int(a.keep);
    g.pool = a.pool;
    for (int p = 0; p < kMaxPatterns; ++p) {
        g.shape[p] = -1;
        g.mask[p] = p < tab.m ? tab.mask[p] : 0;
        if (p < tab.m)
            for (int t = 0; t < 56; ++t)
                if (kCentre3.code[t] == tab.mask[p]) g.shape[p] = int8_t(t);
    }
    // wide form (4 columns per lane, 4 rows): widths 28..252, multiples of 4,
    // segments padded to a multiple of 4 lanes.  Taken for fp32 rows of 64+
    // columns on 64-byte boundaries (faster at batch 1 too), and otherwise
    // when the grid is large enough to be bound by the vector-memory path
    // rather than by the latency of each wave's kernel chain: there 4 columns
    // per load instruction beat 1 (32x32 fp32 at batch 256: 2.1x; 56x56 fp16
    // at batch 32: 1.2x).
    if (a.w % 4 == 0 && a.w >= 28 && a.w / 4 + 1 <= 64) {
        constexpr int R = 4;
        const int seg_len = (a.w / 4 + 1 + 3) / 4 * 4;
        const int S = 64 / seg_len;
        const int RB = (a.h + R - 1) / R;
        const int64_t U = int64_t(a.n) * RB;
        const int64_t sgroups = (U + S - 1) / S;
        const bool aligned64 = a.dtype == DT_F32 && a.w % 16 == 0 && a.w >= 64;
        // fp32 rows of 28 columns: a wave holds whole 28-row images (8 bands
        // of 4 rows); where 8 shares of each filter make about 4096 waves
        // (deep layers at small batch) the wide form takes them.  Measured
        // on the batch-1 VGG-16 28x28 layers: 8 shares beat the one-column
        // staged form by 6-8 % (2 shares lose).
        const bool rows28 = a.dtype == DT_F32 && a.w == 28 && a.cin >= 16 * kMaxSplit &&
                            sgroups * a.cout * kMaxSplit >= 4096;
        if (aligned64 || rows28 || sgroups * a.cout >= kWideMinWaves) {
            g.cols_mode = 0;
            g.seg_len = seg_len;
            g.S = S;
            g.Wt = a.w;
            g.CT = 1;
            g.RB = RB;
            g.U = int(U);
            // shares only below about one wave per SIMD (at 112-224 columns
            // one share measured fastest)
            g.KS = 1;
            const int64_t target = rows28 && sgroups * a.cout < kWideMinWaves ? 4096 : 1024;
            while (g.KS < kMaxSplit && sgroups * a.cout * g.KS < target && a.cin >= 16 * g.KS) g.KS *= 2;
            g.FW = g.KS >= 4 ? 1 : 4 / g.KS;
            if (g.FW > a.cout) g.FW = a.cout;
            g.groups_x = (a.cout + g.FW - 1) / g.FW;
            g.nblocks = int(g.groups_x * sgroups);
            g.R = R;
            g.form = 1;
            return true;
        }
    }
    // lane layout: full-row segments if they use the lanes at least as well
    // as haloed column tiles
    const int S_rows = a.w <= 63 ? 65 / (a.w + 1) : 0;
    const int use_rows = S_rows * a.w;
    int ct = (a.w + 61) / 62, use_cols = 0;
    for (int t = ct; t <= a.w && t <= 64; ++t) {
        const int wt = (a.w + t - 1) / t;
        const int use = (64 / (wt + 2)) * a.w / t;
        if (use > use_cols) {
            use_cols = use;
            ct = t;
        }
    }
    if (S_rows > 0 && use_rows >= use_cols) {
        g.cols_mode = 0;
        g.S = S_rows;
        g.seg_len = a.w + 1;
        g.Wt = a.w;
        g.CT = 1;
    } else {
        if (a.pool) return false;   // pooling needs full-row segments
        const int Wt = (a.w + ct - 1) / ct;
        g.cols_mode = 1;
        g.S = 64 / (Wt + 2);
        g.seg_len = Wt + 2;
        g.Wt = Wt;
        g.CT = ct;
    }
    // rows per lane.  A grid of many waves (throughput-bound) is limited by
    // the rows a lane loads, R + 2 per R output rows, so its cost counts
    // loaded rows; a small grid (batch 1) is limited by the per-kernel
    // latency of its waves, so its cost counts output rows.
    const int cand[4] = {8, 7, 4, 2};
    int R = 8;
    int64_t best = -1;
    const int64_t units4 = int64_t(a.n) * ((a.h + 3) / 4) * g.CT;
    const bool many_waves = (units4 + g.S - 1) / g.S * a.cout >= kManyWaves;
    // 8 rows per lane only with one segment per wave (see the note on R = 8
    // above)
    // filters with long kernel chains (32 or more kept kernels) on one
    // full-row segment per wave run staged (below); there R = 7 beats R = 8
    // at the same cost (one more band, more waves)
    const bool long_chains = a.cout > 0 && a.keep >= 32 * int64_t(a.cout);
    const bool prefer_small = !g.cols_mode && g.S == 1 && long_chains;
    for (int rr : cand) {
        if (a.pool && (rr & 1)) continue;               // pooled rows pair up inside a lane
        if (rr == 8 && g.S > 1) continue;
        const int64_t units = int64_t(a.n) * ((a.h + rr - 1) / rr) * g.CT;
        const int64_t cost = (units + g.S - 1) / g.S * (many_waves ? rr + 2 : rr);
        if (best < 0 || cost < best || (prefer_small && cost == best && rr == 7 && R == 8)) {
            best = cost;
            R = rr;
        }
    }
    g.RB = (a.h + R - 1) / R;
    g.U = a.n * g.RB * g.CT;
    const int sgroups = (g.U + g.S - 1) / g.S;
    g.KS = 1;
    while (g.KS < kMaxSplit && int64_t(sgroups) * a.cout * g.KS < kSplitWaves && a.cin >= 16 * g.KS) g.KS *= 2;
    if (prefer_small && g.KS > 2) g.KS = 2;   // staged long chains: 2 shares measured best
    g.FW = g.KS >= 4 ? 1 : 4 / g.KS;
    if (g.FW > a.cout) g.FW = a.cout;
    const int fgroups = (a.cout + g.FW - 1) / g.FW;
    g.groups_x = fgroups;
    g.nblocks = fgroups * sgroups;
    // LDS staging for full-row segments: runs per wave (images its segments
    // touch) and the LDS bytes of the largest run
    if (!g.cols_mode) {
        const int esz = a.dtype == DT_F16 ? 2 : 4;
        int nruns_max = 0, bytes_max = 0;
        for (int sg = 0; sg < sgroups; ++sg) {
            const int uf = sg * g.S, ul = (uf + g.S < g.U ? uf + g.S : g.U) - 1;
            const int nf = uf / g.RB, nl = ul / g.RB;
            nruns_max = nruns_max > nl - nf + 1 ? nruns_max : nl - nf + 1;
            for (int n = nf; n <= nl; ++n) {
                const int ua = uf > n * g.RB ? uf : n * g.RB;
                const int ub = ul < n * g.RB + g.RB - 1 ? ul : n * g.RB + g.RB - 1;
                int lo = (ua - n * g.RB) * R - 1, hi = (ub - n * g.RB + 1) * R + 1;
                lo = lo < 0 ? 0 : lo;
                hi = hi > a.h ? a.h : hi;
                const int bytes = (hi - lo) * a.w * esz;
                bytes_max = bytes_max > bytes ? bytes_max : bytes;
            }
        }
        // a run's copy spans [data - 63, data + bytes + 1024) around its data
        g.region = (64 + bytes_max + 1024 + 63) / 64 * 64;
        // copy 0: the runs, then 64 zero bytes; copy 1 kLdsCopy bytes later
        g.wave_bytes = kLdsCopy + nruns_max * g.region + 64;
        // fp16 copies shift the LDS destination in 4-byte steps only: rows of
        // even width keep every offset a multiple of 4 bytes
        const bool fits = (bytes_max + 63 + 1023) / 1024 <= kMaxDma && nruns_max <= kMaxRuns &&
                          nruns_max * g.region + 64 <= kLdsCopy &&
                          int64_t(g.FW) * g.KS * g.wave_bytes <= 64 * 1024 &&
                          (a.dtype != DT_F16 || a.w % 2 == 0);
        // one full-row segment per wave and a grid of about one round of
        // waves (batch 1 at W >= 32) is bound by the per-kernel latency,
        // which the direct loads keep shorter -- unless each filter has a
        // long chain of kernels, where the staged copies run ahead better
        // (measured on the 56x56 VGG-16 layers at batch 1)
        const int64_t waves = int64_t(sgroups) * a.cout * 4;   // at 4 shares per filter
        const bool throughput = g.S >= 2 || waves >= 2 * 6 * 1024 || long_chains;
        g.lds = fits && throughput ? 1 : 0;
        if (g.lds && nruns_max > 1) g.lds = 2;             // several runs per wave: the general form
    }
    g.R = R;
    g.form = 0;
    return true;
}

hipError_t launch_conv_stream(const PatTable& tab, const PackedView& pk, const ConvArgs& a,
                              hipStream_t stream) {
    Geo g;
    if (!plan_conv_stream(tab, a, g)) return hipErrorNotSupported;
    if (g.form == 1) return a.dtype == DT_F16 ? launch_wide<DT_F16, 4>(pk, a, g, stream)
                                              : launch_wide<DT_F32, 4>(pk, a, g, stream);
    switch (g.R) {
        case 8: return a.dtype == DT_F16 ? launch_r<DT_F16, 8>(pk, a, g, stream)
                                         : launch_r<DT_F32, 8>(pk, a, g, stream);
        case 7: return a.dtype == DT_F16 ? launch_r<DT_F16, 7>(pk, a, g, stream)
                                         : launch_r<DT_F32, 7>(pk, a, g, stream);
        case 4: return a.dtype == DT_F16 ? launch_r<DT_F16, 4>(pk, a, g, stream)
                                         : launch_r<DT_F32, 4>(pk, a, g, stream);
        default: return a.dtype == DT_F16 ? launch_r<DT_F16, 2>(pk, a, g, stream)
                                          : launch_r<DT_F32, 2>(pk, a, g, stream);
    }
}

// The launch configuration of a tuned-kernel call, for the configuration
// query of the C ABI.  Host only.
bool describe_conv_stream(const PatTable& tab, const ConvArgs& a, ConvForm& out) {
    Geo g;
    if (!plan_conv_stream(tab, a, g)) return false;
    out.kernel = g.form == 1 ? 1 : 0;
    out.staged = g.form == 1 ? 0 : g.lds;
    out.rows_per_lane = g.R;
    out.cols_per_lane = g.form == 1 ? 4 : 1;
    out.segments_per_wave = g.S;
    out.column_tiles = g.CT;
    out.shares = g.KS;
    out.filters_per_block = g.FW;
    out.blocks = g.nblocks;
    out.threads_per_block = g.FW * g.KS * 64;
    return true;
}

}  // namespace psc
