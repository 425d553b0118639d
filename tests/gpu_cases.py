"""Shared helpers for the GPU parity tests: build a case from seeded inputs,
run the HIP path through the C ABI and compare with the oracle.

Every conv reference is computed by the oracle from the oracle's own
projection, selection and packing, after asserting that the HIP packing
equals it byte for byte.  Outputs pass two gates:

* normwise: max|y - ref| / max|ref| <= 1e-4 (fp32) or 1e-2 (fp16 storage);
* element-wise: |y - ref| <= gamma_n * s (+ the fp16 output rounding), where
  s = sum |v*x| + |b| is the oracle's error scale of that output and
  gamma_n = n u / (1 - n u), u = 2^-24, n the number of terms summed into
  one output (4 per kept kernel of its filter, plus the bias).  This is the
  classical bound for a sum of n terms in fp32 in any order (the products
  are exact inside the fused multiply-adds), so a dropped, doubled or
  misaddressed tap exceeds it while any summation order stays inside.
"""
import sys

import numpy as np

import oracle
from paper_2003_06513_amd import binding as B

NP2TORCH = {np.float32: "float32", np.float16: "float16"}
TOL = {np.float32: 1e-4, np.float16: 1e-2}
U32 = 2.0 ** -24          # fp32 unit roundoff
U16 = 2.0 ** -11          # binary16 unit roundoff (output rounding)
SUB16 = 2.0 ** -25        # half the smallest binary16 subnormal


def torch_mod():
    import torch
    return torch


def dev(a):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def note(msg):
    """Name the case before a GPU step (flushed, so it survives a crash)."""
    sys.stdout.write("[case] %s\n" % msg)
    sys.stdout.flush()


def host_prepare(w, masks, keep):
    pat, energy = oracle.project(w, masks)
    keep_mask = oracle.select(energy, keep)
    return pat, energy, keep_mask, oracle.pack(w, masks, pat, keep_mask)


def gpu_prepare(w, masks, keep):
    prep = B.prepare(dev(w), masks, keep)
    torch_mod().cuda.synchronize()
    return prep


def compare_prepared(prep, w, masks, keep):
    """Bit-exact comparison of projection, selection and packing; returns the
    oracle's results (pat, energy, keep mask, packed)."""
    pat, energy, keep_mask, packed = host_prepare(w, masks, keep)
    g_pat = prep.pat.cpu().numpy()
    g_energy = prep.energy.cpu().numpy()
    g_keep = prep.keep_mask.cpu().numpy()
    assert np.array_equal(g_pat, pat), "pattern ids differ"
    assert g_energy.tobytes() == energy.tobytes(), "energies differ in some bit"
    assert np.array_equal(g_keep, keep_mask), "keep masks differ"
    gp = prep.packed.to_host()
    for name in B.PACKED_FIELDS:
        assert gp[name].tobytes() == packed[name].tobytes(), "packed %s differs" % name
    return pat, energy, keep_mask, packed


def prepared_case(w, masks, keep):
    """GPU preparation checked bit for bit; returns (GPU result, the oracle's
    packed storage)."""
    prep = gpu_prepare(w, masks, keep)
    packed = compare_prepared(prep, w, masks, keep)[3]
    return prep, packed


def max_terms(packed) -> int:
    """Terms summed into one output: 4 per kept kernel of the longest filter,
    plus the bias."""
    fp = np.asarray(packed["filter_ptr"], dtype=np.int64)
    return 4 * int(np.diff(fp).max(initial=0)) + 1


def gamma(n: int) -> float:
    return n * U32 / (1.0 - n * U32)


def oracle_ref(x, packed, masks, cout, bias=None, relu=False, stride=1, pool=False):
    """The oracle's output and error scale (pooled: the max of the window's
    values and of their scales; max is 1-Lipschitz, so the pooled bound is
    the window's largest bound)."""
    ref, s = oracle.conv_sparse_strided(x, packed, masks, cout, stride, bias=bias, relu=relu, want_scale=True)
    if pool:
        ref, s = oracle.maxpool2x2(ref), oracle.maxpool2x2(s)
    return ref, s


def norm_err(y, ref):
    y = np.asarray(y, dtype=np.float64)
    den = float(np.abs(ref).max()) if ref.size else 0.0
    num = float(np.abs(y - ref).max()) if ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den


def check_output(y, ref, s, dtype, nterms, what=""):
    """Both gates; returns (normwise error, largest |y - ref| / s)."""
    y = np.asarray(y, dtype=np.float64)
    assert y.shape == ref.shape, "%s: shape %s vs %s" % (what, y.shape, ref.shape)
    err = norm_err(y, ref)
    assert err <= TOL[dtype], "%s: normwise error %.3e above %.0e" % (what, err, TOL[dtype])
    d = np.abs(y - ref)
    bound = gamma(nterms) * s
    if dtype == np.float16:
        bound = bound + U16 * (np.abs(ref) + bound) + SUB16
    over = d - bound
    if over.size and over.max() > 0:
        i = np.unravel_index(int(np.argmax(over)), over.shape)
        raise AssertionError("%s: element-wise bound exceeded at %s: |y-ref|=%.3e > %.3e (y=%r ref=%r s=%.3e)"
                             % (what, i, d[i], bound[i], y[i], ref[i], s[i]))
    scaled = float((d / np.where(s > 0, s, 1.0)).max()) if d.size else 0.0
    return err, scaled


def check_conv(prep, packed, x, masks, bias=None, relu=False, algo=0, dtype=np.float32, what=""):
    """Run the HIP conv on x and compare with the oracle's result from its own
    packing ``packed``."""
    torch = torch_mod()
    cout = prep.layer.cout
    xd = dev(x)
    bd = dev(bias) if bias is not None else None
    y = B.conv(prep, xd, bias=bd, relu=relu, algo=algo)
    torch.cuda.synchronize()
    yh = y.cpu().numpy()
    ref, s = oracle_ref(x, packed, masks, cout, bias=bias, relu=relu)
    check_output(yh, ref, s, dtype, max_terms(packed), what)
    return yh


# ------------------------------------------------------------------ kernel forms
FORM_MASKS = (23, 282, 58, 90)     # 4 centre+3 masks; the cases below use the workload library instead


def form_key(cfg, pool, dtype_code):
    return (cfg["kernel"], cfg["staged"], cfg["column_tiles"] > 1, cfg["shares"] > 1, bool(pool),
            cfg["rows_per_lane"], dtype_code)


def form_cases():
    """For every launch form the conv entry points can take -- kernel, load
    form, column tiles or full rows, split filters, pooled epilogue, rows per
    lane, dtype -- the smallest shape (n, cin, cout, h, w) of a fixed grid
    that takes it, found with the host-side configuration query; plus the
    stride-2 kernel, the one-row-per-lane kernel (algo 2) and the algo-1
    simple kernel.  Returns a sorted list of
    (key, n, cin, cout, h, w, dtype_code, pool, stride, algo)."""
    found = {}
    for n in (1, 2, 3, 4, 8):
        for cin in (3, 8, 16, 24, 40):
            for cout in (5, 8, 12):
                for hw in (4, 6, 7, 8, 10, 13, 14, 16, 17, 20, 24, 28, 32, 40, 56, 62, 64, 96, 112, 128, 130):
                    for dt in (B.PSC_F32, B.PSC_F16):
                        for pool in (False, True):
                            if pool and hw % 2:
                                continue
                            L = B.Layer(cout, cin, list(FORM_MASKS), cin * cout // 2, dt)
                            cfg = B.conv3x3_config(L, dt, n, hw, hw, pool, 1, 0)
                            key = form_key(cfg, pool, dt)
                            work = n * cin * cout * hw * hw
                            if key not in found or work < found[key][0]:
                                found[key] = (work, (key, n, cin, cout, hw, hw, dt, pool, 1, 0))
    out = [v[1] for v in found.values()]
    for dt in (B.PSC_F32, B.PSC_F16):
        # the tuned stride-2 kernel, one output column per lane (w = 2 mod 4)
        # and two (w a multiple of 4): whole filters and split filters,
        # ragged output bands, several bands per wave, a band of one lane,
        # the widest rows
        for n, cin, cout, h, w in ((2, 9, 7, 14, 12), (1, 64, 8, 16, 16), (3, 5, 6, 13, 6), (1, 24, 5, 9, 126),
                                   (5, 7, 5, 9, 4), (1, 32, 6, 11, 124), (2, 48, 4, 28, 28), (1, 17, 9, 21, 56),
                                   (3, 40, 5, 10, 14)):
            L = B.Layer(cout, cin, list(FORM_MASKS), cin * cout // 2, dt)
            cfg = B.conv3x3_config(L, dt, n, h, w, False, 2, 0)
            out.append((("stride2", cfg["kernel"], cfg["cols_per_lane"], w, cfg["shares"] > 1),
                        n, cin, cout, h, w, dt, False, 2, 0))
        # the one-row-per-lane kernel (algo 2) at every compiled width: ragged
        # image groups, a partial wave, split filters, rows unequal to columns,
        # fp32 16 x 16 planes through LDS (a ragged last group, one partial
        # wave, 2 and 4 shares),
        # and (fp16, width 7, odd cin and n) the last row of x read through a
        # window that reaches past the end of x
        rows_shapes = ((13, 5, 6, 4, 4), (1, 40, 5, 4, 4), (9, 7, 5, 7, 7), (5, 3, 4, 7, 7), (3, 33, 6, 7, 7),
                       (8, 16, 9, 8, 8), (4, 24, 4, 5, 8), (5, 6, 7, 14, 14), (2, 48, 3, 13, 14),
                       (4, 10, 6, 16, 16), (1, 64, 4, 11, 16), (3, 9, 5, 28, 28), (1, 40, 3, 20, 28),
                       (1, 64, 4, 16, 16), (7, 40, 5, 16, 16))
        for n, cin, cout, h, w in rows_shapes:
            if dt == B.PSC_F16 and (w & 1) and w != 7:
                continue
            L = B.Layer(cout, cin, list(FORM_MASKS), cin * cout // 2, dt)
            cfg = B.conv3x3_config(L, dt, n, h, w, False, 1, 2)
            out.append((("rows", cfg["kernel"], w, cfg["shares"] > 1, cfg["staged"]), n, cin, cout, h, w, dt,
                        False, 1, 2))
        # its stride-2 form: every compiled width, odd and even heights (the
        # last output row's odd input row past the image), ragged groups,
        # split filters; fp32 8 x 8 and 16 x 16 planes go through LDS: a
        # ragged last group (images past the batch), one partial wave, and 2
        # and 4 shares (their sums reuse the staging areas)
        for n, cin, cout, h, w in ((13, 5, 6, 8, 8), (2, 40, 5, 7, 8), (9, 7, 5, 16, 16), (1, 48, 4, 15, 16),
                                   (4, 9, 5, 32, 32), (1, 40, 3, 31, 32), (1, 48, 4, 8, 8), (25, 70, 9, 8, 8),
                                   (1, 48, 4, 16, 16), (15, 70, 9, 16, 16)):
            L = B.Layer(cout, cin, list(FORM_MASKS), cin * cout // 2, dt)
            cfg = B.conv3x3_config(L, dt, n, h, w, False, 2, 2)
            out.append((("rows2", cfg["kernel"], w, cfg["shares"] > 1, cfg["staged"]), n, cin, cout, h, w, dt,
                        False, 2, 2))
        # the wide form below 64 columns and in fp16, which the automatic
        # choice takes only for grids of 6144+ waves: many filters over few
        # channels keep the oracle cheap; ragged bands, a pooled epilogue,
        # every segment count from 3 to 8 per wave
        for n, cin, cout, h, w, pool in ((64, 5, 1024, 5, 28, False), (40, 3, 1024, 6, 32, False),
                                         (16, 4, 1024, 7, 56, False), (16, 3, 1024, 8, 56, True),
                                         (12, 3, 2048, 4, 64, False), (4, 3, 1024, 7, 252, False)):
            if dt == B.PSC_F32 and w in (64, 252):
                continue
            L = B.Layer(cout, cin, list(FORM_MASKS), cin * cout // 2, dt)
            cfg = B.conv3x3_config(L, dt, n, h, w, pool, 1, 0)
            out.append((("wide", cfg["kernel"], cfg["cols_per_lane"], w), n, cin, cout, h, w, dt, pool, 1, 0))
        out.append((("simple-stride2",), 2, 9, 7, 13, 11, dt, False, 2, 0))
        out.append((("simple-algo1",), 2, 9, 7, 13, 11, dt, False, 1, 1))
        out.append((("simple-algo1-pool",), 2, 9, 7, 12, 10, dt, True, 1, 1))
    return sorted(out, key=lambda c: str(c))
