"""Shared helpers for the GPU parity tests: build a case from seeded inputs,
run the HIP path through the C ABI and compare with the oracle."""
import sys

import numpy as np

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs

NP2TORCH = {np.float32: "float32", np.float16: "float16"}
TOL = {np.float32: 1e-4, np.float16: 1e-2}


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
    """Bit-exact comparison of projection, selection and packing."""
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


def norm_err(y, ref):
    y = np.asarray(y, dtype=np.float64)
    den = float(np.abs(ref).max()) if ref.size else 0.0
    num = float(np.abs(y - ref).max()) if ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den


def check_conv(prep, x, masks, bias=None, relu=False, algo=0, dtype=np.float32, ref=None,
               images=None):
    """Run the HIP conv on x and compare (normwise) with the oracle; only the
    listed images are compared when ``images`` is given."""
    torch = torch_mod()
    cout = prep.layer.cout
    xd = dev(x)
    bd = dev(bias) if bias is not None else None
    y = B.conv(prep, xd, bias=bd, relu=relu, algo=algo)
    torch.cuda.synchronize()
    yh = y.cpu().numpy()
    if ref is None:
        packed = prep.packed.to_host()
        xs = x if images is None else x[images]
        ref = oracle.conv_sparse(xs, packed, masks, cout, bias=bias, relu=relu)
    ys = yh if images is None else yh[images]
    err = norm_err(ys, ref)
    assert err <= TOL[dtype], "normwise error %.3e above %.0e" % (err, TOL[dtype])
    return yh, err
