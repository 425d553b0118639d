"""GPU parity of the retraining kernels (Sec. 3.3) against the oracle:

* the transposed layer's dense inputs (psc_transpose_prep) equal the numpy
  transpose + 180-degree rotation bit for bit, and psc_pack of them equals
  the oracle's packing of the same inputs byte for byte;
* dx (the tuned forward kernels on the transposed packing) and the masked
  gradient dv, db (psc_conv3x3_bwd_weight) pass the normwise gate and the
  element-wise fp32 summation bound against the oracle's fp64 backward,
  computed from the original (untransposed) storage."""
import numpy as np
import pytest

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import (TOL, check_output, dev, gamma, host_prepare, max_terms, norm_err, note, prepared_case,
                       torch_mod)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


def rotate_masks(masks):
    return np.array([sum(1 << (8 - q) for q in range(9) if (int(m) >> q) & 1) for m in masks], dtype=np.uint16)


SHAPES = [
    # n, cin, cout, h, w: ragged and tiny planes, several tiles, wide rows,
    # cin != cout, and full-size layers of the VGG-16 and ResNet-50 workloads
    (2, 5, 7, 9, 11), (1, 3, 8, 1, 1), (3, 8, 5, 6, 70), (2, 16, 24, 14, 14), (1, 24, 12, 28, 28),
    (2, 9, 6, 7, 130), (1, 512, 512, 28, 28), (32, 256, 256, 14, 14),
    # whole waves of small images (one image row per lane in both passes):
    # every compiled width, ragged image groups, rows unequal to columns, odd
    # n, cin and cout (fp16 width 7: rows read through a shifted window, the
    # last row of x and of dy at the end of its buffer)
    (13, 5, 6, 4, 4), (9, 7, 5, 7, 7), (11, 3, 5, 7, 7), (8, 16, 9, 8, 8), (7, 4, 5, 5, 8),
    (5, 6, 7, 14, 14), (4, 10, 6, 16, 16), (32, 64, 64, 7, 7),
    # widths that are multiples of 4 below a whole wave of images (4 columns
    # per lane in the weight gradient): one to sixteen row bands per wave,
    # ragged last bands, a 63-lane segment
    (1, 3, 5, 6, 4), (3, 9, 7, 11, 32), (2, 6, 5, 7, 64), (1, 8, 4, 9, 224), (1, 3, 4, 5, 252),
    # one band group per wave at batch 1 (the weight gradient pipelines a
    # wave's chunks): full-size VGG-16 14x14 and ResNet-50 7x7 layers
    (1, 512, 512, 14, 14), (1, 512, 512, 7, 7),
    # batch 1, fp32, at least 16 channels: the masked gradient gathered from
    # the matrix-core dense one (two filter blocks, a channel tail, ragged
    # pixel tiles, partial sums over several blocks)
    (1, 16, 70, 9, 17), (1, 33, 5, 6, 40), (1, 64, 64, 56, 56),
]


def _case(shape, dtype):
    n, cin, cout, h, w = shape
    wt = inputs.he_weights(cin * 7 + cout + h, cout, cin, dtype)
    masks = oracle.select_library(wt, 8)
    keep = inputs.keep_after_drop(cout * cin, 60)
    x = inputs.normal_activations(h * w + 1, (n, cin, h, w), dtype)
    dy = inputs.normal_activations(h * w + 2, (n, cout, h, w), dtype)
    return wt, masks, keep, x, dy


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", SHAPES)
def test_bwd_data_via_transposed_packing(shape, dtype):
    torch = torch_mod()
    n, cin, cout, h, w = shape
    wt, masks, keep, x, dy = _case(shape, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    note("transpose prep %s %s" % (shape, np.dtype(dtype).name))
    wd = dev(wt)
    pt = B.prepare_transposed(prep, wd)
    torch.cuda.synchronize()
    pat, _, keep_mask, _ = host_prepare(wt, masks, keep)
    w_t = np.ascontiguousarray(wt.transpose(1, 0, 2, 3)[:, :, ::-1, ::-1])
    pat_t = np.ascontiguousarray(pat.reshape(cout, cin).T).reshape(-1)
    keep_t = np.ascontiguousarray(keep_mask.reshape(cout, cin).T).reshape(-1)
    assert pt.w.cpu().numpy().tobytes() == w_t.tobytes()
    assert np.array_equal(pt.pat.cpu().numpy(), pat_t) and np.array_equal(pt.keep_mask.cpu().numpy(), keep_t)
    masks_t = rotate_masks(masks)
    assert np.array_equal(pt.layer.masks, masks_t)
    packed_t = oracle.pack(w_t, masks_t, pat_t, keep_t)
    gp = pt.packed.to_host()
    for name in B.PACKED_FIELDS:
        assert gp[name].tobytes() == packed_t[name].tobytes(), "transposed packed %s differs" % name
    note("bwd data %s %s" % (shape, np.dtype(dtype).name))
    dx = B.conv(pt, dev(dy))
    torch.cuda.synchronize()
    ref, s = oracle.conv_sparse_bwd_data(dy, packed, masks, cin, want_scale=True)
    check_output(dx.cpu().numpy(), ref, s, dtype, max_terms(packed_t), "dx %s" % (shape,))


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", SHAPES)
def test_bwd_weight_masked_gradient(shape, dtype):
    torch = torch_mod()
    n, cin, cout, h, w = shape
    wt, masks, keep, x, dy = _case(shape, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    dv = torch.full((4 * keep,), 99.0, dtype=torch.float32, device="cuda")
    db = torch.full((cout,), 99.0, dtype=torch.float32, device="cuda")
    note("bwd weight %s %s" % (shape, np.dtype(dtype).name))
    B.conv3x3_bwd_weight(prep.layer, prep.packed, dev(x), dev(dy), dv, db)
    torch.cuda.synchronize()
    ref_v, ref_b, s_v = oracle.conv_sparse_bwd_weight(x, dy, packed, masks, want_scale=True)
    terms = n * h * w
    what = "dv %s %s" % (shape, np.dtype(dtype).name)
    got = dv.cpu().numpy().astype(np.float64)
    assert norm_err(got, ref_v) <= TOL[np.float32], what
    assert (np.abs(got - ref_v) <= gamma(terms) * s_v).all(), what
    gb = db.cpu().numpy().astype(np.float64)
    s_b = np.abs(dy.astype(np.float64)).sum(axis=(0, 2, 3))
    assert (np.abs(gb - ref_b) <= gamma(terms) * s_b).all(), "db " + what
    # deterministic: a second call reproduces the result bit for bit
    dv2 = torch.empty_like(dv)
    B.conv3x3_bwd_weight(prep.layer, prep.packed, dev(x), dev(dy), dv2)
    torch.cuda.synchronize()
    assert torch.equal(dv, dv2)
