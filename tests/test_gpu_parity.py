"""GPU parity: every HIP entry point against the CPU oracle on the same
seeded inputs.  Preparation (projection, selection, packing, unpacking) must
be bit-exact; convolution outputs are compared with the oracle's result from
its own packing, within a normwise relative error of 1e-4 (fp32) or 1e-2
(fp16 storage, fp32 accumulation) and within the element-wise fp32
summation bound gamma_n * sum|v*x| (plus the fp16 output rounding)."""
import numpy as np
import pytest

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import (TOL, check_conv, check_output, compare_prepared, dev, gpu_prepare, host_prepare,
                       max_terms, norm_err, note, oracle_ref, prepared_case, torch_mod)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


def _case(seed, cout, cin, m, drop, dtype, masks=None):
    w = inputs.he_weights(seed, cout, cin, dtype)
    if masks is None:
        masks = oracle.select_library(w, m)
    keep = inputs.keep_after_drop(cout * cin, drop)
    return w, np.asarray(masks, dtype=np.uint16), keep


# ---------------------------------------------------------------- preparation
PREP_CASES = [
    (4, 3, 8, 0, np.float32), (64, 64, 8, 50, np.float32), (33, 17, 6, 70, np.float16),
    (128, 64, 12, 60, np.float16), (7, 5, 1, 40, np.float32), (16, 16, 56, 30, np.float32),
    (8, 8, 4, 100, np.float32), (3, 2, 4, 50, np.float16), (200, 3, 8, 0, np.float32),
    (512, 512, 8, 60, np.float16), (256, 512, 8, 67, np.float32),
]


@pytest.mark.parametrize("cout,cin,m,drop,dtype", PREP_CASES)
def test_prepare_bitexact(cout, cin, m, drop, dtype):
    w, masks, keep = _case(cout * 7 + cin, cout, cin, m, drop, dtype)
    note("prepare %dx%d m=%d keep=%d %s" % (cout, cin, m, keep, np.dtype(dtype).name))
    prep = gpu_prepare(w, masks, keep)
    compare_prepared(prep, w, masks, keep)


def test_prepare_adversarial_ties():
    rng = np.random.default_rng(17)
    cases = []
    # all-zero layer: every energy ties at 0
    cases.append((np.zeros((16, 8, 3, 3), dtype=np.float32), 8, 50))
    # small integers: many equal energies across the keep boundary
    cases.append((rng.integers(-2, 3, size=(40, 30, 3, 3)).astype(np.float32), 6, 45))
    # duplicated kernels
    base = inputs.he_weights(3, 1, 1)
    cases.append((np.repeat(np.repeat(base, 12, axis=0), 10, axis=1).astype(np.float32), 8, 30))
    # equal-magnitude neighbours with mixed signs
    k = np.array([[1, -1, 1], [-1, 2, 1], [1, 1, -1]], dtype=np.float16)
    cases.append((np.tile(k, (9, 11, 1, 1)), 8, 60))
    # many ties at both sizes of the selection: 65536 kernels (one
    # workgroup) and 76800 (the multi-block passes)
    cases.append((rng.integers(-2, 3, size=(256, 256, 3, 3)).astype(np.float32), 8, 55))
    cases.append((rng.integers(-2, 3, size=(300, 256, 3, 3)).astype(np.float32), 8, 55))
    for w, m, drop in cases:
        cout, cin = w.shape[:2]
        masks = oracle.select_library(w, m)
        keep = inputs.keep_after_drop(cout * cin, drop)
        note("adversarial prepare %dx%d keep=%d" % (cout, cin, keep))
        compare_prepared(gpu_prepare(w, masks, keep), w, masks, keep)


@pytest.mark.parametrize("keep_mode", ["zero", "one", "all", "last"])
def test_prepare_keep_extremes(keep_mode):
    cout, cin = 12, 9
    K = cout * cin
    keep = {"zero": 0, "one": 1, "all": K, "last": K - 1}[keep_mode]
    w, masks, _ = _case(5, cout, cin, 8, 0, np.float32)
    note("prepare keep=%d" % keep)
    compare_prepared(gpu_prepare(w, masks, keep), w, masks, keep)


def test_prepare_non_centre_masks():
    w = inputs.he_weights(77, 24, 20)
    masks = inputs.random_masks(3, 10, centre=False)
    note("prepare non-centre masks")
    compare_prepared(gpu_prepare(w, masks, 150), w, masks, 150)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_unpack_dense_bitexact(dtype):
    torch = torch_mod()
    w, masks, keep = _case(31, 40, 24, 8, 55, dtype)
    prep = gpu_prepare(w, masks, keep)
    pat, _, keep_mask, _ = host_prepare(w, masks, keep)
    wd = torch.empty(w.shape, dtype=getattr(torch, np.dtype(dtype).name), device="cuda")
    note("unpack %s" % np.dtype(dtype).name)
    B.unpack_dense(prep.layer, prep.packed, wd)
    torch.cuda.synchronize()
    assert wd.cpu().numpy().tobytes() == oracle.mask_weights(w, masks, pat, keep_mask).tobytes()


def test_library_host_matches_oracle_on_workloads():
    for wl in (inputs.vgg16_stack(1), inputs.resnet18_cifar_3x3(256)):
        allk = inputs.all_kernels(wl)
        assert np.array_equal(B.select_library(allk, wl.m), oracle.select_library(allk, wl.m))


# ---------------------------------------------------------------- convolution
CONV_SHAPES = [
    # n, cin, cout, h, w
    (1, 3, 8, 5, 5), (2, 5, 7, 9, 11), (1, 16, 16, 1, 1), (1, 8, 8, 2, 3), (3, 4, 5, 3, 4),
    (1, 8, 16, 4, 4), (2, 6, 9, 7, 7), (1, 5, 4, 13, 13), (1, 4, 8, 6, 130), (1, 8, 8, 10, 32),
    (1, 4, 4, 3, 63), (1, 4, 4, 3, 64), (2, 3, 6, 8, 62), (1, 6, 10, 17, 16), (5, 7, 3, 4, 8),
    (1, 3, 8, 9, 224), (2, 5, 6, 7, 112), (1, 20, 9, 5, 240), (3, 17, 5, 3, 64),
]


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", CONV_SHAPES)
def test_conv_shapes(shape, dtype, algo):
    n, cin, cout, h, w = shape
    wt, masks, keep = _case(n * 1000 + cin * 31 + cout, cout, cin, 8, 40, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(h * w + cin, (n, cin, h, w), dtype)
    bias = inputs.bias_vector(cout, cout, dtype) if (h + w) % 2 else None
    note("conv %s %s algo=%d" % (shape, np.dtype(dtype).name, algo))
    check_conv(prep, packed, x, masks, bias=bias, relu=bool(cin % 2), algo=algo, dtype=dtype, what=str(shape))


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("m,centre", [(1, True), (4, True), (6, True), (12, True), (56, True),
                                      (6, False), (20, False)])
def test_conv_library_sizes(m, centre, algo):
    cin, cout = 24, 20
    masks = inputs.random_masks(m + 100, m, centre=centre)
    wt = inputs.he_weights(m, cout, cin)
    keep = inputs.keep_after_drop(cout * cin, 30)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(m, (2, cin, 12, 14))
    note("conv m=%d centre=%s algo=%d" % (m, centre, algo))
    check_conv(prep, packed, x, masks, algo=algo)


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("keep_mode", ["zero", "one", "all"])
def test_conv_keep_extremes(keep_mode, algo):
    cin, cout = 9, 11
    keep = {"zero": 0, "one": 1, "all": cin * cout}[keep_mode]
    wt, masks, _ = _case(8, cout, cin, 8, 0, np.float32)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(9, (2, cin, 6, 7))
    bias = inputs.bias_vector(10, cout)
    note("conv keep=%d algo=%d" % (keep, algo))
    check_conv(prep, packed, x, masks, bias=bias, relu=True, algo=algo)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_conv_many_channel_chunks(dtype):
    # cin well above one LDS chunk, cout not a multiple of the filter group
    n, cin, cout, h, w = 2, 300, 70, 9, 10
    wt, masks, keep = _case(123, cout, cin, 8, 60, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(5, (n, cin, h, w), dtype)
    note("conv many chunks %s" % np.dtype(dtype).name)
    check_conv(prep, packed, x, masks, dtype=dtype)


@pytest.mark.parametrize("cin,kernel", [(8191, 0), (8192, 2)])
def test_conv_at_the_2gib_input_limit(cin, kernel):
    """fp32 x at the limit of a buffer descriptor's range (2^31 - 1 bytes):
    2^31 - 256 KiB bytes run the tuned kernel, whose last channel ends just
    below the limit; exactly 2^31 bytes take the one-output-per-lane kernel.
    The last channel's kernels carry the largest weights, so they are kept
    and its last rows are read."""
    n, cout, h, w = 1, 4, 256, 256
    wt, masks, _ = _case(777, cout, cin, 8, 0, np.float32)
    wt[:, cin - 1] *= 100.0
    prep, packed = prepared_case(wt, masks, 64)
    assert (packed["cin_idx"] == cin - 1).sum() == cout
    assert B.conv3x3_config(prep.layer, B.PSC_F32, n, h, w, False, 1, 0)["kernel"] == kernel
    x = inputs.normal_activations(778, (n, cin, h, w))
    assert x.nbytes == (1 << 31) - (8192 - cin) * h * w * 4
    note("conv at the 2 GiB input limit, cin=%d" % cin)
    check_conv(prep, packed, x, masks, what="2 GiB limit cin=%d" % cin)


def test_conv_deterministic_and_in_bounds():
    torch = torch_mod()
    n, cin, cout, h, w = 2, 40, 24, 14, 14
    wt, masks, keep = _case(55, cout, cin, 8, 50, np.float32)
    prep = gpu_prepare(wt, masks, keep)
    x = dev(inputs.normal_activations(6, (n, cin, h, w)))
    guard = 4096
    numel = n * cout * h * w
    buf = torch.full((numel + 2 * guard,), 1234.5, dtype=torch.float32, device="cuda")
    y1 = buf[guard:guard + numel].view(n, cout, h, w)
    note("determinism/guard")
    B.conv3x3_fwd(prep.layer, prep.packed, x, y1)
    first = y1.clone()
    B.conv3x3_fwd(prep.layer, prep.packed, x, y1)
    torch.cuda.synchronize()
    assert torch.equal(first, y1)
    assert bool((buf[:guard] == 1234.5).all()) and bool((buf[guard + numel:] == 1234.5).all())


# ---------------------------------------------------------------- comparators
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", [(1, 3, 8, 5, 5), (2, 20, 17, 19, 23), (1, 64, 64, 32, 32),
                                   # the matrix-core tiles: 64 filters x 8x8 pixels, 8 channels a stage
                                   (1, 13, 70, 9, 11), (2, 130, 96, 16, 24), (1, 9, 65, 7, 33),
                                   # at most 8 channels: the vector-ALU tile kernel
                                   (1, 3, 64, 40, 36), (3, 1, 1, 1, 1)])
def test_dense_comparator(shape, dtype):
    torch = torch_mod()
    n, cin, cout, h, w = shape
    wt, masks, keep = _case(9, cout, cin, 8, 50, dtype)
    pat, _, keep_mask, _ = host_prepare(wt, masks, keep)
    wm = oracle.mask_weights(wt, masks, pat, keep_mask)
    x = inputs.normal_activations(4, shape[:1] + (cin, h, w), dtype)
    bias = inputs.bias_vector(3, cout, dtype)
    y = torch.empty((n, cout, h, w), dtype=getattr(torch, np.dtype(dtype).name), device="cuda")
    note("dense %s" % (shape,))
    B.dense3x3_fwd(dev(x), dev(wm), y, bias=dev(bias), relu=True)
    torch.cuda.synchronize()
    ref = oracle.conv_dense(x, wm, bias=bias, relu=True)
    assert norm_err(y.cpu().numpy(), ref) <= TOL[dtype]


POOL_SHAPES = [
    # n, cin, cout, h, w: full-row segments of each width class, haloed column
    # tiles (the one-output-per-lane kernel), wide rows, ragged bands, splits
    (1, 6, 5, 14, 14), (2, 9, 7, 28, 28), (1, 40, 12, 56, 56), (2, 3, 4, 6, 2), (1, 5, 6, 10, 130),
    (1, 7, 9, 8, 112), (1, 4, 8, 6, 224), (1, 300, 20, 14, 14), (3, 12, 5, 18, 62),
]


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", POOL_SHAPES)
def test_conv_pool_fused(shape, dtype, algo):
    torch = torch_mod()
    n, cin, cout, h, w = shape
    wt, masks, keep = _case(n * 700 + cin * 13 + cout, cout, cin, 8, 50, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(h * 3 + w, (n, cin, h, w), dtype)
    bias = inputs.bias_vector(cout + 5, cout, dtype) if (cin % 2) else None
    relu = bool(cout % 2)
    y = torch.empty((n, cout, h // 2, w // 2), dtype=getattr(torch, np.dtype(dtype).name), device="cuda")
    note("conv+pool %s %s algo=%d" % (shape, np.dtype(dtype).name, algo))
    B.conv3x3_fwd_pool2(prep.layer, prep.packed, dev(x), y, bias=None if bias is None else dev(bias),
                        relu=relu, algo=algo)
    torch.cuda.synchronize()
    ref, s = oracle_ref(x, packed, masks, cout, bias=bias, relu=relu, pool=True)
    check_output(y.cpu().numpy(), ref, s, dtype, max_terms(packed), "pool %s" % (shape,))


STRIDE_SHAPES = [
    # n, cin, cout, h, w: ResNet stage entries (even sizes), odd and ragged
    # sizes, 1x1 and 1-row images, more outputs than one block of lanes
    (2, 64, 128, 32, 32), (1, 128, 256, 16, 16), (2, 256, 64, 8, 8), (1, 5, 7, 9, 11), (3, 4, 5, 1, 1),
    (1, 6, 4, 2, 3), (2, 7, 9, 13, 6), (1, 3, 8, 1, 40), (1, 9, 6, 45, 37),
]


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", STRIDE_SHAPES)
def test_conv_strided(shape, dtype, algo):
    torch = torch_mod()
    tdt = getattr(torch, np.dtype(dtype).name)
    n, cin, cout, h, w = shape
    wt, masks, keep = _case(n * 500 + cin * 7 + cout, cout, cin, 8, 60, dtype)
    prep, packed = prepared_case(wt, masks, keep)
    x = inputs.normal_activations(h * 5 + w, (n, cin, h, w), dtype)
    bias = inputs.bias_vector(cout + 9, cout, dtype) if (cout % 2) else None
    relu = bool(cin % 2)
    xd = dev(x)
    bd = None if bias is None else dev(bias)
    y = torch.empty((n, cout, (h - 1) // 2 + 1, (w - 1) // 2 + 1), dtype=tdt, device="cuda")
    note("conv stride 2 %s %s algo=%d" % (shape, np.dtype(dtype).name, algo))
    B.conv3x3_fwd_strided(prep.layer, prep.packed, xd, y, 2, bias=bd, relu=relu, algo=algo)
    torch.cuda.synchronize()
    ref, s = oracle_ref(x, packed, masks, cout, bias=bias, relu=relu, stride=2)
    check_output(y.cpu().numpy(), ref, s, dtype, max_terms(packed), "stride 2 %s" % (shape,))
    # stride 1 through the strided entry point is the plain conv, bit for bit
    y1 = torch.empty((n, cout, h, w), dtype=tdt, device="cuda")
    y1s = torch.empty_like(y1)
    note("conv stride 1 via strided entry %s" % (shape,))
    B.conv3x3_fwd_strided(prep.layer, prep.packed, xd, y1s, 1, bias=bd, relu=relu, algo=algo)
    B.conv3x3_fwd(prep.layer, prep.packed, xd, y1, bias=bd, relu=relu, algo=algo)
    torch.cuda.synchronize()
    assert torch.equal(y1, y1s)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_maxpool(dtype):
    torch = torch_mod()
    x = inputs.normal_activations(2, (3, 5, 8, 12), dtype)
    y = torch.empty((3, 5, 4, 6), dtype=getattr(torch, np.dtype(dtype).name), device="cuda")
    note("maxpool")
    B.maxpool2x2(dev(x), y)
    torch.cuda.synchronize()
    ref = oracle.maxpool2x2(x.astype(np.float64))
    assert np.array_equal(y.cpu().numpy().astype(np.float64), ref)
