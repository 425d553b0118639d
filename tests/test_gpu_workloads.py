"""GPU parity at the full sizes of every benchmark workload, in the launch
configuration the benchmark times (the default kernel choice for each layer
shape).

For each layer: the library is chosen over all kernels of the workload,
projection / selection / packing run on the GPU and must equal the oracle's
bit for bit, and the convolution output of every image must pass both parity
gates (normwise and element-wise) against the oracle's fp64 result from its
own packing on the same input.  The VGG-16 stack runs chained exactly as in
the benchmark (conv + ReLU, GPU max-pool or the fused conv + pool launch),
each layer checked on the input the GPU layer actually received.
"""
import numpy as np
import pytest

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import check_output, compare_prepared, dev, max_terms, note, oracle_ref, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


def _check_layer(wl, li, lay, masks, x_dev, bias=None):
    """Prepare layer li on the GPU, compare the preparation bit-exactly, run
    the conv on x_dev and compare every image with the oracle; returns the
    GPU output, the prepared layer and the oracle's packing."""
    torch = torch_mod()
    w = inputs.layer_weights(wl, li)
    note("%s %s prepare" % (wl.name, lay.name))
    prep = B.prepare(dev(w), masks, lay.keep)
    torch.cuda.synchronize()
    _, _, _, packed = compare_prepared(prep, w, masks, lay.keep)
    note("%s %s conv (%d images)" % (wl.name, lay.name, wl.batch))
    bd = None if bias is None else dev(bias)
    y = torch.empty((wl.batch, lay.cout) + lay.out_hw, dtype=x_dev.dtype, device="cuda")
    B.conv3x3_fwd_strided(prep.layer, prep.packed, x_dev, y, lay.stride, bias=bd, relu=lay.relu)
    torch.cuda.synchronize()
    ref, s = oracle_ref(x_dev.cpu().numpy(), packed, masks, lay.cout, bias=bias, relu=lay.relu,
                        stride=lay.stride)
    check_output(y.cpu().numpy(), ref, s, wl.np_dtype, max_terms(packed), "%s %s" % (wl.name, lay.name))
    return y, prep, packed


def _workload(name):
    for wl in inputs.all_workloads():
        if wl.name == name:
            return wl
    raise KeyError(name)


def test_vgg16_stack_chained():
    torch = torch_mod()
    wl = _workload("vgg16_224_b1_f32")
    masks = B.select_library(inputs.all_kernels(wl), wl.m)
    x = dev(inputs.layer_input(wl, 0))
    for li, lay in enumerate(wl.layers):
        y, prep, packed = _check_layer(wl, li, lay, masks, x)
        if lay.pool_after:
            # the fused conv + ReLU + pool launch the benchmark may use
            fused = torch.empty((wl.batch, lay.cout, lay.h // 2, lay.w // 2), dtype=y.dtype, device="cuda")
            note("%s %s fused conv+pool" % (wl.name, lay.name))
            B.conv3x3_fwd_pool2(prep.layer, prep.packed, x, fused, relu=lay.relu)
            torch.cuda.synchronize()
            ref, s = oracle_ref(x.cpu().numpy(), packed, masks, lay.cout, relu=lay.relu, pool=True)
            check_output(fused.cpu().numpy(), ref, s, wl.np_dtype, max_terms(packed),
                         "%s %s fused" % (wl.name, lay.name))
            p = torch.empty((wl.batch, lay.cout, lay.h // 2, lay.w // 2), dtype=y.dtype, device="cuda")
            note("%s %s pool" % (wl.name, lay.name))
            B.maxpool2x2(y, p)
            torch.cuda.synchronize()
            ref = oracle.maxpool2x2(y.cpu().numpy().astype(np.float64))
            assert np.array_equal(p.cpu().numpy().astype(np.float64), ref)
            y = p
        x = y


@pytest.mark.parametrize("name", [wl.name for wl in inputs.all_workloads() if not wl.chained])
def test_workload_layers(name):
    wl = _workload(name)
    masks = B.select_library(inputs.all_kernels(wl), wl.m)
    for li, lay in enumerate(wl.layers):
        x = dev(inputs.layer_input(wl, li))
        bias = inputs.layer_bias(wl, li) if li == 0 else None
        _check_layer(wl, li, lay, masks, x, bias=bias)
