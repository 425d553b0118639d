"""GPU parity at the full sizes of every benchmark workload, in the launch
configuration the benchmark times (the default kernel choice for each layer
shape).

For each layer: the library is chosen over all kernels of the workload,
projection / selection / packing run on the GPU and must equal the oracle's
bit for bit, and the convolution output must be within the normwise bound of
the oracle's fp64 result on the same input.  Batched layers are compared on
sampled images (first, middle, last), which the oracle computes one by one;
the VGG-16 stack runs chained exactly as in the benchmark (conv + ReLU, GPU
max-pool), each layer checked against the oracle on the input the GPU layer
actually received.
"""
import numpy as np
import pytest

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import TOL, compare_prepared, dev, note, norm_err, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


def _sample(n):
    return sorted({0, n // 2, n - 1})


def _check_layer(wl, li, lay, masks, x_dev, bias=None):
    """Prepare layer li on the GPU, compare the preparation bit-exactly, run
    the conv on x_dev and compare sampled images with the oracle; returns the
    GPU output."""
    torch = torch_mod()
    w = inputs.layer_weights(wl, li)
    note("%s %s prepare" % (wl.name, lay.name))
    prep = B.prepare(dev(w), masks, lay.keep)
    torch.cuda.synchronize()
    _, _, _, packed = compare_prepared(prep, w, masks, lay.keep)
    note("%s %s conv" % (wl.name, lay.name))
    bd = None if bias is None else dev(bias)
    if lay.stride == 1:
        y = B.conv(prep, x_dev, bias=bd, relu=lay.relu)
    else:
        y = torch.empty((wl.batch, lay.cout) + lay.out_hw, dtype=x_dev.dtype, device="cuda")
        B.conv3x3_fwd_strided(prep.layer, prep.packed, x_dev, y, lay.stride, bias=bd, relu=lay.relu)
    torch.cuda.synchronize()
    imgs = _sample(wl.batch)
    xs = x_dev[imgs].cpu().numpy()
    ref = oracle.conv_sparse_strided(xs, packed, masks, lay.cout, lay.stride, bias=bias, relu=lay.relu)
    err = norm_err(y[imgs].cpu().numpy(), ref)
    assert err <= TOL[wl.np_dtype], "%s %s: normwise error %.3e" % (wl.name, lay.name, err)
    return y


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
        y = _check_layer(wl, li, lay, masks, x)
        if lay.pool_after:
            # the fused conv + ReLU + pool launch the benchmark uses
            prep = B.prepare(dev(inputs.layer_weights(wl, li)), masks, lay.keep)
            fused = torch.empty((wl.batch, lay.cout, lay.h // 2, lay.w // 2), dtype=y.dtype, device="cuda")
            note("%s %s fused conv+pool" % (wl.name, lay.name))
            B.conv3x3_fwd_pool2(prep.layer, prep.packed, x, fused, relu=lay.relu)
            torch.cuda.synchronize()
            ref = oracle.maxpool2x2(oracle.conv_sparse(x.cpu().numpy(), prep.packed.to_host(), masks, lay.cout,
                                                       relu=lay.relu))
            err = norm_err(fused.cpu().numpy(), ref)
            assert err <= TOL[wl.np_dtype], "%s %s fused: normwise error %.3e" % (wl.name, lay.name, err)
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
    # identical layer shapes inside a stack take the same launch
    # configuration: check the first layer of each distinct shape
    seen = set()
    for li, lay in enumerate(wl.layers):
        key = (lay.cin, lay.cout, lay.h, lay.w, lay.keep, lay.stride)
        if key in seen:
            continue
        seen.add(key)
        x = dev(inputs.layer_input(wl, li))
        bias = inputs.layer_bias(wl, li) if li == 0 else None
        _check_layer(wl, li, lay, masks, x, bias=bias)
