"""CPU checks of the GPU tests' machinery (no device needed):

* the parity gates accept an fp32 summation of the right terms in another
  order (the oracle's own fp32-accumulating build) and reject the mistakes a
  kernel could make -- a dropped tap, a doubled tap, a tap read from the
  neighbouring column -- planted in copies of the oracle's storage;
* the launch-form search reaches every kernel, load form, rows-per-lane
  value and epilogue of the tuned conv, and the configuration query
  validates its arguments."""
import numpy as np
import pytest

import oracle
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import check_output, form_cases, host_prepare, max_terms, oracle_ref


def _layer(dtype, seed=3, cout=9, cin=30):
    w = inputs.he_weights(seed, cout, cin, dtype)
    masks = oracle.select_library(w, 8)
    _, _, keep, packed = host_prepare(w, masks, inputs.keep_after_drop(cout * cin, 40))
    x = inputs.normal_activations(seed + 1, (2, cin, 9, 11), dtype)
    b = inputs.bias_vector(seed + 2, cout, dtype)
    return w, masks, packed, x, b


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("stride", [1, 2])
def test_gate_accepts_fp32_sum_in_another_order(dtype, stride):
    w, masks, packed, x, b = _layer(dtype)
    ref, s = oracle_ref(x, packed, masks, w.shape[0], bias=b, relu=True, stride=stride)
    y = oracle.conv_sparse_f32acc(x, packed, masks, w.shape[0], stride, bias=b, relu=True).astype(dtype)
    check_output(y, ref, s, dtype, max_terms(packed))


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("mistake", ["drop", "double", "shift"])
def test_gate_rejects_planted_tap_mistakes(dtype, mistake):
    w, masks, packed, x, b = _layer(dtype, seed=11)
    cout = w.shape[0]
    ref, s = oracle_ref(x, packed, masks, cout, bias=b)
    bad = {k: v.copy() for k, v in packed.items()}
    k = len(bad["cin_idx"]) // 2
    if mistake == "drop":
        bad["values"][4 * k + 1] = 0
    elif mistake == "double":
        bad["values"][4 * k + 1] = bad["values"][4 * k + 1] * 2
    else:
        # the kernel's pattern replaced by another library pattern (taps at
        # other positions, same values)
        bad["pat_id"][k] = (int(bad["pat_id"][k]) + 1) % len(masks)
    y = oracle.conv_sparse_f32acc(x, bad, masks, cout, 1, bias=b).astype(dtype)
    with pytest.raises(AssertionError):
        check_output(y, ref, s, dtype, max_terms(packed))


def test_form_search_reaches_every_form():
    cases = form_cases()
    keys = [c[0] for c in cases if isinstance(c[0][0], int)]
    kinds = {(k[0], k[1]) for k in keys}
    assert {(0, 0), (0, 1), (0, 2), (1, 0), (2, 0)} <= kinds
    for dt in (B.PSC_F32, B.PSC_F16):
        assert {k[5] for k in keys if k[0] == 0 and k[6] == dt} == {2, 4, 7, 8}
        for staged in (0, 1, 2):
            assert any(k[0] == 0 and k[1] == staged and k[3] and k[6] == dt for k in keys)   # split filters
            assert any(k[0] == 0 and k[1] == staged and k[4] and k[6] == dt for k in keys)   # pooled epilogue
    assert any(k[0] == 1 and k[3] for k in keys) and any(k[0] == 1 and k[4] for k in keys)
    assert any(k[2] for k in keys)                                                         # column tiles
    assert {c[0][0] for c in cases if not isinstance(c[0][0], int)} == \
        {"stride2", "rows", "rows2", "wide", "simple-stride2", "simple-algo1", "simple-algo1-pool"}
    wide = [c for c in cases if c[0][0] == "wide"]
    assert all(c[0][1] == 1 and c[0][2] == 4 for c in wide)
    assert {(c[6], c[5]) for c in wide} == {(B.PSC_F32, 28), (B.PSC_F32, 32), (B.PSC_F32, 56), (B.PSC_F16, 28),
                                           (B.PSC_F16, 32), (B.PSC_F16, 56), (B.PSC_F16, 64), (B.PSC_F16, 252)}
    assert any(c[7] for c in wide if c[6] == B.PSC_F16) and any(c[7] for c in wide if c[6] == B.PSC_F32)
    rows = [c for c in cases if c[0][0] == "rows"]
    assert all(c[0][1] == 4 for c in rows)
    for dt in (B.PSC_F32, B.PSC_F16):
        assert {c[5] for c in rows if c[6] == dt} == {4, 7, 8, 14, 16, 28}
        assert any(c[0][3] for c in rows if c[6] == dt) and any(not c[0][3] for c in rows if c[6] == dt)
    rows2 = [c for c in cases if c[0][0] == "rows2"]
    for dt in (B.PSC_F32, B.PSC_F16):
        assert {c[5] for c in rows2 if c[6] == dt} == {8, 16, 32}
        assert any(c[0][3] for c in rows2 if c[6] == dt) and any(c[4] % 2 for c in rows2 if c[6] == dt)
    # the automatic choice takes the rows kernel for whole-wave batches on small planes
    assert any(isinstance(c[0][0], int) and c[0][0] == 4 for c in cases)
    s2 = [c[0] for c in cases if c[0][0] == "stride2"]
    assert all(k[1] == 3 for k in s2) and any(k[4] for k in s2) and any(not k[4] for k in s2)
    assert {k[2] for k in s2} == {1, 2} and all(k[2] == (2 if k[3] % 4 == 0 else 1) for k in s2)
    assert any(k[2] == 2 and k[4] for k in s2) and any(k[2] == 2 and not k[4] for k in s2)


def test_config_query_validates():
    L = B.Layer(8, 4, [23, 282], 10, B.PSC_F32)
    for args in [(B.PSC_F16, 1, 8, 8, False, 1, 0), (B.PSC_F32, 1, 8, 8, False, 3, 0),
                 (B.PSC_F32, 1, 7, 8, True, 1, 0), (B.PSC_F32, 1, 8, 8, True, 2, 0),
                 (B.PSC_F32, 1, 8, 8, False, 1, 4), (B.PSC_F32, 1, 8, 9, False, 1, 2),
                 (B.PSC_F32, 1, 8, 8, True, 1, 2), (B.PSC_F32, 1, 8, 10, False, 2, 2),
                 (B.PSC_F32, 1, 64, 8, False, 1, 2), (B.PSC_F32, -1, 8, 8, False, 1, 0)]:
        with pytest.raises(B.PscError):
            B.conv3x3_config(L, *args)
    assert B.conv3x3_config(L, B.PSC_F32, 2, 16, 16, False, 2, 0)["kernel"] == 3      # tuned stride 2
    assert B.conv3x3_config(L, B.PSC_F32, 2, 16, 16, False, 2, 0)["cols_per_lane"] == 2
    assert B.conv3x3_config(L, B.PSC_F32, 2, 16, 14, False, 2, 0)["cols_per_lane"] == 1
    assert B.conv3x3_config(L, B.PSC_F32, 2, 16, 15, False, 2, 0)["kernel"] == 2      # odd width
    assert B.conv3x3_config(L, B.PSC_F32, 2, 16, 16, False, 2, 1)["kernel"] == 2      # algo 1
    assert B.conv3x3_config(L, B.PSC_F32, 1, 8, 8, False, 1, 2)["kernel"] == 4        # algo 2: one row per lane
    assert B.conv3x3_config(L, B.PSC_F32, 7, 8, 8, False, 1, 0)["kernel"] == 4        # a whole wave of images
    assert B.conv3x3_config(L, B.PSC_F32, 6, 8, 8, False, 1, 0)["kernel"] == 0        # less than a wave
    assert B.conv3x3_config(L, B.PSC_F32, 7, 8, 8, False, 1, 3)["kernel"] == 0        # algo 3: column per lane
    assert B.conv3x3_config(L, B.PSC_F32, 64, 28, 28, False, 1, 0)["kernel"] == 0     # wider than 16


def test_r8_with_several_segments_is_never_planned():
    """R = 8 rows per lane with more than one row band per wave (direct form)
    faulted the device once, on the batch-256 fp32 layers 128@16x16 and
    256@8x8; the cause was not found, so the planner must never choose it.
    The configuration query covers every stride-1 shape class of the
    workloads and the form grid, at batch 1 to 256."""
    for dt in (B.PSC_F32, B.PSC_F16):
        for n in (1, 4, 32, 64, 256):
            for cin, cout in ((3, 64), (64, 64), (128, 128), (256, 256), (512, 512)):
                for hw in (4, 7, 8, 10, 14, 16, 20, 28, 32, 56, 62, 63):
                    L = B.Layer(cout, cin, [23, 282, 58, 90, 153, 216, 120, 57], cin * cout // 3, dt)
                    for pool in ((False, True) if hw % 2 == 0 else (False,)):
                        for algo in (0, 3):
                            cfg = B.conv3x3_config(L, dt, n, hw, hw, pool, 1, algo)
                            if cfg["kernel"] == 0:
                                assert not (cfg["rows_per_lane"] == 8 and cfg["segments_per_wave"] > 1), \
                                    (dt, n, cin, cout, hw, pool, algo, cfg)


def test_deep_28_column_layers_take_the_wide_form_with_shares():
    """fp32 rows of 28 columns with 128+ input channels at small batch take
    the 4-column form with 8 shares (a wave holds whole images; measured on
    the batch-1 VGG-16 28x28 layers), shallow ones and fp16 keep their
    forms."""
    codes = [c for c in range(512) if bin(c).count("1") == 4 and (c >> 4) & 1][:8]
    def cfg(cin, cout, n, dtype):
        L = B.Layer(cout, cin, codes, (cout * cin) // 3, dtype)
        return B.conv3x3_config(L, dtype, n, 28, 28, False, 1, 0)
    for cin, cout in ((256, 512), (512, 512)):
        c = cfg(cin, cout, 1, B.PSC_F32)
        assert (c["kernel"], c["cols_per_lane"], c["shares"]) == (1, 4, 8)
    assert cfg(64, 64, 1, B.PSC_F32)["cols_per_lane"] == 1        # too few channels for 8 shares
    assert cfg(128, 128, 1, B.PSC_F16)["cols_per_lane"] == 1      # fp16 keeps the one-column form


def test_row_kernel_stages_whole_planes_on_three_fp32_geometries():
    """At batch 256 the automatic choice runs the one-row-per-lane kernel
    with whole channel planes copied through LDS on fp32 16x16 at stride 1
    and on 8x8 and 16x16 at stride 2 (the CIFAR ResNet-18 shapes); fp16 and
    non-square planes of the same widths load their rows directly, and 32x32
    at stride 2 keeps the stride-2 kernel."""
    codes = [c for c in range(512) if bin(c).count("1") == 4 and (c >> 4) & 1][:6]
    def cfg(cin, cout, h, w, stride, dtype, n=256):
        L = B.Layer(cout, cin, codes, (cout * cin) * 3 // 10, dtype)
        return B.conv3x3_config(L, dtype, n, h, w, False, stride, 0)
    for cin, cout, hw, stride in ((128, 128, 16, 1), (256, 512, 8, 2), (128, 256, 16, 2)):
        c = cfg(cin, cout, hw, hw, stride, B.PSC_F32)
        assert (c["kernel"], c["staged"], c["rows_per_lane"]) == (4, 1, 1), (cin, cout, hw, stride, c)
        assert c["cols_per_lane"] == hw // stride
    for cin, cout, h, w, stride, dtype in ((256, 512, 8, 8, 2, B.PSC_F16), (128, 128, 16, 16, 1, B.PSC_F16),
                                           (128, 128, 15, 16, 1, B.PSC_F32), (256, 256, 8, 8, 1, B.PSC_F32)):
        c = cfg(cin, cout, h, w, stride, dtype)
        assert c["kernel"] == 4 and c["staged"] == 0, (cin, cout, h, w, stride, dtype, c)
    assert cfg(64, 128, 32, 32, 2, B.PSC_F32)["kernel"] == 3
    # batches that do not fill a wave with whole images stay off the row kernel
    assert cfg(128, 256, 16, 16, 2, B.PSC_F32, n=2)["kernel"] == 3
