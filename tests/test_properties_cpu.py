"""Property tests over small random shapes (hypothesis), CPU only.

The oracle is checked against facts that hold for any input, computed
independently of it: Eq. 1 as a numpy cross-correlation of the masked dense
weights (stride 1 and 2, any height and width), the invariants of the
compressed storage of Sec. 3.4 and of the top-beta selection of Sec. 4.4,
and the adjoint identities of the retraining backward (Sec. 3.3).  The
library's host code is checked against the oracle (library selection) and
against the rules of its own configuration query."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
from paper_2003_06513_amd import binding as B

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])
CENTRE3 = [c for c in range(512) if (c >> 4) & 1 and bin(c).count("1") == 4]


@st.composite
def layers(draw, max_c=5, max_hw=9):
    cout = draw(st.integers(1, max_c))
    cin = draw(st.integers(1, max_c))
    m = draw(st.integers(1, 6))
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    integer = draw(st.booleans())             # small integers: many exact ties
    w = (rng.integers(-3, 4, size=(cout, cin, 3, 3)) if integer else rng.standard_normal((cout, cin, 3, 3)))
    w = w.astype(np.float32)
    keep = draw(st.integers(0, cout * cin))
    h = draw(st.integers(1, max_hw))
    wd = draw(st.integers(1, max_hw))
    n = draw(st.integers(1, 3))
    return w, m, keep, n, h, wd, rng


def prepared(w, m, keep):
    masks = oracle.select_library(w, m)
    pat, energy = oracle.project(w, masks)
    km = oracle.select(energy, keep)
    packed = oracle.pack(w, masks, pat, km)
    return masks, pat, energy, km, packed


def masked_dense(w, masks, pat, km):
    """M o W for the chosen patterns, dropped kernels zeroed (numpy)."""
    out = np.zeros_like(w, dtype=np.float64)
    cout, cin = w.shape[:2]
    for f in range(cout):
        for c in range(cin):
            k = f * cin + c
            if km[k]:
                code = int(masks[pat[k]])
                for q in range(9):
                    if (code >> q) & 1:
                        out[f, c, q // 3, q % 3] = w[f, c, q // 3, q % 3]
    return out


def xcorr(x, wd, stride, bias=None):
    """Eq. 1: 3x3 cross-correlation, zero padding 1, stride 1 or 2 (numpy)."""
    n, cin, h, w = x.shape
    cout = wd.shape[0]
    oh, ow = (h - 1) // stride + 1, (w - 1) // stride + 1
    xp = np.zeros((n, cin, h + 2, w + 2))
    xp[:, :, 1:-1, 1:-1] = x
    y = np.zeros((n, cout, oh, ow))
    for r in range(3):
        for s in range(3):
            patch = xp[:, :, r:r + stride * (oh - 1) + 1:stride, s:s + stride * (ow - 1) + 1:stride]
            y += np.einsum("ncij,fc->nfij", patch, wd[:, :, r, s])
    if bias is not None:
        y += np.asarray(bias, dtype=np.float64)[None, :, None, None]
    return y


@SETTINGS
@given(layers())
def test_conv_is_eq1_on_masked_weights(case):
    w, m, keep, n, h, wd_, rng = case
    masks, pat, _, km, packed = prepared(w, m, keep)
    wm = masked_dense(w, masks, pat, km)
    x = rng.standard_normal((n, w.shape[1], h, wd_)).astype(np.float32)
    bias = rng.standard_normal(w.shape[0]).astype(np.float32)
    for stride in (1, 2):
        got = oracle.conv_sparse_strided(x, packed, masks, w.shape[0], stride, bias=bias)
        ref = xcorr(x.astype(np.float64), wm, stride, bias)
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@SETTINGS
@given(layers())
def test_storage_invariants(case):
    w, m, keep, *_ = case
    cout, cin = w.shape[:2]
    masks, pat, energy, km, p = prepared(w, m, keep)
    assert sorted(p["filter_perm"].tolist()) == list(range(cout))
    fp = p["filter_ptr"]
    assert fp[0] == 0 and fp[-1] == keep and np.all(np.diff(fp) >= 0)
    counts = np.diff(fp)
    assert np.all(np.diff(counts) <= 0)                       # filters by kept count, descending
    seg = p["seg_ptr"].reshape(cout, m + 1)
    for i in range(cout):
        assert seg[i, 0] == fp[i] and seg[i, m] == fp[i + 1] and np.all(np.diff(seg[i]) >= 0)
        for q in range(m):
            ks = slice(seg[i, q], seg[i, q + 1])
            assert np.all(p["pat_id"][ks] == q)
            assert np.all(np.diff(p["cin_idx"][ks]) > 0)       # channels ascending, no repeats
    assert km.sum() == keep
    np.testing.assert_array_equal(oracle.unpack(p, masks, cout, cin), masked_dense(w, masks, pat, km))


@SETTINGS
@given(layers())
def test_selection_is_top_beta(case):
    w, m, keep, *_ = case
    masks, pat, energy, km, _ = prepared(w, m, keep)
    kept, dropped = energy[km == 1], energy[km == 0]
    if len(kept) and len(dropped):
        assert kept.min() >= dropped.max()
        # ties at the boundary go to the lower flat index
        e = kept.min()
        if dropped.max() == e:
            assert np.flatnonzero((energy == e) & (km == 1)).max() < np.flatnonzero((energy == e) & (km == 0)).min()
    # the projection keeps the largest energy over the library (first index on ties)
    for k in range(len(pat)):
        ek = [sum(float(w.reshape(-1, 9)[k, q]) ** 2 for q in range(9) if (int(c) >> q) & 1) for c in masks]
        assert pat[k] == int(np.argmax(ek))


@SETTINGS
@given(layers())
def test_backward_adjoints(case):
    w, m, keep, n, h, wd_, rng = case
    cout, cin = w.shape[:2]
    masks, pat, _, km, packed = prepared(w, m, keep)
    x = rng.standard_normal((n, cin, h, wd_))
    dy = rng.standard_normal((n, cout, h, wd_))
    y = oracle.conv_sparse(x.astype(np.float32), packed, masks, cout)
    x32 = x.astype(np.float32).astype(np.float64)
    dx = oracle.conv_sparse_bwd_data(dy, packed, masks, cin)
    dv, db = oracle.conv_sparse_bwd_weight(x32, dy, packed, masks)
    lhs = float(np.sum(y * dy))
    scale = float(np.sum(np.abs(y * dy))) + 1.0
    assert abs(lhs - float(np.sum(x32 * dx))) <= 1e-11 * scale              # <W x, dy> = <x, W^T dy>
    v = packed["values"].astype(np.float64)
    assert abs(lhs - float(np.sum(v * dv))) <= 1e-11 * scale                 # y is linear in the stored values
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2, 3)), rtol=1e-12, atol=1e-12)


@SETTINGS
@given(st.integers(1, 60), st.integers(1, 56), st.integers(0, 2**31 - 1), st.booleans(), st.booleans())
def test_library_selection_matches_oracle(nk, m, seed, integer, half):
    rng = np.random.default_rng(seed)
    w = rng.integers(-2, 3, size=(nk, 9)) if integer else rng.standard_normal((nk, 9))
    w = w.astype(np.float16 if half else np.float32)
    np.testing.assert_array_equal(B.select_library(w, m), oracle.select_library(w, m))


@SETTINGS
@given(st.integers(0, 300), st.integers(1, 70), st.integers(1, 260), st.sampled_from([1, 2]), st.booleans(),
       st.sampled_from([B.PSC_F32, B.PSC_F16]), st.integers(0, 3), st.integers(1, 600), st.integers(1, 600))
def test_config_query_rules(n, h, w, stride, pool, dt, algo, cin, cout):
    L = B.Layer(cout, cin, CENTRE3[:6], cin * cout // 3, dt)
    try:
        c = B.conv3x3_config(L, dt, n, h, w, pool, stride, algo)
    except B.PscError as e:
        assert (pool and (h % 2 or w % 2 or stride != 1)) or algo == 2 or \
            n * max(cin, cout) * h * w >= 2**31, str(e)
        return
    assert 0 <= c["kernel"] <= 4 and 1 <= c["shares"] <= 8
    assert c["threads_per_block"] % 64 == 0 and 64 <= c["threads_per_block"] <= 1024
    assert c["filters_per_block"] * c["shares"] * 64 == c["threads_per_block"] or c["kernel"] == 2
    if algo == 1:
        assert c["kernel"] == 2
    if algo == 2:
        assert c["kernel"] == 4 and not pool
    if c["kernel"] == 4:
        oh = (h - 1) // stride + 1
        assert c["segments_per_wave"] == 64 // (oh + 1) and c["cols_per_lane"] == (w - 1) // stride + 1
    if algo in (0, 3) and stride == 1 and c["kernel"] in (0, 1):
        assert c["rows_per_lane"] in (2, 4, 7, 8)


@SETTINGS
@given(st.integers(1, 40), st.integers(1, 40), st.lists(st.sampled_from(list(range(512))), min_size=1, max_size=12))
def test_transposed_layer_rotates_masks(cout, cin, codes):
    codes = sorted({c for c in codes if bin(c).count("1") == 4}) or [23]
    L = B.Layer(cout, cin, codes, cout * cin // 2, B.PSC_F32)
    T = B.transpose_layer(L)
    assert (T.cout, T.cin, T.keep) == (cin, cout, L.keep)
    rot = [int("".join(reversed(format(c, "09b"))), 2) for c in codes]   # bit q -> bit 8-q
    assert list(T.masks) == rot
    assert list(B.transpose_layer(T).masks) == codes
