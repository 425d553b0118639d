"""Pins for the CPU oracle: each test checks it against something other than
itself -- hand-worked examples, closed forms, brute force on tiny layers,
invariants and a library routine (torch.conv2d in float64 on the CPU).

Paper: Gong et al., "A Privacy-Preserving-Oriented DNN Pruning and Mobile
Acceleration Framework", GLSVLSI'20.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from synthetic import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")
CENTRE3 = [c for c in range(512) if (c >> 4) & 1 and bin(c).count("1") == 4]
ALL4 = [c for c in range(512) if bin(c).count("1") == 4]


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _mask_array(code):
    return np.array([(code >> q) & 1 for q in range(9)], dtype=np.float64).reshape(3, 3)


def _pack_one_kernel(w33, mask, dtype=np.float32):
    """A 1x1 layer holding a single kernel, pruned to ``mask`` and packed."""
    w = np.asarray(w33, dtype=dtype).reshape(1, 1, 3, 3)
    masks = np.array([mask], dtype=np.uint16)
    pat, _ = oracle.project(w, masks)
    keep = np.ones(1, dtype=np.uint8)
    return oracle.pack(w, masks, pat, keep), masks


# ------------------------------------------------------------ worked examples
def test_worked_conv_tap_offsets():
    """Sec. 4.1 Eq. 1: the hand-computed 3x3 example (one digit per tap)."""
    g = _golden()["conv_tap_offsets"]
    packed, masks = _pack_one_kernel(np.zeros((3, 3)), g["mask"])
    packed["values"] = np.array(g["values"], dtype=np.float32)
    x = np.array(g["x"], dtype=np.float32).reshape(1, 1, 3, 3)
    y = oracle.conv_sparse(x, packed, masks, cout=1)
    assert np.array_equal(y[0, 0], np.array(g["y"], dtype=np.float64))


def test_worked_library_and_projection():
    """Sec. 4.2 + Eq. 6 on the hand-worked kernel."""
    g = _golden()["library_and_projection"]
    w = np.array(g["kernel"], dtype=np.float32).reshape(1, 1, 3, 3)
    lib = oracle.select_library(w, 1)
    assert int(lib[0]) == g["code"]
    masks = np.array(g["library"], dtype=np.uint16)
    pat, energy = oracle.project(w, masks)
    assert int(pat[0]) == g["pat"]
    assert energy[0] == g["energy"]
    assert float((w.astype(np.float64) ** 2).sum()) - energy[0] == 1.0


def test_worked_library_magnitude_tie():
    g = _golden()["library_tie"]
    w = np.array(g["kernel"], dtype=np.float32).reshape(1, 1, 3, 3)
    assert int(oracle.select_library(w, 1)[0]) == g["code"]


# ------------------------------------------------------------ Sec. 4.2 library
def _kernel_with_code(rng, code):
    """A kernel whose 3 largest-magnitude neighbours are exactly the
    non-centre bits of ``code`` (magnitudes 5..7 vs below 1, random signs)."""
    k = np.zeros(9, dtype=np.float32)
    big = [q for q in range(9) if (code >> q) & 1 and q != 4]
    for q in range(9):
        if q == 4:
            k[q] = rng.standard_normal()
        elif q in big:
            k[q] = (5 + 2 * rng.random()) * rng.choice([-1, 1])
        else:
            k[q] = rng.random() * rng.choice([-1, 1])
    return k.reshape(3, 3)


def test_library_frequency_order_and_fill():
    rng = np.random.default_rng(7)
    plan = {CENTRE3[10]: 5, CENTRE3[3]: 3, CENTRE3[20]: 3, CENTRE3[40]: 1}
    ks = []
    for code, cnt in plan.items():
        ks += [_kernel_with_code(rng, code) for _ in range(cnt)]
    rng.shuffle(ks)
    w = np.stack(ks)
    lib = [int(v) for v in oracle.select_library(w, 7)]
    # count 5, then the two count-3 codes in ascending code order, then count 1,
    # then unseen centre+3 codes in ascending order.
    expect = [CENTRE3[10], CENTRE3[3], CENTRE3[20], CENTRE3[40]]
    expect += [c for c in CENTRE3 if c not in expect][:3]
    assert lib == expect


def test_library_invariants_and_prefix_nesting():
    w = inputs.he_weights(11, 64, 32)
    libs = {m: [int(v) for v in oracle.select_library(w, m)] for m in (1, 4, 6, 8, 12, 56)}
    for m, lib in libs.items():
        assert len(lib) == m and len(set(lib)) == m
        for c in lib:
            assert (c >> 4) & 1 and bin(c).count("1") == 4
    for a, b in ((1, 4), (4, 6), (6, 8), (8, 12), (12, 56)):
        assert libs[a] == libs[b][:a]
    assert sorted(libs[56]) == CENTRE3


def test_library_fp16_matches_fp32_of_same_values():
    w = inputs.he_weights(12, 16, 16, np.float16)
    assert np.array_equal(oracle.select_library(w, 8),
                          oracle.select_library(w.astype(np.float32), 8))


def test_library_rejects_bad_m():
    w = np.zeros((1, 1, 3, 3), dtype=np.float32)
    for m in (0, 57):
        with pytest.raises(ValueError):
            oracle.select_library(w, m)


# ------------------------------------------------------------ Sec. 4.3 Eq. 6
def test_projection_is_nearest_pattern_bruteforce():
    """Eq. 6 closed form: ||W - M o W||^2 = ||W||^2 - e.  With small integer
    weights every sum is exact, so argmin distance and ties are exact."""
    rng = np.random.default_rng(3)
    w = rng.integers(-3, 4, size=(400, 3, 3)).astype(np.float32)
    masks = np.array(ALL4[::5][:12], dtype=np.uint16)
    pat, energy = oracle.project(w, masks)
    for k in range(w.shape[0]):
        wk = w[k].astype(np.float64)
        dist = [float(((wk - wk * _mask_array(c)) ** 2).sum()) for c in masks]
        best = min(dist)
        assert dist[pat[k]] == best
        assert pat[k] == dist.index(best)           # lowest index among ties
        assert energy[k] == float((wk ** 2).sum()) - best


def test_projection_special_cases():
    masks = np.array(CENTRE3[:8], dtype=np.uint16)
    # a zero kernel keeps pattern 0 with zero energy
    pat, e = oracle.project(np.zeros((2, 3, 3), dtype=np.float32), masks)
    assert list(pat) == [0, 0] and list(e) == [0.0, 0.0]
    # library of one pattern: everything maps to it
    w = inputs.he_weights(5, 8, 8)
    pat, _ = oracle.project(w, masks[:1])
    assert (pat == 0).all()
    # one dominant neighbour: the chosen pattern contains it
    rng = np.random.default_rng(9)
    for q in (0, 1, 2, 3, 5, 6, 7, 8):
        k = rng.standard_normal(9).astype(np.float32) * 0.01
        k[q] = -100.0
        pat, _ = oracle.project(k.reshape(1, 3, 3), masks)
        holders = [i for i, c in enumerate(masks) if (int(c) >> q) & 1]
        if holders:
            assert (int(masks[pat[0]]) >> q) & 1


def test_projection_fp16_exact_squares():
    w16 = inputs.he_weights(6, 8, 8, np.float16)
    masks = np.array(CENTRE3[::7], dtype=np.uint16)
    p16, e16 = oracle.project(w16, masks)
    p32, e32 = oracle.project(w16.astype(np.float32), masks)
    assert np.array_equal(p16, p32) and np.array_equal(e16, e32)


# ------------------------------------------------------------ Sec. 4.4
def _objective(w, masks, pat, keep):
    """||W - A||^2 for A = the pruned layer (exact for integer weights)."""
    tot = 0.0
    for k in range(w.shape[0]):
        wk = w[k].astype(np.float64)
        a = wk * _mask_array(int(masks[pat[k]])) if keep[k] else np.zeros((3, 3))
        tot += float(((wk - a) ** 2).sum())
    return tot


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_projection_onto_patterns_and_connectivity_bruteforce(seed):
    """Projection onto C_n (patterns) intersected with C'_n (at most beta
    nonzero kernels), brute-forced over every kept subset and every pattern
    choice on a 2x3 layer; the oracle's choice must attain the minimum."""
    rng = np.random.default_rng(seed)
    w = rng.integers(-4, 5, size=(6, 3, 3)).astype(np.float32)
    masks = np.array(CENTRE3[seed::9][:4], dtype=np.uint16)
    m = len(masks)
    pat, energy = oracle.project(w, masks)
    for beta in range(0, 7):
        keep = oracle.select(energy, beta)
        assert int(keep.sum()) == beta
        got = _objective(w, masks, pat, keep)
        best = None
        for subset in itertools.combinations(range(6), beta):
            kept = np.zeros(6, dtype=np.uint8)
            kept[list(subset)] = 1
            for choice in itertools.product(range(m), repeat=beta):
                pp = np.zeros(6, dtype=np.uint8)
                pp[list(subset)] = choice
                val = _objective(w, masks, pp, kept)
                best = val if best is None else min(best, val)
        assert got == best


def test_select_invariants_and_ties():
    rng = np.random.default_rng(4)
    e = rng.integers(0, 6, size=1000).astype(np.float64)      # many ties
    for beta in (0, 1, 137, 500, 999, 1000):
        keep = oracle.select(e, beta)
        assert int(keep.sum()) == beta
        if 0 < beta < 1000:
            kept, dropped = e[keep == 1], e[keep == 0]
            assert kept.min() >= dropped.max()
            t = kept.min()
            # at the boundary value, kept ones are exactly the lowest indices
            idx_t = np.nonzero(e == t)[0]
            n_kept_t = int((keep[idx_t] == 1).sum())
            assert (keep[idx_t[:n_kept_t]] == 1).all()
            assert (keep[idx_t[n_kept_t:]] == 0).all()


def test_select_rejects_bad_keep():
    with pytest.raises(ValueError):
        oracle.select(np.zeros(4), 5)


# ------------------------------------------------------------ Sec. 3.4 packing
def _check_pack_invariants(w, masks, pat, keep, packed):
    cout, cin = w.shape[:2]
    m = len(masks)
    perm, fptr = packed["filter_perm"], packed["filter_ptr"]
    seg, cidx, pid = packed["seg_ptr"].reshape(cout, m + 1), packed["cin_idx"], packed["pat_id"]
    beta = int(keep.sum())
    assert sorted(perm.tolist()) == list(range(cout))
    assert fptr[0] == 0 and fptr[-1] == beta and (np.diff(fptr) >= 0).all()
    keys = []
    seen = set()
    for i in range(cout):
        f = int(perm[i])
        kk = keep.reshape(cout, cin)[f]
        pp = pat.reshape(cout, cin)[f]
        n = int(kk.sum())
        assert fptr[i + 1] - fptr[i] == n
        cnt = [int(((kk == 1) & (pp == p)).sum()) for p in range(m)]
        keys.append((-n, [-c for c in cnt], f))
        assert seg[i, 0] == fptr[i] and seg[i, m] == fptr[i + 1]
        for p in range(m):
            a, b = int(seg[i, p]), int(seg[i, p + 1])
            assert b - a == cnt[p]
            assert (pid[a:b] == p).all()
            assert (np.diff(cidx[a:b]) > 0).all()
            for k in range(a, b):
                ci = int(cidx[k])
                assert kk[ci] == 1 and pp[ci] == p
                seen.add((f, ci))
    assert keys == sorted(keys)
    assert len(seen) == beta
    assert packed["values"].size == 4 * beta                  # 4 of 9 kept (Sec. 5.2: 2.25x)


def _second_packer(w, masks, pat, keep):
    """An independent packer: one global stable sort of (filter rank, pattern,
    ci) over kept kernels, with the filter order found by Python's sort."""
    cout, cin = w.shape[:2]
    m = len(masks)
    kk = keep.reshape(cout, cin)
    pp = pat.reshape(cout, cin)
    order = sorted(range(cout), key=lambda f: (-int(kk[f].sum()),
                   [-int(((kk[f] == 1) & (pp[f] == p)).sum()) for p in range(m)], f))
    rank = {f: i for i, f in enumerate(order)}
    items = sorted(((rank[f], int(pp[f, ci]), ci, f) for f in range(cout)
                    for ci in range(cin) if kk[f, ci]))
    vals = []
    for _, p, ci, f in items:
        flat = w[f, ci].reshape(9)
        vals += [flat[q] for q in range(9) if (int(masks[p]) >> q) & 1]
    return (np.array(order, dtype=np.int32),
            np.array([it[2] for it in items], dtype=np.int32),
            np.array([it[1] for it in items], dtype=np.uint8),
            np.array(vals, dtype=w.dtype))


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape,m,drop", [((8, 5), 4, 50), ((33, 17), 8, 60),
                                          ((64, 64), 8, 0), ((16, 3), 12, 100),
                                          ((5, 40), 1, 30)])
def test_pack_invariants_roundtrip_and_second_packer(dtype, shape, m, drop):
    cout, cin = shape
    w = inputs.he_weights(100 + cout, cout, cin, dtype)
    masks = oracle.select_library(w, m)
    pat, energy = oracle.project(w, masks)
    keep = oracle.select(energy, inputs.keep_after_drop(cout * cin, drop))
    packed = oracle.pack(w, masks, pat, keep)
    _check_pack_invariants(w, masks, pat, keep, packed)
    masked = oracle.mask_weights(w, masks, pat, keep)
    back = oracle.unpack(packed, masks, cout, cin)
    assert back.tobytes() == masked.tobytes()                # bitwise
    nz = (masked.reshape(-1, 9) != 0).sum(axis=1)
    assert (nz <= 4).all() and (nz[keep == 0] == 0).all()
    perm, cidx, pid, vals = _second_packer(w, masks, pat, keep)
    assert np.array_equal(perm, packed["filter_perm"])
    assert np.array_equal(cidx, packed["cin_idx"])
    assert np.array_equal(pid, packed["pat_id"])
    assert vals.tobytes() == packed["values"].tobytes()


# ------------------------------------------------------------ Sec. 4.1 Eq. 1
def _prepared(seed, cout, cin, m, drop, dtype=np.float32):
    w = inputs.he_weights(seed, cout, cin, dtype)
    masks = oracle.select_library(w, m)
    pat, energy = oracle.project(w, masks)
    keep = oracle.select(energy, inputs.keep_after_drop(cout * cin, drop))
    return w, masks, pat, keep, oracle.pack(w, masks, pat, keep)


@pytest.mark.parametrize("n,cin,cout,h,w", [(2, 5, 7, 9, 11), (1, 3, 4, 1, 1),
                                            (3, 8, 8, 2, 13), (1, 16, 6, 7, 3)])
@pytest.mark.parametrize("relu,use_bias", [(False, False), (True, True)])
def test_conv_sparse_equals_dense_witness_and_torch(n, cin, cout, h, w, relu, use_bias):
    torch = pytest.importorskip("torch")
    wt, masks, pat, keep, packed = _prepared(cin * 31 + cout, cout, cin, 8, 40)
    x = inputs.normal_activations(5, (n, cin, h, w))
    b = inputs.bias_vector(6, cout) if use_bias else None
    y = oracle.conv_sparse(x, packed, masks, cout, bias=b, relu=relu)
    masked = oracle.mask_weights(wt, masks, pat, keep)
    yd = oracle.conv_dense(x, masked, bias=b, relu=relu)
    scale = max(1.0, float(np.abs(yd).max()))
    assert float(np.abs(y - yd).max()) <= 1e-12 * scale
    yt = torch.nn.functional.conv2d(
        torch.from_numpy(x.astype(np.float64)), torch.from_numpy(masked.astype(np.float64)),
        None if b is None else torch.from_numpy(b.astype(np.float64)), stride=1, padding=1)
    if relu:
        yt = torch.relu(yt)
    assert float(np.abs(y - yt.numpy()).max()) <= 1e-12 * scale


def test_conv_impulse_reads_back_masked_kernel():
    cin, cout, h, w = 4, 6, 7, 8
    wt, masks, pat, keep, packed = _prepared(21, cout, cin, 6, 30)
    masked = oracle.mask_weights(wt, masks, pat, keep).astype(np.float64)
    h0, w0 = 3, 4
    for ci in range(cin):
        x = np.zeros((1, cin, h, w), dtype=np.float32)
        x[0, ci, h0, w0] = 1.0
        y = oracle.conv_sparse(x, packed, masks, cout)
        for co in range(cout):
            for r in range(3):
                for s in range(3):
                    assert y[0, co, h0 - r + 1, w0 - s + 1] == masked[co, ci, r, s]
        # nothing outside the 3x3 footprint
        y[0, :, h0 - 1:h0 + 2, w0 - 1:w0 + 2] = 0
        assert not y.any()


def test_conv_no_kernels_gives_sigma_of_bias():
    cin, cout = 5, 4
    wt, masks, pat, keep, packed = _prepared(22, cout, cin, 4, 100)
    assert packed["cin_idx"].size == 0
    x = inputs.normal_activations(1, (2, cin, 5, 6))
    b = np.array([1.5, -2.0, 0.0, 3.25], dtype=np.float32)
    y = oracle.conv_sparse(x, packed, masks, cout, bias=b, relu=False)
    assert np.array_equal(y, np.broadcast_to(b.reshape(1, cout, 1, 1), y.shape))
    y = oracle.conv_sparse(x, packed, masks, cout, bias=b, relu=True)
    assert np.array_equal(y, np.broadcast_to(np.maximum(b, 0).reshape(1, cout, 1, 1), y.shape))


def test_conv_all_ones_interior_is_weight_sum():
    cin, cout = 6, 5
    wt, masks, pat, keep, packed = _prepared(23, cout, cin, 8, 50)
    masked = oracle.mask_weights(wt, masks, pat, keep).astype(np.float64)
    y = oracle.conv_sparse(np.ones((1, cin, 6, 6), dtype=np.float32), packed, masks, cout)
    sums = masked.sum(axis=(1, 2, 3))
    for co in range(cout):
        assert np.allclose(y[0, co, 1:-1, 1:-1], sums[co], rtol=0, atol=1e-12)


def test_conv_linearity_and_relu():
    cin, cout = 7, 9
    wt, masks, pat, keep, packed = _prepared(24, cout, cin, 8, 60)
    x1 = inputs.normal_activations(1, (2, cin, 6, 5))
    x2 = inputs.normal_activations(2, (2, cin, 6, 5))
    split = np.random.default_rng(0).random(x1.shape) < 0.5
    x1[split] = 0.0           # disjoint supports and power-of-two scalings
    x2[~split] = 0.0          # keep a*x1 + b*x2 exact in fp32
    a, b = 0.5, -2.0
    y1 = oracle.conv_sparse(x1, packed, masks, cout)
    y2 = oracle.conv_sparse(x2, packed, masks, cout)
    y12 = oracle.conv_sparse((a * x1 + b * x2).astype(np.float32), packed, masks, cout)
    assert np.abs(y12 - (a * y1 + b * y2)).max() <= 1e-12 * np.abs(y12).max()
    yr = oracle.conv_sparse(x1, packed, masks, cout, relu=True)
    assert np.array_equal(yr, np.maximum(y1, 0.0))


def test_conv_fp16_converts_exactly():
    cin, cout = 6, 6
    w16, masks, pat, keep, p16 = _prepared(25, cout, cin, 8, 40, np.float16)
    x16 = inputs.normal_activations(3, (2, cin, 5, 7), np.float16)
    p32 = dict(p16)
    p32["values"] = p16["values"].astype(np.float32)
    y16 = oracle.conv_sparse(x16, p16, masks, cout)
    y32 = oracle.conv_sparse(x16.astype(np.float32), p32, masks, cout)
    assert np.array_equal(y16, y32)


def test_conv_scale_bounds_value():
    wt, masks, pat, keep, packed = _prepared(26, 4, 4, 8, 20)
    x = inputs.normal_activations(4, (1, 4, 6, 6))
    y, s = oracle.conv_sparse(x, packed, masks, 4, want_scale=True)
    assert (np.abs(y) <= s + 1e-12).all()


def test_non_centre_library_masks_supported():
    """The oracle accepts any distinct 4-of-9 masks (not only centre+3)."""
    masks = inputs.random_masks(8, 6, centre=False)
    w = inputs.he_weights(27, 5, 4)
    pat, energy = oracle.project(w, masks)
    keep = oracle.select(energy, 12)
    packed = oracle.pack(w, masks, pat, keep)
    masked = oracle.mask_weights(w, masks, pat, keep)
    x = inputs.normal_activations(5, (1, 4, 6, 5))
    y = oracle.conv_sparse(x, packed, masks, 5)
    yd = oracle.conv_dense(x, masked)
    assert np.abs(y - yd).max() <= 1e-12 * max(1.0, np.abs(yd).max())


def test_maxpool_matches_block_max():
    x = np.random.default_rng(0).standard_normal((2, 3, 6, 8))
    y = oracle.maxpool2x2(x)
    assert np.array_equal(y, x.reshape(2, 3, 3, 2, 4, 2).max(axis=(3, 5)))
    with pytest.raises(ValueError):
        oracle.maxpool2x2(np.zeros((1, 1, 3, 4)))


# ------------------------------------------- Eq. 1 with stride (stage entry)
@pytest.mark.parametrize("n,cin,cout,h,w", [(2, 5, 7, 9, 11), (1, 3, 4, 1, 1), (1, 6, 5, 2, 2),
                                            (3, 8, 8, 8, 13), (1, 16, 6, 7, 3)])
@pytest.mark.parametrize("relu,use_bias", [(False, False), (True, True)])
def test_conv_strided_equals_torch_and_subsampled_stride1(n, cin, cout, h, w, relu, use_bias):
    """Stride 2: torch.conv2d (fp64, CPU) on the masked dense weights, and the
    stride-1 output sampled at even rows and columns; stride 1 reduces to the
    pinned stride-1 conv."""
    torch = pytest.importorskip("torch")
    wt, masks, pat, keep, packed = _prepared(cin * 17 + cout, cout, cin, 8, 40)
    x = inputs.normal_activations(7, (n, cin, h, w))
    b = inputs.bias_vector(8, cout) if use_bias else None
    y2 = oracle.conv_sparse_strided(x, packed, masks, cout, 2, bias=b, relu=relu)
    assert y2.shape == (n, cout, (h + 1) // 2, (w + 1) // 2)
    masked = oracle.mask_weights(wt, masks, pat, keep)
    yt = torch.nn.functional.conv2d(
        torch.from_numpy(x.astype(np.float64)), torch.from_numpy(masked.astype(np.float64)),
        None if b is None else torch.from_numpy(b.astype(np.float64)), stride=2, padding=1)
    if relu:
        yt = torch.relu(yt)
    y1 = oracle.conv_sparse(x, packed, masks, cout, bias=b, relu=relu)
    scale = max(1.0, float(np.abs(y1).max()))
    assert yt.shape == y2.shape
    assert float(np.abs(y2 - yt.numpy()).max()) <= 1e-12 * scale
    assert float(np.abs(y2 - y1[:, :, ::2, ::2]).max()) <= 1e-12 * scale
    assert float(np.abs(oracle.conv_sparse_strided(x, packed, masks, cout, 1, bias=b, relu=relu) - y1).max()) \
        <= 1e-12 * scale


def test_conv_strided_impulse_footprint():
    """A unit impulse at input (h0, w0) reaches exactly the stride-2 outputs
    (oh, ow) with 2*oh + r - 1 = h0 and 2*ow + s - 1 = w0, with weight (r, s)."""
    cin, cout, h, w = 3, 4, 9, 8
    wt, masks, pat, keep, packed = _prepared(33, cout, cin, 6, 30)
    masked = oracle.mask_weights(wt, masks, pat, keep).astype(np.float64)
    for h0, w0 in [(0, 0), (3, 4), (4, 5), (8, 7)]:
        x = np.zeros((1, cin, h, w), dtype=np.float32)
        x[0, 1, h0, w0] = 1.0
        y = oracle.conv_sparse_strided(x, packed, masks, cout, 2)
        want = np.zeros_like(y)
        for r in range(3):
            for s in range(3):
                oh2, ow2 = h0 - r + 1, w0 - s + 1
                if oh2 % 2 == 0 and ow2 % 2 == 0 and 0 <= oh2 // 2 < y.shape[2] and 0 <= ow2 // 2 < y.shape[3]:
                    want[0, :, oh2 // 2, ow2 // 2] = masked[:, 1, r, s]
        assert np.array_equal(y, want)


def test_conv_strided_rejects_bad_stride():
    wt, masks, pat, keep, packed = _prepared(3, 2, 2, 4, 0)
    x = inputs.normal_activations(1, (1, 2, 4, 4))
    with pytest.raises(Exception):
        oracle.conv_sparse_strided(x, packed, masks, 2, 3)


# ------------------------------------------- error scale and the CPU baseline
@pytest.mark.parametrize("stride", [1, 2])
def test_conv_scale_equals_abs_conv_torch(stride):
    """The element-wise error scale s = sum |v*x| + |b| is the convolution of
    |x| with the absolute masked weights plus |b| (torch.conv2d in fp64 on
    the CPU), at stride 1 and 2."""
    torch = pytest.importorskip("torch")
    cin, cout = 7, 5
    wt, masks, pat, keep, packed = _prepared(41 + stride, cout, cin, 8, 35)
    x = inputs.normal_activations(9, (2, cin, 9, 10))
    b = inputs.bias_vector(11, cout)
    y, s = oracle.conv_sparse_strided(x, packed, masks, cout, stride, bias=b, want_scale=True)
    masked = np.abs(oracle.mask_weights(wt, masks, pat, keep).astype(np.float64))
    st = torch.nn.functional.conv2d(torch.from_numpy(np.abs(x.astype(np.float64))), torch.from_numpy(masked),
                                    torch.from_numpy(np.abs(b.astype(np.float64))), stride=stride, padding=1)
    assert st.shape == s.shape
    assert float(np.abs(s - st.numpy()).max()) <= 1e-12 * float(st.abs().max())
    assert (np.abs(y) <= s * (1 + 1e-12)).all()
    if stride == 2:
        _, s1 = oracle.conv_sparse(x, packed, masks, cout, bias=b, want_scale=True)
        assert np.array_equal(s, s1[:, :, ::2, ::2])


@pytest.mark.parametrize("stride", [1, 2])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_conv_f32acc_baseline_close_to_fp64(stride, dtype):
    """The fp32-accumulating build of the conv loop (the timed CPU baseline)
    stays within fp32 summation error of the fp64 oracle."""
    cin, cout = 40, 12
    wt, masks, pat, keep, packed = _prepared(52, cout, cin, 8, 50, dtype)
    x = inputs.normal_activations(13, (2, cin, 11, 12), dtype)
    b = inputs.bias_vector(14, cout, dtype)
    y, s = oracle.conv_sparse_strided(x, packed, masks, cout, stride, bias=b, relu=True, want_scale=True)
    y32 = oracle.conv_sparse_f32acc(x, packed, masks, cout, stride, bias=b, relu=True)
    nterms = 4 * cin + 1
    assert (np.abs(y32 - y) <= nterms * 2.0 ** -24 * s + 1e-30).all()


# ------------------------------------------- retraining (Sec. 3.3): backward
@pytest.mark.parametrize("n,cin,cout,h,w", [(2, 5, 7, 9, 11), (1, 3, 4, 1, 1), (1, 6, 5, 2, 3), (3, 8, 6, 7, 6)])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_backward_equals_torch_autograd(n, cin, cout, h, w, dtype):
    """dx, the masked dv and db equal torch autograd (fp64, CPU) of
    conv2d(x, masked weights, bias) against the output gradient dy; the
    weight gradient at pruned positions is what the retraining function
    zeroes, so only the kept positions are compared (all of them)."""
    torch = pytest.importorskip("torch")
    wt, masks, pat, keep, packed = _prepared(cin * 13 + cout, cout, cin, 8, 40, dtype)
    x = inputs.normal_activations(21, (n, cin, h, w), dtype)
    dy = inputs.normal_activations(22, (n, cout, h, w), dtype)
    masked = oracle.mask_weights(wt, masks, pat, keep).astype(np.float64)
    xt = torch.from_numpy(x.astype(np.float64)).requires_grad_(True)
    wt_t = torch.from_numpy(masked).requires_grad_(True)
    bt = torch.zeros(cout, dtype=torch.float64, requires_grad=True)
    y = torch.nn.functional.conv2d(xt, wt_t, bt, padding=1)
    (y * torch.from_numpy(dy.astype(np.float64))).sum().backward()
    dx = oracle.conv_sparse_bwd_data(dy, packed, masks, cin)
    dv, db = oracle.conv_sparse_bwd_weight(x, dy, packed, masks)
    sc = max(1.0, float(xt.grad.abs().max()))
    assert float(np.abs(dx - xt.grad.numpy()).max()) <= 1e-12 * sc
    # dv scattered to the kept positions of a dense array
    gp = dict(packed)
    gp["values"] = dv
    dense = np.zeros((cout, cin, 3, 3))
    for i, f in enumerate(packed["filter_perm"]):
        for k in range(packed["filter_ptr"][i], packed["filter_ptr"][i + 1]):
            pos = [q for q in range(9) if (int(masks[packed["pat_id"][k]]) >> q) & 1]
            for j, q in enumerate(pos):
                dense[f, packed["cin_idx"][k], q // 3, q % 3] = dv[4 * k + j]
    kept = masked != 0
    kept |= oracle.mask_weights(np.ones_like(wt), masks, pat, keep).astype(bool)
    sw = max(1.0, float(wt_t.grad.abs().max()))
    assert float(np.abs(dense - np.where(kept, wt_t.grad.numpy(), 0.0)).max()) <= 1e-12 * sw
    assert float(np.abs(db - bt.grad.numpy()).max()) <= 1e-12 * max(1.0, float(bt.grad.abs().max()))


def test_backward_adjoint_and_linearity_identities():
    """<conv(x), dy> = <x, dx(dy)> (dx is the adjoint), and since the layer is
    linear in its stored values, moving one value by e changes <conv(x), dy>
    by e * dv of that value (brute force through the forward oracle)."""
    cin, cout, h, w = 6, 5, 7, 8
    wt, masks, pat, keep, packed = _prepared(71, cout, cin, 6, 30)
    x = inputs.normal_activations(31, (2, cin, h, w))
    dy = inputs.normal_activations(32, (2, cout, h, w))
    y = oracle.conv_sparse(x, packed, masks, cout)
    dx = oracle.conv_sparse_bwd_data(dy, packed, masks, cin)
    lhs, rhs = float((y * dy.astype(np.float64)).sum()), float((x.astype(np.float64) * dx).sum())
    assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + 1.0)
    dv, _ = oracle.conv_sparse_bwd_weight(x, dy, packed, masks)
    rng = np.random.default_rng(5)
    for e in rng.choice(len(dv), size=6, replace=False):
        p2 = {k: v.copy() for k, v in packed.items()}
        p2["values"][e] += np.float32(0.5)
        step = float(p2["values"][e]) - float(packed["values"][e])   # the fp32 step actually taken
        y2 = oracle.conv_sparse(x, p2, masks, cout)
        delta = float(((y2 - y) * dy.astype(np.float64)).sum())
        assert abs(delta - step * dv[e]) <= 1e-10 * (abs(dv[e]) + 1.0)


def test_backward_scales_bound_values():
    cin, cout = 5, 4
    wt, masks, pat, keep, packed = _prepared(81, cout, cin, 8, 20)
    x = inputs.normal_activations(41, (2, cin, 6, 5))
    dy = inputs.normal_activations(42, (2, cout, 6, 5))
    dx, s = oracle.conv_sparse_bwd_data(dy, packed, masks, cin, want_scale=True)
    assert (np.abs(dx) <= s * (1 + 1e-12)).all()
    dv, db, sv = oracle.conv_sparse_bwd_weight(x, dy, packed, masks, want_scale=True)
    assert (np.abs(dv) <= sv * (1 + 1e-12)).all() and (sv > 0).all()
