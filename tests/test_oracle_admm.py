"""Pins of the ADMM oracle (Sec. 4.3 Eq. 4-7, Algorithm 1) against what the
mathematics fixes: torch autograd (fp64) for the weight gradient, central
differences of the Eq. 4 objective for the whole primal gradient, brute
force over the constraint set for the proximal step, and Eq. 7 for the dual
step."""
import itertools

import numpy as np
import pytest

import oracle
from oracle import admm
from synthetic import inputs


def _layer(seed=3, cout=4, cin=3, h=6, w=5, n=2):
    rng = np.random.default_rng(seed)
    x = (rng.integers(0, 256, size=(n, cin, h, w)) / 255.0).astype(np.float32)
    w0 = inputs.he_weights(seed, cout, cin)
    b0 = inputs.bias_vector(seed + 1, cout)
    return x, w0, b0


def test_dense_weight_grad_equals_torch_autograd():
    torch = pytest.importorskip("torch")
    x, w0, b0 = _layer()
    g = np.random.default_rng(7).standard_normal((2, 4, 6, 5))
    xt = torch.from_numpy(x.astype(np.float64))
    wt = torch.from_numpy(w0.astype(np.float64)).requires_grad_(True)
    bt = torch.from_numpy(b0.astype(np.float64)).requires_grad_(True)
    (torch.nn.functional.conv2d(xt, wt, bt, padding=1) * torch.from_numpy(g)).sum().backward()
    dw, db = admm.dense_weight_grad(x, g)
    assert np.abs(dw - wt.grad.numpy()).max() <= 1e-12 * float(wt.grad.abs().max())
    assert np.abs(db - bt.grad.numpy()).max() <= 1e-12 * float(bt.grad.abs().max())


def test_primal_gradient_matches_central_differences():
    """The SGD step of Eq. 4 moves W along -(dloss/dW + rho (W - A + D)): that
    gradient agrees with central differences of the objective computed by
    torch conv2d in fp64 (a different routine) at every weight and bias."""
    torch = pytest.importorskip("torch")
    x, w0, b0 = _layer(seed=5)
    target = np.maximum(admm.dense_layer(x, w0, b0), 0.0) * 0.9 + 0.01
    rng = np.random.default_rng(2)
    w = (w0 + 0.05 * rng.standard_normal(w0.shape)).astype(np.float32)
    b = b0.copy()
    a = (w0 * (rng.random(w0.shape) < 0.5)).astype(np.float32)
    d = (0.01 * rng.standard_normal(w0.shape)).astype(np.float32)
    rho, scale = 0.3, 1.0 / target.size

    def f(wv, bv):
        z = torch.nn.functional.conv2d(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(wv),
                                       torch.from_numpy(bv), padding=1)
        e = torch.relu(z) - torch.from_numpy(target)
        return float(scale * (e * e).sum() + rho / 2 * ((torch.from_numpy(wv - a + d)) ** 2).sum())

    z = admm.dense_layer(x, w, b)
    assert np.abs(z).min() > 1e-4        # no Z at the kink of ReLU
    _, g = admm.residual(z, target, scale)
    dw, db = admm.dense_weight_grad(x, g)
    grad_w = dw + rho * (w.astype(np.float64) - a + d)
    w64, b64 = w.astype(np.float64), b.astype(np.float64)
    eps = 1e-6
    for idx in itertools.product(range(4), range(3), range(3), range(3)):
        wp, wm = w64.copy(), w64.copy()
        wp[idx] += eps
        wm[idx] -= eps
        fd = (f(wp, b64) - f(wm, b64)) / (2 * eps)
        assert abs(fd - grad_w[idx]) <= 1e-6 * (abs(grad_w[idx]) + 1e-3)
    for o in range(4):
        bp, bm = b64.copy(), b64.copy()
        bp[o] += eps
        bm[o] -= eps
        fd = (f(w64, bp) - f(w64, bm)) / (2 * eps)
        assert abs(fd - db[o]) <= 1e-6 * (abs(db[o]) + 1e-3)


def test_proximal_step_is_the_nearest_point_of_the_constraint_set():
    """Brute force over every choice of pattern per kernel and every subset
    of `keep` kernels of a 2x2 layer: A is a minimiser of ||V - A||."""
    rng = np.random.default_rng(11)
    masks = inputs.random_masks(4, 4)
    for trial in range(5):
        v = rng.standard_normal((2, 2, 3, 3)).astype(np.float32)
        for keep in range(0, 5):
            a, pat, keep_mask = admm.proximal_step(v, masks, keep)
            assert int(keep_mask.sum()) == keep
            best = np.inf
            vk = v.reshape(4, 9).astype(np.float64)
            for subset in itertools.combinations(range(4), keep):
                for pats in itertools.product(range(len(masks)), repeat=keep):
                    cand = np.zeros((4, 9))
                    for kk, p in zip(subset, pats):
                        for q in range(9):
                            if (int(masks[p]) >> q) & 1:
                                cand[kk, q] = vk[kk, q]
                    best = min(best, float(((vk - cand) ** 2).sum()))
            got = float(((vk - a.reshape(4, 9).astype(np.float64)) ** 2).sum())
            assert got == best


def test_dual_step_is_eq7_and_equals_v_minus_a():
    """Eq. 7 literally, and its closed form given the projection: A keeps
    bit copies of V's entries or zeros them, so D + W - A is V - A up to the
    one rounding of V = W + D to fp32."""
    x, w0, b0 = _layer(seed=9, cout=6, cin=5)
    masks = oracle.select_library(w0, 6)
    target = np.maximum(admm.dense_layer(x, w0, b0), 0.0)
    rng = np.random.default_rng(4)
    w = (w0 + 0.1 * rng.standard_normal(w0.shape)).astype(np.float32)
    d = (0.05 * rng.standard_normal(w0.shape)).astype(np.float32)
    it = admm.iteration(x, target, w, w0, d, b0, masks, 15, 1e-2, 0.1, 1.0 / target.size)
    eq7 = d.astype(np.float64) + it["w"] - it["a"].astype(np.float64)
    closed = it["v"].astype(np.float64) - it["a"].astype(np.float64)
    assert np.array_equal(it["d"], eq7)
    assert (np.abs(eq7 - closed) <= 2.0 ** -24 * np.abs(it["v"].astype(np.float64)) + 1e-300).all()
    # A lies in the constraint set: kept kernels use their pattern's positions only
    a = it["a"].reshape(-1, 9)
    for k in range(a.shape[0]):
        allowed = [(int(masks[it["pat"][k]]) >> q) & 1 for q in range(9)] if it["keep"][k] else [0] * 9
        assert all(allowed[q] or a[k, q] == 0 for q in range(9))
    assert int(it["keep"].sum()) == 15
