"""GPU parity of the data-free ADMM pruning of one layer (Sec. 4.3, Eq. 4-7,
Algorithm 1) against the oracle, step by step: every step of an iteration
is compared with the oracle's fp64 arithmetic on the inputs that step got on
the GPU, so each step is held to its own bound; the integer decisions of
the projection (pattern ids, keep mask) and the bit copies of Eq. 6-7 (A,
D = V - A) must be bit-exact.  Runs several iterations in a row, with the
penalty schedule of the paper's settings, on small shapes and on the two
full-size ADMM workloads."""
import numpy as np
import pytest

import oracle
from oracle import admm
from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import U32, check_output, dev, gamma, note, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


def _h(t):
    return t.detach().cpu().numpy()


def _check_iteration(st, x, target_d, rho, scale, what):
    """Run one GPU iteration and compare every step with the oracle."""
    torch = torch_mod()
    w0, b0, a0, d0 = _h(st.w), _h(st.b), _h(st.a), _h(st.d)
    st.iteration(dev(x), target_d, rho, scale)
    torch.cuda.synchronize()
    n, cin, h, wd = x.shape
    cout = w0.shape[0]
    tgt = _h(target_d)
    z = _h(st._bufs["z"])
    # Z = W X + b: both gates against the dense oracle conv
    zr = admm.dense_layer(x, w0, b0)
    sz = oracle.conv_dense(np.abs(x), np.abs(w0), bias=np.abs(b0))
    check_output(z, zr, sz, np.float32, 9 * cin + 1, what + " Z")
    # residual: from the GPU's Z and target
    lr_, gr = admm.residual(z, tgt, scale)
    g = _h(st._bufs["g"])
    e_abs = np.abs(np.maximum(z.astype(np.float64), 0) - tgt)
    assert (np.abs(g - gr) <= 4 * U32 * 2 * scale * (e_abs + np.abs(tgt)) + 1e-38).all(), what + " G"
    loss = float(_h(st.loss)[0])
    assert abs(loss - lr_) <= 8 * U32 * abs(lr_) + 1e-30, what + " loss"
    # dense weight gradient of the GPU's G
    dwr, dbr = admm.dense_weight_grad(x, g)
    sdw, sdb = admm.dense_weight_grad(np.abs(x), np.abs(g))
    terms = n * h * wd
    assert (np.abs(_h(st.dw) - dwr) <= gamma(terms) * sdw + 1e-38).all(), what + " dW"
    assert (np.abs(_h(st.db) - dbr) <= gamma(terms) * sdb + 1e-38).all(), what + " db"
    # SGD step of Eq. 4 from the GPU's gradient
    dw, db = _h(st.dw), _h(st.db)
    wr, br = admm.primal_step(w0, dw, a0, d0, b0, db, st.lr, rho)
    bound = 8 * U32 * (np.abs(w0) + st.lr * (np.abs(dw) + rho * (np.abs(w0) + np.abs(a0) + np.abs(d0))))
    assert (np.abs(_h(st.w) - wr) <= bound + 1e-38).all(), what + " W"
    assert (np.abs(_h(st.b) - br) <= 4 * U32 * (np.abs(b0) + st.lr * np.abs(db)) + 1e-38).all(), what + " b"
    v = _h(st.v)
    assert v.tobytes() == (_h(st.w) + d0).astype(np.float32).tobytes(), what + " V = W + D"
    # Eq. 6-7 on the GPU's V: bit-exact
    ar, patr, keepr = admm.proximal_step(v, st.layer.masks, st.layer.keep)
    assert np.array_equal(_h(st.pat), patr), what + " pattern ids"
    assert np.array_equal(_h(st.keep_mask), keepr), what + " keep mask"
    assert _h(st.a).tobytes() == ar.tobytes(), what + " A"
    assert _h(st.d).tobytes() == (v - ar).tobytes(), what + " D"
    return loss


CASES = [
    # cout, cin, h, w, T, m, drop
    (8, 3, 9, 11, 2, 4, 0), (12, 10, 7, 6, 3, 6, 50), (16, 24, 14, 14, 2, 8, 60), (5, 7, 1, 1, 4, 8, 30),
    (20, 6, 5, 70, 2, 8, 40), (6, 5, 9, 12, 2, 6, 40), (4, 3, 6, 28, 3, 8, 50),
    # the matrix-core weight gradient: 16-channel blocks, 64-filter blocks,
    # ragged pixel tiles, partial sums over several blocks
    (70, 40, 9, 17, 2, 8, 50), (16, 16, 4, 5, 3, 4, 30),
]


@pytest.mark.parametrize("case", CASES)
def test_admm_iterations_stepwise(case):
    torch = torch_mod()
    cout, cin, h, w, T, m, drop = case
    w0 = inputs.he_weights(cout + 3 * cin, cout, cin)
    b0 = inputs.bias_vector(cout, cout)
    masks = oracle.select_library(w0, m)
    keep = inputs.keep_after_drop(cout * cin, drop)
    st = B.AdmmLayer(dev(w0), dev(b0), masks, keep, lr=0.05, noalloc=(cout % 2 == 1))
    rng = np.random.default_rng(cout)
    for k in range(1, 5):
        x = (rng.integers(0, 256, size=(T, cin, h, w)) / 255.0).astype(np.float32)
        note("admm %s iteration %d" % (case, k))
        tgt = st.target(dev(x))
        torch.cuda.synchronize()
        tr = admm.dense_layer(x, w0, b0)
        check_output(_h(tgt), np.maximum(tr, 0), oracle.conv_dense(np.abs(x), np.abs(w0), bias=np.abs(b0)),
                     np.float32, 9 * cin + 1, "target")
        # a large rho from the second iteration on, so A and D move
        _check_iteration(st, x, tgt, B.admm_rho(k) if k == 1 else 0.5, 1.0 / tgt.numel(), "%s k=%d" % (case, k))


@pytest.mark.parametrize("name", [wl.name for wl in inputs.admm_workloads()])
def test_admm_workload_full_size(name):
    torch = torch_mod()
    wl = [w for w in inputs.admm_workloads() if w.name == name][0]
    w0, b0 = wl.weights(), wl.bias()
    masks = oracle.select_library(w0, wl.m)
    st = B.AdmmLayer(dev(w0), dev(b0), masks, wl.layer.keep, lr=wl.lr)
    for k in ((1,) if wl.layer.h > 100 else (1, 2)):
        x = wl.batch_input(k)
        note("admm %s iteration %d" % (name, k))
        tgt = st.target(dev(x))
        torch.cuda.synchronize()
        _check_iteration(st, x, tgt, B.admm_rho(k), 1.0 / tgt.numel(), "%s k=%d" % (name, k))
