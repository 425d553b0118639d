"""CPU oracle of one iteration of the data-free ADMM pattern pruning of one
layer (test infrastructure only, like the rest of ``oracle/``).

Gong et al., Sec. 4.3 and Algorithm 1 (Sec. 4.5): for layer n with input
X (a batch of synthetic data), pre-trained weights W0, b0 and target
X' = sigma(W0 X + b0), iteration k

  1. primal step (Eq. 4): one SGD step on
        f(W, b) = c * ||sigma(W X + b) - X'||_F^2 + rho/2 * ||W - A + D||_F^2
     W <- W - lr * (df/dW), b <- b - lr * (df/db);
  2. proximal step (Eq. 5-6): A = Euclidean projection of W + D onto the
     constraint set -- a pattern from the library per kernel (Sec. 4.3) and
     at most beta nonzero kernels (Sec. 4.4);
  3. dual step (Eq. 7): D <- D + W - A.

sigma is ReLU; c is the loss scale (1/numel(X') for the mean squared error
of the readings, 1 for the plain Frobenius norm of Eq. 2).  Everything is
fp64 except where a step's integer decision must be taken in the kernel's
precision: the proximal step projects W + D rounded once to fp32.  Each
function is the plain definition of its step; none shares code with the HIP
path.
"""
from __future__ import annotations

import numpy as np

from . import conv_dense, mask_weights, project, select


def dense_layer(x: np.ndarray, w: np.ndarray, b=None) -> np.ndarray:
    """Z = W X + b (Eq. 1 before sigma), 3x3, stride 1, zero padding 1, fp64."""
    return conv_dense(x, w, bias=b, relu=False)


def residual(z: np.ndarray, target: np.ndarray, scale: float):
    """The loss term of Eq. 4 and its gradient at Z: with e = relu(Z) - X',
    loss = c * sum e^2 and dloss/dZ = 2 c e * [Z > 0]."""
    z = np.asarray(z, dtype=np.float64)
    e = np.maximum(z, 0.0) - np.asarray(target, dtype=np.float64)
    loss = float(scale * np.sum(e * e))
    g = 2.0 * scale * e * (z > 0.0)
    return loss, g


def dense_weight_grad(x: np.ndarray, g: np.ndarray):
    """dW[o, i, r, s] = sum over n, h, w of g[n, o, h, w] * x[n, i, h + r - 1, w + s - 1]
    (zero padding) and db[o] = sum of g[n, o, :, :], fp64."""
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    n, cin, h, w = x.shape
    xp = np.zeros((n, cin, h + 2, w + 2))
    xp[:, :, 1:h + 1, 1:w + 1] = x
    cout = g.shape[1]
    dw = np.zeros((cout, cin, 3, 3))
    for img in range(n):
        gm = g[img].reshape(cout, h * w)                      # [o][(h, w)]
        for r in range(3):
            for s in range(3):
                xs = xp[img, :, r:r + h, s:s + w].reshape(cin, h * w)   # [i][(h, w)], shifted
                dw[:, :, r, s] += gm @ xs.T
    return dw, g.sum(axis=(0, 2, 3))


def primal_step(w, dw_loss, a, d, b, db, lr: float, rho: float):
    """Eq. 4, one SGD step: the gradient of the penalty rho/2 ||W - A + D||^2
    is rho (W - A + D)."""
    w, a, d = (np.asarray(t, dtype=np.float64) for t in (w, a, d))
    w_new = w - lr * (np.asarray(dw_loss, dtype=np.float64) + rho * (w - a + d))
    b_new = np.asarray(b, dtype=np.float64) - lr * np.asarray(db, dtype=np.float64)
    return w_new, b_new


def proximal_step(v32: np.ndarray, masks, keep: int):
    """Eq. 6 with the connectivity constraint: the projection of V = W + D
    (given as fp32) onto patterns + at most ``keep`` kernels -- per kernel the
    library pattern of largest kept energy, then the ``keep`` kernels of
    largest kept energy (the exact projection onto the intersection).
    Returns A (fp32, bit copies of V's kept entries), pattern ids and keep
    mask."""
    v32 = np.ascontiguousarray(v32, dtype=np.float32)
    pat, energy = project(v32, masks)
    keep_mask = select(energy, keep)
    return mask_weights(v32, masks, pat, keep_mask), pat, keep_mask


def dual_step(d, w, a):
    """Eq. 7: D <- D + W - A."""
    return np.asarray(d, dtype=np.float64) + np.asarray(w, dtype=np.float64) - np.asarray(a, dtype=np.float64)


def iteration(x, target, w, a, d, b, masks, keep: int, lr: float, rho: float, scale: float):
    """One full iteration (steps 1-3) from fp32 state; returns a dict of every
    intermediate (fp64 except A, which is fp32)."""
    z = dense_layer(x, w, b)
    loss, g = residual(z, target, scale)
    dw, db = dense_weight_grad(x, g)
    w_new, b_new = primal_step(w, dw, a, d, b, db, lr, rho)
    v32 = (w_new + np.asarray(d, dtype=np.float64)).astype(np.float32)
    a_new, pat, keep_mask = proximal_step(v32, masks, keep)
    d_new = dual_step(d, w_new, a_new)
    return dict(z=z, loss=loss, g=g, dw=dw, db=db, w=w_new, b=b_new, v=v32, a=a_new, pat=pat,
                keep=keep_mask, d=d_new)
