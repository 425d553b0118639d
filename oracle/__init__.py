"""CPU oracle for pattern-sparse 3x3 convolution (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (the HIP library and its
Python binding) never does, and shares no code with it.

The arithmetic lives in ``pso.c`` (plain C, fp64, OpenMP over output planes);
this module compiles it on demand and wraps it with numpy.  Each wrapper names
the passage of Gong et al., "A Privacy-Preserving-Oriented DNN Pruning and
Mobile Acceleration Framework" (GLSVLSI'20), that it implements:

  select_library  Sec. 4.2   pattern-library heuristic (centre + 3 largest)
  project         Sec. 4.3   Eq. 6, projection onto the pattern set C_n
  select          Sec. 4.4   connectivity pruning, at most beta_n kernels
  pack / unpack   Sec. 3.4   filter kernel reorder + compressed weight storage
  mask_weights    Sec. 3.2   M o W with dropped kernels zeroed
  conv_sparse     Sec. 4.1   Eq. 1 layer, 3x3 stride 1 pad 1, from the storage
  conv_sparse_strided        the same layer with stride 2 (ResNet stage entries)
  conv_sparse_f32acc         the same loop in fp32 (timed CPU baseline only)
  conv_sparse_bwd_data   Sec. 3.3  retraining: dx, the adjoint of the Eq. 1 layer
  conv_sparse_bwd_weight Sec. 3.3  retraining: masked gradient of the stored values, bias
  conv_dense      Sec. 4.1   the same layer as a textbook dense loop (witness)
  maxpool2x2                 2x2/2 max-pool between the VGG-16 layers

Pins (see tests/test_oracle_*.py): brute-force projections on tiny layers,
closed forms, invariants, impulse responses and float64 torch.conv2d agreement.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pso.c")
_LIB_PATH = os.path.join(_HERE, "libpso.so")
_BENCH_PATH = os.path.join(_HERE, "libpso_bench.so")
_lib = None
_bench_lib = None

F32, F16 = 0, 1


def _compile(out: str, flags) -> None:
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc"] + list(flags) + ["-std=c99", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)


def build(force: bool = True) -> str:
    """Compile pso.c into oracle/libpso.so (gcc, OpenMP, no fast-math, no
    contraction: every add and multiply rounds as written) and, for the
    timed CPU baseline only, into oracle/libpso_bench.so (-O3, AVX2 + FMA:
    x86-64-v3, which this container and the GPU hosts both run)."""
    if force or not os.path.exists(_LIB_PATH):
        _compile(_LIB_PATH, ["-O3", "-ffp-contract=off", "-fno-fast-math"])
    if force or not os.path.exists(_BENCH_PATH):
        _compile(_BENCH_PATH, ["-O3", "-march=x86-64-v3"])
    return _LIB_PATH


def _declare(lib):
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.pso_num_threads.restype = ctypes.c_int
    lib.pso_set_num_threads.argtypes = [ctypes.c_int]
    lib.pso_set_num_threads.restype = None
    lib.pso_select_library.argtypes = [P, i32, i64, i32, P]
    lib.pso_project.argtypes = [P, i32, i64, P, i32, P, P]
    lib.pso_select.argtypes = [P, i64, i64, P]
    lib.pso_pack.argtypes = [P, i32, i32, i32, i32, P, P, P, P, P, P, P, P, P]
    lib.pso_mask_weights.argtypes = [P, i32, i64, P, i32, P, P, P]
    lib.pso_unpack.argtypes = [i32, i32, i32, i32, P, P, P, P, P, P, P]
    lib.pso_conv_sparse_st.argtypes = [P, i32, i32, i32, i32, i32, i32, P,
                                       P, P, P, P, P, i32, P, i32, i32, P, P]
    lib.pso_conv_sparse_f32acc.argtypes = [P, i32, i32, i32, i32, i32, i32, P,
                                           P, P, P, P, P, i32, P, i32, i32, P]
    lib.pso_conv_sparse_bwd_data.argtypes = [P, i32, i32, i32, i32, i32, i32, P,
                                             P, P, P, P, P, i32, P, P]
    lib.pso_conv_sparse_bwd_weight.argtypes = [P, P, i32, i32, i32, i32, i32, i32, P,
                                               P, P, P, P, P, P, P]
    lib.pso_conv_dense.argtypes = [P, i32, i32, i32, i32, i32, P, i32, P, i32, P]
    lib.pso_maxpool2x2.argtypes = [P, i64, i32, i32, P]
    for name in ("pso_select_library", "pso_project", "pso_select", "pso_pack",
                 "pso_mask_weights", "pso_unpack", "pso_conv_sparse_st",
                 "pso_conv_sparse_f32acc", "pso_conv_sparse_bwd_data", "pso_conv_sparse_bwd_weight",
                 "pso_conv_dense", "pso_maxpool2x2"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    _lib = _declare(ctypes.CDLL(_LIB_PATH))
    return _lib


def _load_bench():
    global _bench_lib
    if _bench_lib is not None:
        return _bench_lib
    if not os.path.exists(_BENCH_PATH):
        build(force=True)
    _bench_lib = _declare(ctypes.CDLL(_BENCH_PATH))
    return _bench_lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float16:
        return F16
    raise TypeError("oracle handles float32 and float16 arrays, got %s" % a.dtype)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s rejected its arguments" % what)


def num_threads() -> int:
    return int(_load().pso_num_threads())


def select_library(w: np.ndarray, m: int) -> np.ndarray:
    """Sec. 4.2: library of m centre+3 masks (bit 3r+s) from every 3x3 kernel
    in ``w`` (any shape ending in 3x3)."""
    w = np.ascontiguousarray(w)
    k = w.size // 9
    out = np.zeros(m, dtype=np.uint16)
    _check(_load().pso_select_library(_ptr(w), _dtype_code(w), k, m, _ptr(out)),
           "select_library")
    return out


def project(w: np.ndarray, masks: np.ndarray):
    """Sec. 4.3 Eq. 6: per kernel, the library index keeping the largest
    energy, and that energy (fp64)."""
    w = np.ascontiguousarray(w)
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    k = w.size // 9
    pat = np.zeros(k, dtype=np.uint8)
    energy = np.zeros(k, dtype=np.float64)
    _check(_load().pso_project(_ptr(w), _dtype_code(w), k, _ptr(masks),
                               len(masks), _ptr(pat), _ptr(energy)), "project")
    return pat, energy


def select(energy: np.ndarray, keep: int) -> np.ndarray:
    """Sec. 4.4: keep mask with exactly ``keep`` ones (largest energies,
    ties to the lower flat index)."""
    energy = np.ascontiguousarray(energy, dtype=np.float64)
    out = np.zeros(energy.size, dtype=np.uint8)
    _check(_load().pso_select(_ptr(energy), energy.size, int(keep), _ptr(out)),
           "select")
    return out


def pack(w: np.ndarray, masks: np.ndarray, pat: np.ndarray, keep: np.ndarray) -> dict:
    """Sec. 3.4: reordered, compressed storage of the pruned layer ``w``
    (OIHW, [cout][cin][3][3])."""
    w = np.ascontiguousarray(w)
    cout, cin = int(w.shape[0]), int(w.shape[1])
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    m = len(masks)
    pat = np.ascontiguousarray(pat, dtype=np.uint8)
    keep = np.ascontiguousarray(keep, dtype=np.uint8)
    beta = int(keep.astype(np.int64).sum())
    out = {
        "filter_perm": np.zeros(cout, dtype=np.int32),
        "filter_ptr": np.zeros(cout + 1, dtype=np.int32),
        "seg_ptr": np.zeros(cout * (m + 1), dtype=np.int32),
        "cin_idx": np.zeros(beta, dtype=np.int32),
        "pat_id": np.zeros(beta, dtype=np.uint8),
        "values": np.zeros(beta * 4, dtype=w.dtype),
    }
    _check(_load().pso_pack(_ptr(w), _dtype_code(w), cout, cin, m, _ptr(masks),
                            _ptr(pat), _ptr(keep), _ptr(out["filter_perm"]),
                            _ptr(out["filter_ptr"]), _ptr(out["seg_ptr"]),
                            _ptr(out["cin_idx"]), _ptr(out["pat_id"]),
                            _ptr(out["values"])), "pack")
    return out


def mask_weights(w, masks, pat, keep) -> np.ndarray:
    """Sec. 3.2: M o W for the chosen patterns, dropped kernels zeroed."""
    w = np.ascontiguousarray(w)
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    out = np.zeros_like(w)
    _check(_load().pso_mask_weights(
        _ptr(w), _dtype_code(w), w.size // 9, _ptr(masks), len(masks),
        _ptr(np.ascontiguousarray(pat, dtype=np.uint8)),
        _ptr(np.ascontiguousarray(keep, dtype=np.uint8)), _ptr(out)),
        "mask_weights")
    return out


def unpack(packed: dict, masks, cout: int, cin: int) -> np.ndarray:
    """Compressed storage back to dense OIHW in the original filter order."""
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    vals = np.ascontiguousarray(packed["values"])
    out = np.zeros((cout, cin, 3, 3), dtype=vals.dtype)
    _check(_load().pso_unpack(
        _dtype_code(vals), cout, cin, len(masks), _ptr(masks),
        _ptr(np.ascontiguousarray(packed["filter_perm"], dtype=np.int32)),
        _ptr(np.ascontiguousarray(packed["filter_ptr"], dtype=np.int32)),
        _ptr(np.ascontiguousarray(packed["cin_idx"], dtype=np.int32)),
        _ptr(np.ascontiguousarray(packed["pat_id"], dtype=np.uint8)),
        _ptr(vals), _ptr(out)), "unpack")
    return out


def _conv_args(x, packed, masks):
    x = np.ascontiguousarray(x)
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    vals = np.ascontiguousarray(packed["values"])
    if vals.size and vals.dtype != x.dtype:
        raise TypeError("weights and activations must share a dtype")
    idx = [np.ascontiguousarray(packed["filter_perm"], dtype=np.int32),
           np.ascontiguousarray(packed["filter_ptr"], dtype=np.int32),
           np.ascontiguousarray(packed["cin_idx"], dtype=np.int32),
           np.ascontiguousarray(packed["pat_id"], dtype=np.uint8)]
    vcode = _dtype_code(vals) if vals.size else F32
    return x, masks, vals, vcode, idx


def conv_sparse_strided(x: np.ndarray, packed: dict, masks, cout: int, stride: int, bias=None,
                        relu: bool = False, want_scale: bool = False):
    """Sec. 4.1 Eq. 1 with the compressed storage, stride 1 or 2, zero
    padding 1: fp64 output [n][cout][(h-1)//stride+1][(w-1)//stride+1] (and,
    with ``want_scale``, the per-output sum of |v*x| plus |b|).  fp32 and
    fp16 activations and bias are widened to fp64 (exactly) before the call."""
    x, masks, vals, vcode, idx = _conv_args(x, packed, masks)
    n, cin, h, w = (int(d) for d in x.shape)
    x64 = np.ascontiguousarray(x, dtype=np.float64)
    b64 = None if bias is None else np.ascontiguousarray(np.asarray(bias, dtype=x.dtype), dtype=np.float64)
    y = np.zeros((n, cout, (h - 1) // stride + 1, (w - 1) // stride + 1), dtype=np.float64)
    s = np.zeros_like(y) if want_scale else None
    _check(_load().pso_conv_sparse_st(
        _ptr(x64), n, cin, h, w, cout, len(masks), _ptr(masks), _ptr(idx[0]), _ptr(idx[1]),
        _ptr(idx[2]), _ptr(idx[3]), _ptr(vals), vcode, _ptr(b64), int(bool(relu)), int(stride),
        _ptr(y), _ptr(s)), "conv_sparse")
    return (y, s) if want_scale else y


def conv_sparse(x: np.ndarray, packed: dict, masks, cout: int, bias=None,
                relu: bool = False, want_scale: bool = False):
    """Sec. 4.1 Eq. 1 with the compressed storage, stride 1, zero padding 1:
    fp64 NCHW output (and, with ``want_scale``, the per-output sum of |v*x|
    plus |b|)."""
    return conv_sparse_strided(x, packed, masks, cout, 1, bias=bias, relu=relu, want_scale=want_scale)


def conv_sparse_f32acc(x: np.ndarray, packed: dict, masks, cout: int, stride: int = 1, bias=None,
                       relu: bool = False) -> np.ndarray:
    """The same loop accumulating in fp32 (-O3 x86-64-v3 build): the CPU
    baseline the benchmark times, never a parity reference.  Activations
    are taken as fp32 (fp16 widened before the call)."""
    x, masks, vals, vcode, idx = _conv_args(x, packed, masks)
    n, cin, h, w = (int(d) for d in x.shape)
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    b32 = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    y = np.zeros((n, cout, (h - 1) // stride + 1, (w - 1) // stride + 1), dtype=np.float32)
    _check(_load_bench().pso_conv_sparse_f32acc(
        _ptr(x32), n, cin, h, w, cout, len(masks), _ptr(masks), _ptr(idx[0]), _ptr(idx[1]),
        _ptr(idx[2]), _ptr(idx[3]), _ptr(vals), vcode, _ptr(b32), int(bool(relu)), int(stride),
        _ptr(y)), "conv_sparse_f32acc")
    return y


def bench_num_threads() -> int:
    return int(_load_bench().pso_num_threads())


def bench_set_num_threads(n: int) -> None:
    """Threads the fp32-accumulating baseline build uses from now on."""
    _load_bench().pso_set_num_threads(int(n))


def conv_sparse_bwd_data(dy: np.ndarray, packed: dict, masks, cin: int, want_scale: bool = False):
    """Sec. 3.3 retraining, backpropagation through the Eq. 1 layer (stride 1,
    pad 1): dx = the adjoint of the pattern-sparse conv applied to dy
    [n][cout][h][w]; fp64 [n][cin][h][w] (and, with ``want_scale``, the sum
    of the absolute terms)."""
    dy = np.ascontiguousarray(dy)
    n, cout, h, w = (int(d) for d in dy.shape)
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    vals = np.ascontiguousarray(packed["values"])
    idx = [np.ascontiguousarray(packed[k], dtype=t) for k, t in
           (("filter_perm", np.int32), ("filter_ptr", np.int32), ("cin_idx", np.int32), ("pat_id", np.uint8))]
    dy64 = np.ascontiguousarray(dy, dtype=np.float64)
    dx = np.zeros((n, cin, h, w), dtype=np.float64)
    s = np.zeros_like(dx) if want_scale else None
    _check(_load().pso_conv_sparse_bwd_data(
        _ptr(dy64), n, cin, h, w, cout, len(masks), _ptr(masks), _ptr(idx[0]), _ptr(idx[1]), _ptr(idx[2]),
        _ptr(idx[3]), _ptr(vals), _dtype_code(vals) if vals.size else F32, _ptr(dx), _ptr(s)),
        "conv_sparse_bwd_data")
    return (dx, s) if want_scale else dx


def conv_sparse_bwd_weight(x: np.ndarray, dy: np.ndarray, packed: dict, masks, want_scale: bool = False):
    """Sec. 3.3 retraining: the masked gradient -- dv [keep*4] of the stored
    values (storage order; pruned weights get none) and db [cout] of the
    bias -- of the Eq. 1 layer for the output gradient dy; fp64 (and, with
    ``want_scale``, the sum of the absolute terms of each dv entry)."""
    x = np.ascontiguousarray(x)
    dy = np.ascontiguousarray(dy)
    n, cin, h, w = (int(d) for d in x.shape)
    cout = int(dy.shape[1])
    if dy.shape != (n, cout, h, w):
        raise ValueError("dy must be [n][cout][h][w] of the layer's input size")
    masks = np.ascontiguousarray(masks, dtype=np.uint16)
    idx = [np.ascontiguousarray(packed[k], dtype=t) for k, t in
           (("filter_perm", np.int32), ("filter_ptr", np.int32), ("cin_idx", np.int32), ("pat_id", np.uint8))]
    keep = int(idx[2].size)
    dv = np.zeros(keep * 4, dtype=np.float64)
    s = np.zeros_like(dv) if want_scale else None
    db = np.zeros(cout, dtype=np.float64)
    _check(_load().pso_conv_sparse_bwd_weight(
        _ptr(np.ascontiguousarray(x, dtype=np.float64)), _ptr(np.ascontiguousarray(dy, dtype=np.float64)),
        n, cin, h, w, cout, len(masks), _ptr(masks), _ptr(idx[0]), _ptr(idx[1]), _ptr(idx[2]), _ptr(idx[3]),
        _ptr(dv), _ptr(s), _ptr(db)), "conv_sparse_bwd_weight")
    return (dv, db, s) if want_scale else (dv, db)


def conv_dense(x: np.ndarray, wdense: np.ndarray, bias=None, relu: bool = False):
    """Witness: textbook dense 3x3 convolution of OIHW weights, fp64 output."""
    x = np.ascontiguousarray(x)
    wdense = np.ascontiguousarray(wdense, dtype=x.dtype)
    n, cin, h, w = (int(d) for d in x.shape)
    cout = int(wdense.shape[0])
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=x.dtype)
    y = np.zeros((n, cout, h, w), dtype=np.float64)
    _check(_load().pso_conv_dense(_ptr(x), _dtype_code(x), n, cin, h, w,
                                  _ptr(wdense), cout, _ptr(bias),
                                  int(bool(relu)), _ptr(y)), "conv_dense")
    return y


def maxpool2x2(y: np.ndarray) -> np.ndarray:
    """2x2/2 max-pool of an fp64 NCHW array (the VGG-16 pooling)."""
    y = np.ascontiguousarray(y, dtype=np.float64)
    n, c, h, w = (int(d) for d in y.shape)
    out = np.zeros((n, c, h // 2, w // 2), dtype=np.float64)
    _check(_load().pso_maxpool2x2(_ptr(y), n * c, h, w, _ptr(out)), "maxpool2x2")
    return out
