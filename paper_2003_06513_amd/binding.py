"""Python binding of libpsc (ctypes).  Argument marshalling only: every step
of the path runs in the library's HIP kernels; torch supplies device memory
and the stream.

Function names follow the C entry points of include/psc.h without the
``psc_`` prefix.  If the shared library is missing it is built with hipcc; if
it cannot be loaded an ImportError is raised -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libpsc.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "psc.h")

PSC_OK, PSC_ERR_ARG, PSC_ERR_UNSUPPORTED, PSC_ERR_WORKSPACE, PSC_ERR_DEVICE, PSC_ERR_INTERNAL = range(6)
PSC_F32, PSC_F16 = 0, 1
PSC_OP_SELECT, PSC_OP_PACK = 0, 1
MAX_PATTERNS = 126

STATUS_NAMES = {0: "PSC_OK", 1: "PSC_ERR_ARG", 2: "PSC_ERR_UNSUPPORTED", 3: "PSC_ERR_WORKSPACE",
                4: "PSC_ERR_DEVICE", 5: "PSC_ERR_INTERNAL"}


class PscError(RuntimeError):
    def __init__(self, status: int, message: str, where: str):
        super().__init__("%s: %s (%s)" % (where, STATUS_NAMES.get(status, status), message))
        self.status = status
        self.message = message


class CLayer(ctypes.Structure):
    _fields_ = [("cout", ctypes.c_int32), ("cin", ctypes.c_int32), ("m", ctypes.c_int32),
                ("wdtype", ctypes.c_int32), ("keep", ctypes.c_int64),
                ("masks", ctypes.c_uint16 * MAX_PATTERNS)]


class CConvConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "kernel", "staged", "rows_per_lane", "cols_per_lane", "segments_per_wave", "column_tiles",
        "shares", "filters_per_block", "blocks", "threads_per_block")]


PACKED_FIELDS = ("filter_perm", "filter_ptr", "seg_ptr", "cin_idx", "pat_id", "values")


class CPacked(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PACKED_FIELDS]


_lib = None


def exported_names():
    """Function names declared in include/psc.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(psc_[a-z0-9_]+)\s*\(", text)))


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build()
    # torch ships its own HIP runtime under the same soname as the system's;
    # load it first so that libpsc binds to the runtime that owns the tensors
    # and streams it is given (one runtime per process)
    import torch  # noqa: F401
    try:
        L = ctypes.CDLL(LIB_PATH)
    except OSError as e:
        raise ImportError("cannot load %s: %s" % (LIB_PATH, e)) from e
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    LP, PP = ctypes.POINTER(CLayer), ctypes.POINTER(CPacked)
    sig = {
        "psc_last_error": ([], ctypes.c_char_p),
        "psc_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "psc_abi_version": ([], i32),
        "psc_select_library": ([P, i32, i64, i32, P], ctypes.c_int),
        "psc_workspace_size": ([LP, i32, ctypes.POINTER(sz)], ctypes.c_int),
        "psc_project": ([LP, P, P, P, P], ctypes.c_int),
        "psc_select": ([LP, P, P, P, sz, P], ctypes.c_int),
        "psc_select_noalloc": ([LP, P, P, P], ctypes.c_int),
        "psc_pack": ([LP, P, P, P, PP, P, sz, P], ctypes.c_int),
        "psc_unpack_dense": ([LP, PP, P, P], ctypes.c_int),
        "psc_conv3x3_fwd": ([LP, PP, i32, P, i32, i32, i32, P, i32, P, P], ctypes.c_int),
        "psc_conv3x3_fwd_algo": ([LP, PP, i32, P, i32, i32, i32, P, i32, P, i32, P], ctypes.c_int),
        "psc_probe_fma": ([i32, i32, P, P], ctypes.c_int),
        "psc_probe_mfma": ([i32, i32, P, P], ctypes.c_int),
        "psc_conv3x3_fwd_pool2": ([LP, PP, i32, P, i32, i32, i32, P, i32, P, i32, P], ctypes.c_int),
        "psc_conv3x3_fwd_strided": ([LP, PP, i32, P, i32, i32, i32, P, i32, P, i32, i32, P], ctypes.c_int),
        "psc_conv3x3_config": ([LP, i32, i32, i32, i32, i32, i32, i32, ctypes.POINTER(CConvConfig)],
                               ctypes.c_int),
        "psc_transpose_layer": ([LP, LP], ctypes.c_int),
        "psc_transpose_prep": ([LP, P, P, P, P, P, P, P], ctypes.c_int),
        "psc_conv3x3_bwd_weight_workspace": ([LP, i32, i32, i32, i32, ctypes.POINTER(sz)], ctypes.c_int),
        "psc_conv3x3_bwd_weight": ([LP, PP, i32, P, P, i32, i32, i32, P, P, P, sz, P], ctypes.c_int),
        "psc_admm_residual": ([P, P, i64, ctypes.c_float, P, P, P, sz, P], ctypes.c_int),
        "psc_dense3x3_bwd_weight_workspace": ([i32, i32, i32, i32, i32, ctypes.POINTER(sz)], ctypes.c_int),
        "psc_dense3x3_bwd_weight": ([P, P, i32, i32, i32, i32, i32, P, P, P, sz, P], ctypes.c_int),
        "psc_admm_primal": ([i64, P, P, P, P, i32, P, P, ctypes.c_float, ctypes.c_float, P, P], ctypes.c_int),
        "psc_admm_dual": ([LP, P, P, P, P, P, P], ctypes.c_int),
        "psc_dense3x3_fwd": ([i32, P, i32, i32, i32, i32, P, i32, P, i32, P, P], ctypes.c_int),
        "psc_maxpool2x2": ([i32, P, i32, i32, i32, i32, P, P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def last_error() -> str:
    return lib().psc_last_error().decode()


def _check(rc: int, where: str):
    if rc != PSC_OK:
        raise PscError(rc, last_error(), where)


# ------------------------------------------------------------------ helpers
def _torch():
    import torch
    return torch


def dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return PSC_F32
    if t.dtype == torch.float16:
        return PSC_F16
    raise TypeError("only float32 and float16 tensors are supported, got %s" % t.dtype)


def _dev(t, name):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Layer:
    """The per-layer representation (psc_layer)."""

    def __init__(self, cout: int, cin: int, masks, keep: int, dtype: int):
        masks = [int(v) for v in np.asarray(masks).reshape(-1)]
        self.c = CLayer()
        self.c.cout, self.c.cin, self.c.m = int(cout), int(cin), len(masks)
        self.c.wdtype = int(dtype)
        self.c.keep = int(keep)
        for i, v in enumerate(masks[:MAX_PATTERNS]):
            self.c.masks[i] = v
        self.masks = np.array(masks, dtype=np.uint16)

    cout = property(lambda self: self.c.cout)
    cin = property(lambda self: self.c.cin)
    m = property(lambda self: self.c.m)
    keep = property(lambda self: self.c.keep)
    dtype = property(lambda self: self.c.wdtype)

    def ref(self):
        return ctypes.byref(self.c)


class Packed:
    """Compressed weight storage held in device tensors (psc_packed)."""

    def __init__(self, layer: Layer, device="cuda"):
        torch = _torch()
        cout, m, keep = layer.cout, layer.m, layer.keep
        vdt = torch.float16 if layer.dtype == PSC_F16 else torch.float32
        self.filter_perm = torch.empty(cout, dtype=torch.int32, device=device)
        self.filter_ptr = torch.empty(cout + 1, dtype=torch.int32, device=device)
        self.seg_ptr = torch.empty(cout * (m + 1), dtype=torch.int32, device=device)
        self.cin_idx = torch.empty(keep, dtype=torch.int32, device=device)
        self.pat_id = torch.empty(keep, dtype=torch.uint8, device=device)
        self.values = torch.empty(keep * 4, dtype=vdt, device=device)

    def c(self) -> CPacked:
        cp = CPacked()
        for n in PACKED_FIELDS:
            t = getattr(self, n)
            setattr(cp, n, t.data_ptr() if t.numel() else None)
        return cp

    def to_host(self) -> dict:
        return {n: getattr(self, n).cpu().numpy() for n in PACKED_FIELDS}


# ------------------------------------------------------------------ entry points
def select_library(w: np.ndarray, m: int) -> np.ndarray:
    """Sec. 4.2 pattern library over every 3x3 kernel of ``w`` (host array)."""
    w = np.ascontiguousarray(w)
    if w.dtype == np.float32:
        dt = PSC_F32
    elif w.dtype == np.float16:
        dt = PSC_F16
    else:
        raise TypeError("w must be float32 or float16")
    out = np.zeros(m, dtype=np.uint16)
    _check(lib().psc_select_library(w.ctypes.data_as(ctypes.c_void_p), dt, w.size // 9, m,
                                    out.ctypes.data_as(ctypes.c_void_p)), "psc_select_library")
    return out


def workspace_size(layer: Layer, op: int) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().psc_workspace_size(layer.ref(), op, ctypes.byref(b)), "psc_workspace_size")
    return int(b.value)


def workspace(layer: Layer, op: int, device="cuda"):
    torch = _torch()
    n = workspace_size(layer, op)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def project(layer: Layer, w, pat, energy, stream=None):
    _check(lib().psc_project(layer.ref(), _dev(w, "w"), _dev(pat, "pat"), _dev(energy, "energy"),
                             _stream(stream)), "psc_project")


def select(layer: Layer, energy, keep_mask, ws, stream=None):
    _check(lib().psc_select(layer.ref(), _dev(energy, "energy"), _dev(keep_mask, "keep"),
                            _dev(ws, "ws"), ws.numel(), _stream(stream)), "psc_select")


def select_noalloc(layer: Layer, energy, keep_mask, stream=None):
    """psc_select_noalloc: psc_select with the library's own device scratch
    (no workspace, no allocation)."""
    _check(lib().psc_select_noalloc(layer.ref(), _dev(energy, "energy"), _dev(keep_mask, "keep"),
                                    _stream(stream)), "psc_select_noalloc")


def pack(layer: Layer, w, pat, keep_mask, packed: Packed, ws, stream=None):
    cp = packed.c()
    _check(lib().psc_pack(layer.ref(), _dev(w, "w"), _dev(pat, "pat"), _dev(keep_mask, "keep"),
                          ctypes.byref(cp), _dev(ws, "ws"), ws.numel(), _stream(stream)), "psc_pack")


def unpack_dense(layer: Layer, packed: Packed, w_dense, stream=None):
    cp = packed.c()
    _check(lib().psc_unpack_dense(layer.ref(), ctypes.byref(cp), _dev(w_dense, "w_dense"),
                                  _stream(stream)), "psc_unpack_dense")


def conv3x3_fwd(layer: Layer, packed: Packed, x, y, bias=None, relu: bool = False, algo: int = 0,
                stream=None):
    n, cin, h, w = (int(d) for d in x.shape)
    if cin != layer.cin or tuple(y.shape) != (n, layer.cout, h, w):
        raise ValueError("x/y shapes do not match the layer")
    cp = packed.c()
    _check(lib().psc_conv3x3_fwd_algo(layer.ref(), ctypes.byref(cp), dtype_code(x), _dev(x, "x"), n, h,
                                      w, _dev(bias, "bias"), int(bool(relu)), _dev(y, "y"), int(algo),
                                      _stream(stream)), "psc_conv3x3_fwd")


def conv3x3_fwd_pool2(layer: Layer, packed: Packed, x, y, bias=None, relu: bool = False, algo: int = 0,
                      stream=None):
    """psc_conv3x3_fwd_pool2: conv, sigma and the 2x2/2 max-pool in one pass;
    y is [n][cout][h/2][w/2]."""
    n, cin, h, w = (int(d) for d in x.shape)
    if cin != layer.cin or tuple(y.shape) != (n, layer.cout, h // 2, w // 2):
        raise ValueError("x/y shapes do not match the layer and the 2x2 pool")
    cp = packed.c()
    _check(lib().psc_conv3x3_fwd_pool2(layer.ref(), ctypes.byref(cp), dtype_code(x), _dev(x, "x"), n, h,
                                       w, _dev(bias, "bias"), int(bool(relu)), _dev(y, "y"), int(algo),
                                       _stream(stream)), "psc_conv3x3_fwd_pool2")


def conv3x3_fwd_strided(layer: Layer, packed: Packed, x, y, stride: int, bias=None, relu: bool = False,
                        algo: int = 0, stream=None):
    """psc_conv3x3_fwd_strided: y is [n][cout][(h-1)//stride+1][(w-1)//stride+1]."""
    n, cin, h, w = (int(d) for d in x.shape)
    stride = int(stride)
    if stride not in (1, 2):
        raise ValueError("stride must be 1 or 2")
    if cin != layer.cin or tuple(y.shape) != (n, layer.cout, (h - 1) // stride + 1, (w - 1) // stride + 1):
        raise ValueError("x/y shapes do not match the layer and the stride")
    cp = packed.c()
    _check(lib().psc_conv3x3_fwd_strided(layer.ref(), ctypes.byref(cp), dtype_code(x), _dev(x, "x"), n, h, w,
                                         _dev(bias, "bias"), int(bool(relu)), _dev(y, "y"), stride,
                                         int(algo), _stream(stream)), "psc_conv3x3_fwd_strided")


def conv3x3_config(layer: Layer, dtype: int, n: int, h: int, w: int, pool: bool = False, stride: int = 1,
                   algo: int = 0) -> dict:
    """psc_conv3x3_config: the launch configuration of a conv call (host only)."""
    c = CConvConfig()
    _check(lib().psc_conv3x3_config(layer.ref(), int(dtype), int(n), int(h), int(w), int(bool(pool)),
                                    int(stride), int(algo), ctypes.byref(c)), "psc_conv3x3_config")
    return {name: int(getattr(c, name)) for name, _ in CConvConfig._fields_}


def dense3x3_fwd(x, wd, y, bias=None, relu: bool = False, stream=None):
    n, cin, h, w = (int(d) for d in x.shape)
    cout = int(wd.shape[0])
    if tuple(wd.shape) != (cout, cin, 3, 3) or tuple(y.shape) != (n, cout, h, w):
        raise ValueError("shape mismatch")
    _check(lib().psc_dense3x3_fwd(dtype_code(x), _dev(x, "x"), n, cin, h, w, _dev(wd, "w"), cout,
                                  _dev(bias, "bias"), int(bool(relu)), _dev(y, "y"), _stream(stream)),
           "psc_dense3x3_fwd")


def probe_fma(blocks: int, iters: int, out, stream=None):
    """psc_probe_fma: 2 * 8 * iters * blocks * 256 fp32 FMA flops into out
    [blocks*256] (measurement only)."""
    _check(lib().psc_probe_fma(int(blocks), int(iters), _dev(out, "out"), _stream(stream)), "psc_probe_fma")


def probe_mfma(blocks: int, iters: int, out, stream=None):
    """psc_probe_mfma: 32768 * iters * blocks fp32 MFMA flops; out [blocks*256]
    (fp32, device) receives 16 * iters per lane."""
    _check(lib().psc_probe_mfma(int(blocks), int(iters), _dev(out, "out"), _stream(stream)), "psc_probe_mfma")


def maxpool2x2(x, y, stream=None):
    n, c, h, w = (int(d) for d in x.shape)
    if tuple(y.shape) != (n, c, h // 2, w // 2):
        raise ValueError("shape mismatch")
    _check(lib().psc_maxpool2x2(dtype_code(x), _dev(x, "x"), n, c, h, w, _dev(y, "y"), _stream(stream)),
           "psc_maxpool2x2")


def transpose_layer(layer: Layer) -> Layer:
    """psc_transpose_layer: the layer of dx = W^T dy (host only)."""
    out = CLayer()
    _check(lib().psc_transpose_layer(layer.ref(), ctypes.byref(out)), "psc_transpose_layer")
    return Layer(out.cout, out.cin, [out.masks[i] for i in range(out.m)], out.keep, out.wdtype)


def transpose_prep(layer: Layer, w, pat, keep_mask, w_t, pat_t, keep_t, stream=None):
    _check(lib().psc_transpose_prep(layer.ref(), _dev(w, "w"), _dev(pat, "pat"), _dev(keep_mask, "keep"),
                                    _dev(w_t, "w_t"), _dev(pat_t, "pat_t"), _dev(keep_t, "keep_t"),
                                    _stream(stream)), "psc_transpose_prep")


def _ws_bytes(tensor):
    return 0 if tensor is None else int(tensor.numel()) * tensor.element_size()


def conv3x3_bwd_weight_workspace(layer: Layer, dtype: int, n: int, h: int, w: int, device="cuda"):
    """A workspace tensor for psc_conv3x3_bwd_weight (None if it needs none)."""
    b = ctypes.c_size_t(0)
    _check(lib().psc_conv3x3_bwd_weight_workspace(layer.ref(), int(dtype), int(n), int(h), int(w), ctypes.byref(b)),
           "psc_conv3x3_bwd_weight_workspace")
    return None if b.value == 0 else _torch().empty(int(b.value), dtype=_torch().uint8, device=device)


def conv3x3_bwd_weight(layer: Layer, packed: Packed, x, dy, dvalues, dbias=None, ws=None, stream=None):
    n, cin, h, w = (int(d) for d in x.shape)
    if cin != layer.cin or tuple(dy.shape) != (n, layer.cout, h, w) or dvalues.numel() != 4 * layer.keep:
        raise ValueError("x/dy/dvalues shapes do not match the layer")
    if ws is None:
        ws = conv3x3_bwd_weight_workspace(layer, dtype_code(x), n, h, w, x.device)
    cp = packed.c()
    _check(lib().psc_conv3x3_bwd_weight(layer.ref(), ctypes.byref(cp), dtype_code(x), _dev(x, "x"), _dev(dy, "dy"),
                                        n, h, w, _dev(dvalues, "dvalues"), _dev(dbias, "dbias"), _dev(ws, "ws"),
                                        _ws_bytes(ws), _stream(stream)), "psc_conv3x3_bwd_weight")
    return ws


ADMM_RESIDUAL_WS_BYTES = 8192


def _f32(t, name):
    torch = _torch()
    if t is not None and t.dtype != torch.float32:
        raise TypeError("%s must be float32" % name)
    return _dev(t, name)


def admm_residual(z, target, scale: float, g, loss, ws, stream=None):
    """psc_admm_residual: g = 2 scale (relu(z) - t) [z > 0], loss (a float64
    device scalar) = scale * sum (relu(z) - t)^2."""
    if z.shape != target.shape or z.shape != g.shape:
        raise ValueError("z, target and g must have one shape")
    _check(lib().psc_admm_residual(_f32(z, "z"), _f32(target, "target"), int(z.numel()), float(scale),
                                   _f32(g, "g"), _dev(loss, "loss"), _dev(ws, "ws"), int(ws.numel()),
                                   _stream(stream)), "psc_admm_residual")


def dense3x3_bwd_weight_workspace(n: int, cin: int, h: int, w: int, cout: int, device="cuda"):
    b = ctypes.c_size_t(0)
    _check(lib().psc_dense3x3_bwd_weight_workspace(int(n), int(cin), int(h), int(w), int(cout), ctypes.byref(b)),
           "psc_dense3x3_bwd_weight_workspace")
    return None if b.value == 0 else _torch().empty(int(b.value), dtype=_torch().uint8, device=device)


def dense3x3_bwd_weight(x, g, dw, db=None, ws=None, stream=None):
    n, cin, h, w = (int(d) for d in x.shape)
    cout = int(g.shape[1])
    if tuple(g.shape) != (n, cout, h, w) or tuple(dw.shape) != (cout, cin, 3, 3):
        raise ValueError("x/g/dw shapes do not match")
    if ws is None:
        ws = dense3x3_bwd_weight_workspace(n, cin, h, w, cout, x.device)
    _check(lib().psc_dense3x3_bwd_weight(_f32(x, "x"), _f32(g, "g"), n, cin, h, w, cout, _f32(dw, "dw"),
                                         _f32(db, "db"), _dev(ws, "ws"), _ws_bytes(ws), _stream(stream)),
           "psc_dense3x3_bwd_weight")
    return ws


def admm_primal(w, dw, a, d, b, db, lr: float, rho: float, v, stream=None):
    _check(lib().psc_admm_primal(int(w.numel()), _f32(w, "w"), _f32(dw, "dw"), _f32(a, "a"), _f32(d, "d"),
                                 int(b.numel()) if b is not None else 0, _f32(b, "b"), _f32(db, "db"),
                                 float(lr), float(rho), _f32(v, "v"), _stream(stream)), "psc_admm_primal")


def admm_dual(layer: Layer, v, pat, keep_mask, a, d, stream=None):
    _check(lib().psc_admm_dual(layer.ref(), _f32(v, "v"), _dev(pat, "pat"), _dev(keep_mask, "keep"),
                               _f32(a, "a"), _f32(d, "d"), _stream(stream)), "psc_admm_dual")


def admm_rho(iteration: int, rho0: float = 1e-4, factor: float = 10.0, every_epochs: int = 11,
             iters_per_epoch: int = 10, rho_max: float = 1e-1) -> float:
    """The penalty schedule of the paper's settings (Sec. 5.1): rho starts at
    1e-4 and grows 10x every 11 epochs of 10 iterations until it reaches
    1e-1.  ``iteration`` counts from 1."""
    epoch = (int(iteration) - 1) // iters_per_epoch
    return min(rho_max, rho0 * factor ** (epoch // every_epochs))


class AdmmLayer:
    """Device state of the data-free ADMM pruning of one fp32 layer
    (Algorithm 1 for one n): W, b (updated by SGD), A, D, and the buffers of
    one iteration; every step runs in the library's kernels."""

    def __init__(self, w0, b0, masks, keep: int, lr: float = 1e-3, noalloc: bool = False):
        torch = _torch()
        self.w0, self.b0 = w0, b0
        self.w, self.b = w0.clone(), b0.clone()
        self.a, self.d = w0.clone(), torch.zeros_like(w0)
        self.dw, self.db, self.v = torch.empty_like(w0), torch.empty_like(b0), torch.empty_like(w0)
        cout, cin = int(w0.shape[0]), int(w0.shape[1])
        self.layer = Layer(cout, cin, masks, keep, PSC_F32)
        K = cout * cin
        self.pat = torch.empty(K, dtype=torch.uint8, device=w0.device)
        self.energy = torch.empty(K, dtype=torch.float64, device=w0.device)
        self.keep_mask = torch.empty(K, dtype=torch.uint8, device=w0.device)
        self.ws_sel = None if noalloc else workspace(self.layer, PSC_OP_SELECT, w0.device)
        self.ws_res = torch.empty(ADMM_RESIDUAL_WS_BYTES, dtype=torch.uint8, device=w0.device)
        self.loss = torch.zeros(1, dtype=torch.float64, device=w0.device)
        self.lr, self.k = float(lr), 0
        self._bufs = {}

    def _buf(self, name, shape):
        torch = _torch()
        t = self._bufs.get(name)
        if t is None or tuple(t.shape) != tuple(shape):
            t = self._bufs[name] = torch.empty(shape, dtype=torch.float32, device=self.w.device)
        return t

    def target(self, x, out=None, stream=None):
        """X' = relu(W0 X + b0): the pre-trained layer's output."""
        n, _, h, w = x.shape
        out = out if out is not None else self._buf("target", (n, self.layer.cout, h, w))
        dense3x3_fwd(x, self.w0, out, bias=self.b0, relu=True, stream=stream)
        return out

    def iteration(self, x, target, rho: float, scale: float, stream=None):
        """One iteration (Eq. 4, 6, 7) on the batch x with target X'."""
        n, _, h, w = x.shape
        z = self._buf("z", (n, self.layer.cout, h, w))
        g = self._buf("g", (n, self.layer.cout, h, w))
        dense3x3_fwd(x, self.w, z, bias=self.b, relu=False, stream=stream)
        admm_residual(z, target, scale, g, self.loss, self.ws_res, stream)
        ws = self._bufs.get("wgrad_ws")
        need = dense3x3_bwd_weight_workspace(n, self.layer.cin, h, w, self.layer.cout, x.device) \
            if "wgrad_shape" not in self._bufs or self._bufs["wgrad_shape"] != (n, h, w) else ws
        self._bufs["wgrad_ws"], self._bufs["wgrad_shape"] = need, (n, h, w)
        dense3x3_bwd_weight(x, g, self.dw, self.db, ws=need, stream=stream)
        admm_primal(self.w, self.dw, self.a, self.d, self.b, self.db, self.lr, rho, self.v, stream)
        project(self.layer, self.v, self.pat, self.energy, stream)
        if self.ws_sel is None:
            select_noalloc(self.layer, self.energy, self.keep_mask, stream)
        else:
            select(self.layer, self.energy, self.keep_mask, self.ws_sel, stream)
        admm_dual(self.layer, self.v, self.pat, self.keep_mask, self.a, self.d, stream)
        self.k += 1
        return self.loss


# ------------------------------------------------------------------ conveniences
class Prepared:
    """A pruned, packed layer: the result of project -> select -> pack."""

    def __init__(self, layer: Layer, packed: Packed, pat, energy, keep_mask, workspaces=()):
        self.layer, self.packed = layer, packed
        self.pat, self.energy, self.keep_mask = pat, energy, keep_mask
        # the select and pack workspaces live as long as the result: the
        # kernels that use them may still run on a stream other than torch's
        # current one, whose allocator would otherwise hand them out again
        self.workspaces = tuple(workspaces)


def prepare(w, masks, keep: int, stream=None) -> Prepared:
    """Project (Eq. 6), prune connectivity (Sec. 4.4) and pack (Sec. 3.4) the
    OIHW device tensor ``w``; device buffers are allocated with torch."""
    torch = _torch()
    cout, cin = int(w.shape[0]), int(w.shape[1])
    layer = Layer(cout, cin, masks, keep, dtype_code(w))
    K = cout * cin
    pat = torch.empty(K, dtype=torch.uint8, device=w.device)
    energy = torch.empty(K, dtype=torch.float64, device=w.device)
    keep_mask = torch.empty(K, dtype=torch.uint8, device=w.device)
    packed = Packed(layer, w.device)
    ws_sel = workspace(layer, PSC_OP_SELECT, w.device)
    ws_pack = workspace(layer, PSC_OP_PACK, w.device)
    project(layer, w, pat, energy, stream)
    select(layer, energy, keep_mask, ws_sel, stream)
    pack(layer, w, pat, keep_mask, packed, ws_pack, stream)
    return Prepared(layer, packed, pat, energy, keep_mask, (ws_sel, ws_pack))


def prepare_transposed(prep: Prepared, w, stream=None) -> Prepared:
    """The packed transposed layer of a prepared one (for dx = W^T dy):
    psc_transpose_prep on its dense weights ``w``, pattern ids and keep mask,
    then psc_pack with the rotated library."""
    torch = _torch()
    lt = transpose_layer(prep.layer)
    K = lt.cout * lt.cin
    w_t = torch.empty((lt.cout, lt.cin, 3, 3), dtype=w.dtype, device=w.device)
    pat_t = torch.empty(K, dtype=torch.uint8, device=w.device)
    keep_t = torch.empty(K, dtype=torch.uint8, device=w.device)
    transpose_prep(prep.layer, w, prep.pat, prep.keep_mask, w_t, pat_t, keep_t, stream)
    packed = Packed(lt, w.device)
    ws = workspace(lt, PSC_OP_PACK, w.device)
    pack(lt, w_t, pat_t, keep_t, packed, ws, stream)
    out = Prepared(lt, packed, pat_t, None, keep_t, (ws,))
    out.w = w_t
    return out


def conv(prep: Prepared, x, bias=None, relu: bool = False, algo: int = 0, out=None, stream=None):
    torch = _torch()
    n, _, h, w = x.shape
    y = out if out is not None else torch.empty((n, prep.layer.cout, h, w), dtype=x.dtype, device=x.device)
    conv3x3_fwd(prep.layer, prep.packed, x, y, bias=bias, relu=relu, algo=algo, stream=stream)
    return y
