"""CPU-only checks of the C ABI: the library loads, exports every entry point
of include/psc.h, validates arguments before any HIP call, and its host-side
pattern-library heuristic (Sec. 4.2) agrees bit for bit with the oracle."""
import ctypes

import numpy as np
import pytest

from paper_2003_06513_amd import binding as B
from synthetic import inputs

FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: every call below fails validation


@pytest.fixture(scope="module")
def L():
    return B.lib()


def _layer(cout=4, cin=3, masks=(23, 282), keep=5, dtype=B.PSC_F32):
    return B.Layer(cout, cin, list(masks), keep, dtype)


def test_exports_every_declared_symbol(L):
    names = B.exported_names()
    assert "psc_conv3x3_fwd" in names and len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
    assert L.psc_abi_version() == 1
    assert L.psc_status_string(3) == b"PSC_ERR_WORKSPACE"


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("m", [1, 4, 8, 12, 56])
def test_select_library_matches_oracle(oracle_lib, dtype, m):
    w = inputs.he_weights(40 + m, 32, 16, dtype)
    assert np.array_equal(B.select_library(w, m), oracle_lib.select_library(w, m))


def test_select_library_ties_and_specials_match_oracle(oracle_lib):
    rng = np.random.default_rng(1)
    w = rng.integers(-2, 3, size=(500, 3, 3)).astype(np.float32)   # many magnitude ties
    w[:10] = 0.0
    w[10:20] = -0.0
    for m in (3, 8, 56):
        assert np.array_equal(B.select_library(w, m), oracle_lib.select_library(w, m))
    h = (rng.standard_normal((300, 3, 3)) * 1e-6).astype(np.float16)  # fp16 subnormals
    assert np.array_equal(B.select_library(h, 8), oracle_lib.select_library(h, 8))


def test_select_library_rejects(L):
    w = np.zeros((1, 3, 3), dtype=np.float32)
    for m in (0, 57):
        with pytest.raises(B.PscError) as e:
            B.select_library(w, m)
        assert e.value.status == B.PSC_ERR_ARG
    rc = L.psc_select_library(None, 0, 1, 4, FAKE)
    assert rc == B.PSC_ERR_ARG and "h_w" in B.last_error()


def _status(rc):
    return rc, B.last_error()


def test_layer_validation(L):
    out = ctypes.c_size_t(0)
    rc, msg = _status(L.psc_workspace_size(None, 0, ctypes.byref(out)))
    assert rc == B.PSC_ERR_ARG and "NULL" in msg
    bad = [
        dict(masks=()),                         # m = 0
        dict(masks=tuple(range(127))),          # m > 126
        dict(masks=(23, 7)),                    # popcount 3
        dict(masks=(23, 23)),                   # duplicate
        dict(masks=(23, 600)),                  # not 9-bit
        dict(cout=0),
        dict(dtype=7),
    ]
    for kw in bad:
        lay = _layer(**kw)
        rc, msg = _status(L.psc_workspace_size(lay.ref(), 0, ctypes.byref(out)))
        assert rc == B.PSC_ERR_ARG, kw
        assert msg
    lay = _layer()
    assert L.psc_workspace_size(lay.ref(), 9, ctypes.byref(out)) == B.PSC_ERR_ARG
    assert L.psc_workspace_size(lay.ref(), B.PSC_OP_SELECT, ctypes.byref(out)) == B.PSC_OK
    assert out.value > 0 and out.value % 256 == 0
    assert L.psc_workspace_size(lay.ref(), B.PSC_OP_PACK, ctypes.byref(out)) == B.PSC_OK
    assert out.value > 0


def test_keep_validation(L):
    for keep in (-1, 13):
        lay = _layer(keep=keep)
        rc, msg = _status(L.psc_select(lay.ref(), FAKE, FAKE, FAKE, 1 << 20, None))
        assert rc == B.PSC_ERR_ARG and "keep" in msg


def test_workspace_validation(L):
    lay = _layer()
    rc, msg = _status(L.psc_select(lay.ref(), FAKE, FAKE, FAKE, 16, None))
    assert rc == B.PSC_ERR_WORKSPACE and "workspace" in msg
    rc, _ = _status(L.psc_select(lay.ref(), FAKE, FAKE, None, 0, None))
    assert rc == B.PSC_ERR_WORKSPACE
    rc, _ = _status(L.psc_select(lay.ref(), FAKE, FAKE, ctypes.c_void_p(0x10010), 1 << 20, None))
    assert rc == B.PSC_ERR_WORKSPACE                  # misaligned
    cp = B.CPacked(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    rc, _ = _status(L.psc_pack(lay.ref(), FAKE, FAKE, FAKE, ctypes.byref(cp), FAKE, 8, None))
    assert rc == B.PSC_ERR_WORKSPACE


def test_null_pointer_validation(L):
    lay = _layer()
    assert L.psc_project(lay.ref(), None, FAKE, FAKE, None) == B.PSC_ERR_ARG
    assert L.psc_select(lay.ref(), None, FAKE, FAKE, 1 << 20, None) == B.PSC_ERR_ARG
    cp = B.CPacked(FAKE.value, None, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    rc, msg = _status(L.psc_unpack_dense(lay.ref(), ctypes.byref(cp), FAKE, None))
    assert rc == B.PSC_ERR_ARG and "filter_ptr" in msg
    assert L.psc_unpack_dense(lay.ref(), None, FAKE, None) == B.PSC_ERR_ARG


def test_conv_validation(L):
    lay = _layer()
    cp = B.CPacked(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    # activation dtype differs from the weight dtype
    rc, msg = _status(L.psc_conv3x3_fwd(lay.ref(), ctypes.byref(cp), B.PSC_F16, FAKE, 1, 4, 4, None, 0,
                                        ctypes.c_void_p(0x20000), None))
    assert rc == B.PSC_ERR_UNSUPPORTED
    # misaligned packed values
    cp2 = B.CPacked(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value + 4)
    rc, msg = _status(L.psc_conv3x3_fwd(lay.ref(), ctypes.byref(cp2), B.PSC_F32, FAKE, 1, 4, 4, None, 0,
                                        ctypes.c_void_p(0x20000), None))
    assert rc == B.PSC_ERR_ARG and "aligned" in msg
    # bad shapes and algo
    for n, h, w in ((-1, 4, 4), (1, 0, 4), (1, 4, 0)):
        assert L.psc_conv3x3_fwd(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, n, h, w, None, 0,
                                 ctypes.c_void_p(0x20000), None) == B.PSC_ERR_ARG
    assert L.psc_conv3x3_fwd_algo(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 1, 4, 4, None, 0,
                                  ctypes.c_void_p(0x20000), 5, None) == B.PSC_ERR_ARG
    # the one-row-per-lane kernel has no variant for 5 columns
    rc, msg = _status(L.psc_conv3x3_fwd_algo(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 1, 4, 5, None, 0,
                                             ctypes.c_void_p(0x20000), 2, None))
    assert rc == B.PSC_ERR_UNSUPPORTED and "algo 2" in msg
    # output overlapping the input
    rc, msg = _status(L.psc_conv3x3_fwd(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 1, 4, 4, None, 0,
                                        ctypes.c_void_p(FAKE.value + 8), None))
    assert rc == B.PSC_ERR_ARG and "overlap" in msg
    # n == 0 is a no-op that succeeds without touching the device
    assert L.psc_conv3x3_fwd(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 0, 4, 4, None, 0, FAKE,
                             None) == B.PSC_OK
    # fused 2x2 pool: odd sizes rejected, n == 0 a no-op
    for h, w in ((5, 4), (4, 7)):
        rc, msg = _status(L.psc_conv3x3_fwd_pool2(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 1, h, w, None,
                                                  0, ctypes.c_void_p(0x20000), 0, None))
        assert rc == B.PSC_ERR_ARG and "even" in msg
    assert L.psc_conv3x3_fwd_pool2(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 0, 4, 4, None, 0, FAKE, 0,
                                   None) == B.PSC_OK
    # strided conv: only stride 1 or 2; the output size follows the stride
    for st in (0, 3, -1):
        rc, msg = _status(L.psc_conv3x3_fwd_strided(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 1, 5, 5, None,
                                                    0, ctypes.c_void_p(0x20000), st, 0, None))
        assert rc == B.PSC_ERR_ARG and "stride" in msg
    assert L.psc_conv3x3_fwd_strided(lay.ref(), ctypes.byref(cp), B.PSC_F32, FAKE, 0, 5, 5, None, 0, FAKE, 2, 0,
                                     None) == B.PSC_OK


def test_dense_and_pool_validation(L):
    assert L.psc_dense3x3_fwd(3, FAKE, 1, 2, 4, 4, FAKE, 2, None, 0, FAKE, None) == B.PSC_ERR_ARG
    assert L.psc_dense3x3_fwd(0, FAKE, 1, 0, 4, 4, FAKE, 2, None, 0, FAKE, None) == B.PSC_ERR_ARG
    assert L.psc_maxpool2x2(0, FAKE, 1, 2, 5, 4, FAKE, None) == B.PSC_ERR_ARG
    assert L.psc_maxpool2x2(0, None, 1, 2, 4, 4, FAKE, None) == B.PSC_ERR_ARG


def test_transpose_layer_rotates_masks_and_is_an_involution():
    L = B.Layer(6, 9, [23, 282, 58, 90, 113], 20, B.PSC_F16)
    T = B.transpose_layer(L)
    assert (T.cout, T.cin, T.keep, T.dtype) == (9, 6, 20, B.PSC_F16)
    for a, b in zip(L.masks, T.masks):
        assert all(((int(a) >> q) & 1) == ((int(b) >> (8 - q)) & 1) for q in range(9))
    TT = B.transpose_layer(T)
    assert np.array_equal(TT.masks, L.masks) and (TT.cout, TT.cin) == (6, 9)


def test_bwd_weight_validates(L):
    lay = _layer()
    pk = B.CPacked()
    for n_ in B.PACKED_FIELDS:
        setattr(pk, n_, 0x10000)
    import ctypes
    rc = L.psc_conv3x3_bwd_weight(lay.ref(), ctypes.byref(pk), B.PSC_F32, FAKE, FAKE, 1, 4, 4,
                                  ctypes.c_void_p(0x10004), None, FAKE, 1 << 30, None)
    assert rc == B.PSC_ERR_ARG and "16-byte" in B.last_error()
