"""The C ABI on the host: the library loads, exports every function declared in
include/agnes.h, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "agnes.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(agnes_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def ag():
    import paper_2601_01473_amd as m
    from paper_2601_01473_amd import _binding
    if not os.path.exists(_binding.LIB_PATH):
        from paper_2601_01473_amd import build
        build.build()
    return m


def test_header_declares_the_boundary():
    fns = declared_functions()
    for f in ("agnes_build_blocks", "agnes_hyperbatch_prepare", "agnes_free", "agnes_last_error",
              "agnes_batch_view_get", "agnes_batch_stats"):
        assert f in fns


def test_every_declared_symbol_is_exported(ag):
    from paper_2601_01473_amd import _binding
    lib = ctypes.CDLL(_binding.LIB_PATH)
    for f in declared_functions():
        assert hasattr(lib, f), f
    assert sorted(_binding.EXPORTED) == declared_functions()


def _store(ag, off, idx, feat, bb, **kw):
    return ag.Store(np.asarray(off), np.asarray(idx, dtype=np.int32), feat, bb, **kw)


@pytest.mark.parametrize("off,idx,bb,msg", [
    ([0, 2, 1], [0, 1], 64, "nondecreasing"),
    ([1, 1, 2], [0, 1], 64, "offsets[0]"),
    ([0, 1, 3], [0, 1], 64, "num_edges"),
    ([0, 1, 2], [0, 5], 64, "out of range"),
    ([0, 1, 2], [0, -1], 64, "out of range"),
    ([0, 1, 2], [0, 1], 48, "power of two"),
    ([0, 1, 2], [0, 1], 8, "power of two"),
    ([0, 1, 2], [0, 1], 1 << 25, "power of two"),
])
def test_build_rejects_bad_inputs(ag, off, idx, bb, msg):
    with pytest.raises(ag.AgnesError) as e:
        _store(ag, np.array(off, np.int64), idx, np.zeros((2, 4), np.float32), bb)
    assert e.value.status == 1
    assert msg in str(e.value)
    assert msg in ag.agnes_last_error()


def test_build_rejects_rows_larger_than_blocks(ag):
    with pytest.raises(ag.AgnesError) as e:
        _store(ag, np.array([0, 1, 2], np.int64), [1, 0], np.zeros((2, 32), np.float32), 64)
    assert "block_bytes must be >= row_bytes" in str(e.value)


def test_build_rejects_odd_row_bytes(ag):
    with pytest.raises(ag.AgnesError) as e:
        _store(ag, np.array([0, 1, 2], np.int64), [1, 0], np.zeros((2, 3), np.float16), 64)
    assert "multiple of 4" in str(e.value)


def test_build_rejects_null_and_bad_dtypes(ag):
    from paper_2601_01473_amd import _binding as B
    lib = B.lib()
    out = ctypes.c_void_p()
    assert lib.agnes_build_blocks(None, None, 64, None, ctypes.byref(out)) == B.AGNES_ERR_INVALID
    assert out.value is None
    off = np.array([0, 1], np.int64)
    idx = np.array([0], np.int32)
    feat = np.zeros((1, 4), np.float32)
    csr = B.agnes_csr(1, 1, 7, off.ctypes.data, idx.ctypes.data)
    fs = B.agnes_features(feat.ctypes.data, 4, B.AGNES_FLOAT32)
    assert lib.agnes_build_blocks(ctypes.byref(csr), ctypes.byref(fs), 64, None, ctypes.byref(out)) == 1
    csr = B.agnes_csr(1, 1, B.AGNES_INT64, off.ctypes.data, idx.ctypes.data)
    fs = B.agnes_features(feat.ctypes.data, 4, B.AGNES_INT32)
    assert lib.agnes_build_blocks(ctypes.byref(csr), ctypes.byref(fs), 64, None, ctypes.byref(out)) == 1
    csr = B.agnes_csr(0, 0, B.AGNES_INT64, off.ctypes.data, None)
    fs = B.agnes_features(feat.ctypes.data, 4, B.AGNES_FLOAT32)
    assert lib.agnes_build_blocks(ctypes.byref(csr), ctypes.byref(fs), 64, None, ctypes.byref(out)) == 1
    assert lib.agnes_build_blocks(ctypes.byref(csr), ctypes.byref(fs), 64, None, None) == 1


def test_prepare_rejects_bad_handles(ag):
    from paper_2601_01473_amd import _binding as B
    lib = B.lib()
    out = ctypes.c_void_p()
    fan = (ctypes.c_int32 * 1)(3)
    bogus = (ctypes.c_uint32 * 16)()
    rc = lib.agnes_hyperbatch_prepare(ctypes.cast(bogus, ctypes.c_void_p), None, 1, 1, fan, 1, 0, 0, None,
                                      ctypes.byref(out))
    assert rc == B.AGNES_ERR_INVALID and out.value is None
    assert "store" in ag.agnes_last_error()
    assert lib.agnes_hyperbatch_prepare(None, None, 1, 1, fan, 1, 0, 0, None, None) == 1


def test_free_null_and_unknown_are_noops(ag):
    ag.agnes_free(None)
    from paper_2601_01473_amd import _binding as B
    bogus = (ctypes.c_uint32 * 4)()
    B.lib().agnes_free(ctypes.cast(bogus, ctypes.c_void_p))


def test_view_and_stats_reject_bad_handles(ag):
    from paper_2601_01473_amd import _binding as B
    lib = B.lib()
    bogus = (ctypes.c_uint32 * 4)()
    v = B.agnes_batch_view()
    assert lib.agnes_batch_view_get(ctypes.cast(bogus, ctypes.c_void_p), ctypes.byref(v)) == 1
    s = B.agnes_stats()
    assert lib.agnes_batch_stats(None, ctypes.byref(s)) == 1
    assert lib.agnes_store_set_option(None, 1, 1) == 1
    info = (ctypes.c_int64 * 8)()
    assert lib.agnes_store_info(None, info) == 1


def test_device_allocator_needs_both_callbacks(ag):
    """Host-only: the setter checks its arguments and touches no device."""
    from paper_2601_01473_amd import _binding as B
    alloc = B.DEVICE_ALLOC_FN(lambda nbytes, user: None)
    release = B.DEVICE_FREE_FN(lambda ptr, nbytes, user: None)
    with pytest.raises(B.AgnesError) as e:
        ag.agnes_set_device_allocator(alloc, None)
    assert e.value.status == B.AGNES_ERR_INVALID and "both" in str(e.value)
    with pytest.raises(B.AgnesError):
        ag.agnes_set_device_allocator(None, release)
    ag.agnes_set_device_allocator(alloc, release)       # installed ...
    ag.agnes_set_device_allocator(None, None)           # ... and hipMalloc / hipFree restored
