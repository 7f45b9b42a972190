"""ctypes binding of libagnes.so (the C ABI declared in include/agnes.h).

Argument marshalling only: every step of data preparation runs in the HIP
library.  If libagnes.so is missing the import of the binding fails; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libagnes.san.so" if os.environ.get("AGNES_SANITIZE") else "libagnes.so")

AGNES_OK, AGNES_ERR_INVALID, AGNES_ERR_NOMEM, AGNES_ERR_DEVICE, AGNES_ERR_RANGE, AGNES_ERR_INTERNAL = range(6)
STATUS_NAMES = {0: "OK", 1: "INVALID", 2: "NOMEM", 3: "DEVICE", 4: "RANGE", 5: "INTERNAL"}
AGNES_INT32, AGNES_INT64, AGNES_FLOAT32, AGNES_FLOAT16, AGNES_BFLOAT16 = range(5)
AGNES_MAX_LAYERS = 8
AGNES_OPT_PROFILE = 1
AGNES_OPT_GATHER_GROUPS = 2
AGNES_OPT_GATHER_UNROLL = 3
AGNES_OPT_GATHER_NONTEMPORAL = 4
AGNES_OPT_GATHER_CHUNKS = 5
AGNES_OPT_SAMPLING_GRAPH = 6
AGNES_OPT_JOIN_PATH = 7
AGNES_OPT_BUCKET_CAP = 8
AGNES_OPT_SAMPLING_GROUPS = 9

EXPORTED = ["agnes_build_blocks", "agnes_build_blocks_staged", "agnes_build_blocks_cached", "agnes_hyperbatch_prepare",
            "agnes_hyperbatch_prepare_device", "agnes_hyperbatch_begin", "agnes_hyperbatch_begin_device", "agnes_batch_finish", "agnes_batch_wait", "agnes_batch_view_get",
            "agnes_batch_stats", "agnes_batch_tier_stats", "agnes_store_set_option", "agnes_store_info",
            "agnes_store_object_table", "agnes_sage_forward", "agnes_sage_forward_noalloc", "agnes_philox4x64_10", "agnes_set_device_allocator", "agnes_free",
            "agnes_last_error"]

# void* alloc(uint64_t bytes, void* user); void release(void* ptr, uint64_t bytes, void* user)
DEVICE_ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p)
DEVICE_FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p)


class agnes_csr(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("num_edges", ctypes.c_int64),
                ("offsets_dtype", ctypes.c_int), ("offsets", ctypes.c_void_p),
                ("indices", ctypes.c_void_p)]


class agnes_features(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dim", ctypes.c_int64), ("dtype", ctypes.c_int)]


class agnes_batch_view(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("L", ctypes.c_int32), ("row_bytes", ctypes.c_int64),
                ("node_off", ctypes.POINTER(ctypes.c_int64)),
                ("layer_sizes", ctypes.POINTER(ctypes.c_int32)),
                ("nodes", ctypes.c_void_p),
                ("rp_off", ctypes.POINTER(ctypes.c_int64) * AGNES_MAX_LAYERS),
                ("row_ptr", ctypes.c_void_p * AGNES_MAX_LAYERS),
                ("col_off", ctypes.POINTER(ctypes.c_int64) * AGNES_MAX_LAYERS),
                ("col", ctypes.c_void_p * AGNES_MAX_LAYERS),
                ("features", ctypes.c_void_p)]


class agnes_stats(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32),
                ("requests", ctypes.c_int64 * AGNES_MAX_LAYERS),
                ("sampled", ctypes.c_int64 * AGNES_MAX_LAYERS),
                ("new_nodes", ctypes.c_int64 * AGNES_MAX_LAYERS),
                ("topo_blocks", ctypes.c_int64 * AGNES_MAX_LAYERS),
                ("rows", ctypes.c_int64), ("distinct_rows", ctypes.c_int64),
                ("feat_blocks", ctypes.c_int64),
                ("sample_ms", ctypes.c_float), ("gather_ms", ctypes.c_float),
                ("copy_ms", ctypes.c_float)]


class agnes_tier_stats(ctypes.Structure):
    _fields_ = [("needed_blocks", ctypes.c_int64), ("staged_blocks", ctypes.c_int64),
                ("hit_blocks", ctypes.c_int64), ("rounds", ctypes.c_int64),
                ("staged_bytes", ctypes.c_int64), ("cache_hit_rows", ctypes.c_int64),
                ("admitted_rows", ctypes.c_int64), ("cached_rows", ctypes.c_int64), ("gather_ms", ctypes.c_float)]


class agnes_sage_model(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("dims", ctypes.c_int32 * (AGNES_MAX_LAYERS + 1)),
                ("weight", ctypes.c_void_p * AGNES_MAX_LAYERS), ("bias", ctypes.c_void_p * AGNES_MAX_LAYERS)]


class AgnesError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), msg))
        self.status = status


_lib = None


def lib():
    """The loaded libagnes.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libagnes.so is not built (run __graft_entry__.build() or "
                          "python paper_2601_01473_amd/build.py); there is no CPU fallback")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    st = ctypes.c_int
    L.agnes_build_blocks.restype = st
    L.agnes_build_blocks.argtypes = [ctypes.POINTER(agnes_csr), ctypes.POINTER(agnes_features), u64, vp,
                                     ctypes.POINTER(vp)]
    L.agnes_build_blocks_staged.restype = st
    L.agnes_build_blocks_staged.argtypes = [ctypes.POINTER(agnes_csr), ctypes.POINTER(agnes_features), u64, i64,
                                            vp, ctypes.POINTER(vp)]
    L.agnes_build_blocks_cached.restype = st
    L.agnes_build_blocks_cached.argtypes = [ctypes.POINTER(agnes_csr), ctypes.POINTER(agnes_features), u64, i64,
                                            i64, i64, vp, ctypes.POINTER(vp)]
    L.agnes_batch_tier_stats.restype = st
    L.agnes_batch_tier_stats.argtypes = [vp, ctypes.POINTER(agnes_tier_stats)]
    L.agnes_sage_forward.restype = st
    L.agnes_sage_forward.argtypes = [vp, ctypes.POINTER(agnes_sage_model), vp, vp]
    L.agnes_sage_forward_noalloc.restype = st
    L.agnes_sage_forward_noalloc.argtypes = [vp, ctypes.POINTER(agnes_sage_model), vp, vp]
    L.agnes_hyperbatch_prepare.restype = st
    L.agnes_hyperbatch_prepare.argtypes = [vp, vp, i32, i32, vp, i32, u64, i64, vp, ctypes.POINTER(vp)]
    L.agnes_hyperbatch_begin.restype = st
    L.agnes_hyperbatch_begin.argtypes = [vp, vp, i32, i32, vp, i32, u64, i64, vp, ctypes.POINTER(vp)]
    for name in ("agnes_hyperbatch_prepare_device", "agnes_hyperbatch_begin_device"):
        getattr(L, name).restype = st
        getattr(L, name).argtypes = [vp, vp, i32, i32, vp, i32, u64, i64, vp, ctypes.POINTER(vp)]
    L.agnes_batch_finish.restype = st
    L.agnes_batch_finish.argtypes = [vp, vp]
    L.agnes_batch_wait.restype = st
    L.agnes_batch_wait.argtypes = [vp]
    L.agnes_batch_view_get.restype = st
    L.agnes_batch_view_get.argtypes = [vp, ctypes.POINTER(agnes_batch_view)]
    L.agnes_batch_stats.restype = st
    L.agnes_batch_stats.argtypes = [vp, ctypes.POINTER(agnes_stats)]
    L.agnes_store_set_option.restype = st
    L.agnes_store_set_option.argtypes = [vp, ctypes.c_int, i64]
    L.agnes_store_info.restype = st
    L.agnes_store_info.argtypes = [vp, ctypes.POINTER(i64)]
    L.agnes_store_object_table.restype = st
    L.agnes_store_object_table.argtypes = [vp, vp, vp]
    L.agnes_philox4x64_10.restype = st
    L.agnes_philox4x64_10.argtypes = [vp, vp, i64, vp]
    L.agnes_set_device_allocator.restype = st
    L.agnes_set_device_allocator.argtypes = [DEVICE_ALLOC_FN, DEVICE_FREE_FN, vp]
    L.agnes_free.restype = None
    L.agnes_free.argtypes = [vp]
    L.agnes_last_error.restype = ctypes.c_char_p
    L.agnes_last_error.argtypes = []
    _lib = L
    return L


def check(status: int) -> None:
    if status != AGNES_OK:
        raise AgnesError(status, lib().agnes_last_error().decode(errors="replace"))


# Thin wrappers with the C names ------------------------------------------------

def agnes_build_blocks(csr: agnes_csr, feat: agnes_features, block_bytes: int, stream: int = 0) -> int:
    out = ctypes.c_void_p()
    check(lib().agnes_build_blocks(ctypes.byref(csr), ctypes.byref(feat), block_bytes,
                                   ctypes.c_void_p(stream), ctypes.byref(out)))
    return out.value


def agnes_build_blocks_staged(csr: agnes_csr, feat: agnes_features, block_bytes: int, pool_blocks: int,
                              stream: int = 0) -> int:
    out = ctypes.c_void_p()
    check(lib().agnes_build_blocks_staged(ctypes.byref(csr), ctypes.byref(feat), block_bytes, pool_blocks,
                                          ctypes.c_void_p(stream), ctypes.byref(out)))
    return out.value


def agnes_build_blocks_cached(csr: agnes_csr, feat: agnes_features, block_bytes: int, pool_blocks: int,
                              cache_rows: int, threshold: int, stream: int = 0) -> int:
    out = ctypes.c_void_p()
    check(lib().agnes_build_blocks_cached(ctypes.byref(csr), ctypes.byref(feat), block_bytes, pool_blocks,
                                          cache_rows, threshold, ctypes.c_void_p(stream), ctypes.byref(out)))
    return out.value


def agnes_batch_tier_stats(batch: int) -> agnes_tier_stats:
    s = agnes_tier_stats()
    check(lib().agnes_batch_tier_stats(ctypes.c_void_p(batch), ctypes.byref(s)))
    return s


def agnes_sage_forward(batch: int, model: agnes_sage_model, out_ptr: int, stream: int = 0) -> None:
    check(lib().agnes_sage_forward(ctypes.c_void_p(batch), ctypes.byref(model), ctypes.c_void_p(out_ptr),
                                   ctypes.c_void_p(stream)))


def _start_call(fn, store, targets_ptr, H, B, fanouts_arr, L, seed, mb_base, stream, batch):
    out = ctypes.c_void_p(batch)
    check(fn(ctypes.c_void_p(store), ctypes.c_void_p(targets_ptr), H, B, fanouts_arr, L, seed, mb_base,
             ctypes.c_void_p(stream), ctypes.byref(out)))
    return out.value


def agnes_sage_forward_noalloc(batch: int, model: agnes_sage_model, out_ptr: int, stream: int = 0) -> None:
    check(lib().agnes_sage_forward_noalloc(ctypes.c_void_p(batch), ctypes.byref(model), ctypes.c_void_p(out_ptr),
                                           ctypes.c_void_p(stream)))


def agnes_hyperbatch_prepare(store: int, targets_ptr: int, H: int, B: int, fanouts_arr, L: int,
                             seed: int, mb_base: int, stream: int = 0, batch: int | None = None) -> int:
    """targets_ptr: host int32 [H*B]."""
    return _start_call(lib().agnes_hyperbatch_prepare, store, targets_ptr, H, B, fanouts_arr, L, seed, mb_base,
                       stream, batch)


def agnes_hyperbatch_prepare_device(store: int, targets_ptr: int, H: int, B: int, fanouts_arr, L: int,
                                    seed: int, mb_base: int, stream: int = 0, batch: int | None = None) -> int:
    """targets_ptr: device int32 [H*B]."""
    return _start_call(lib().agnes_hyperbatch_prepare_device, store, targets_ptr, H, B, fanouts_arr, L, seed,
                       mb_base, stream, batch)


def agnes_hyperbatch_begin(store: int, targets_ptr: int, H: int, B: int, fanouts_arr, L: int,
                           seed: int, mb_base: int, stream: int = 0, batch: int | None = None) -> int:
    """targets_ptr: host int32 [H*B]."""
    return _start_call(lib().agnes_hyperbatch_begin, store, targets_ptr, H, B, fanouts_arr, L, seed, mb_base,
                       stream, batch)


def agnes_hyperbatch_begin_device(store: int, targets_ptr: int, H: int, B: int, fanouts_arr, L: int,
                                  seed: int, mb_base: int, stream: int = 0, batch: int | None = None) -> int:
    """targets_ptr: device int32 [H*B]."""
    return _start_call(lib().agnes_hyperbatch_begin_device, store, targets_ptr, H, B, fanouts_arr, L, seed,
                       mb_base, stream, batch)


def agnes_philox4x64_10(counters, keys):
    """Device Philox4x64-10 words: counters uint64 [n, 4], keys uint64 [n, 2] -> uint64 [n, 4]."""
    import numpy as np
    c = np.ascontiguousarray(counters, dtype=np.uint64).reshape(-1, 4)
    k = np.ascontiguousarray(keys, dtype=np.uint64).reshape(-1, 2)
    if len(c) != len(k):
        raise ValueError("one key pair per counter")
    out = np.empty_like(c)
    check(lib().agnes_philox4x64_10(c.ctypes.data, k.ctypes.data, len(c), out.ctypes.data))
    return out


def agnes_set_device_allocator(alloc, release, user: int | None = None) -> None:
    """alloc / release: DEVICE_ALLOC_FN / DEVICE_FREE_FN callbacks, or both None
    (hipMalloc / hipFree).  The caller keeps the callback objects alive."""
    a = alloc if alloc is not None else DEVICE_ALLOC_FN()
    r = release if release is not None else DEVICE_FREE_FN()
    check(lib().agnes_set_device_allocator(a, r, ctypes.c_void_p(user)))


def agnes_batch_finish(batch: int, stream: int = 0) -> None:
    check(lib().agnes_batch_finish(ctypes.c_void_p(batch), ctypes.c_void_p(stream)))


def agnes_batch_wait(batch: int) -> None:
    check(lib().agnes_batch_wait(ctypes.c_void_p(batch)))


def agnes_batch_view_get(batch: int) -> agnes_batch_view:
    v = agnes_batch_view()
    check(lib().agnes_batch_view_get(ctypes.c_void_p(batch), ctypes.byref(v)))
    return v


def agnes_batch_stats(batch: int) -> agnes_stats:
    s = agnes_stats()
    check(lib().agnes_batch_stats(ctypes.c_void_p(batch), ctypes.byref(s)))
    return s


def agnes_store_set_option(store: int, opt: int, value: int) -> None:
    check(lib().agnes_store_set_option(ctypes.c_void_p(store), opt, value))


def agnes_store_info(store: int) -> list:
    arr = (ctypes.c_int64 * 8)()
    check(lib().agnes_store_info(ctypes.c_void_p(store), arr))
    return list(arr)


def agnes_store_object_table(store: int, first_ptr: int, last_ptr: int) -> None:
    check(lib().agnes_store_object_table(ctypes.c_void_p(store), ctypes.c_void_p(first_ptr),
                                         ctypes.c_void_p(last_ptr)))


def agnes_free(handle: int | None) -> None:
    if handle:
        lib().agnes_free(ctypes.c_void_p(handle))


def agnes_last_error() -> str:
    return lib().agnes_last_error().decode(errors="replace")
