"""MI355X (gfx950) hyperbatch GNN data preparation (AGNES, arXiv 2601.01473).

The work runs in libagnes.so (HIP kernels behind the C ABI of include/agnes.h).
This package marshals arguments: numpy arrays in, targets as a host numpy
array (uploaded by the library) or a torch CUDA tensor (already on the device),
torch streams, and copies of the outputs back to numpy.

    store = Store(offsets, indices, features, block_bytes=65536)
    batch = store.prepare(targets_int32_HxB, fanouts=[25, 10], seed=0)
    out = batch.to_host()          # per-minibatch nodes, per-hop CSR, features
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime the library binds to)

from . import _binding as B
from ._binding import AgnesError, agnes_batch_stats, agnes_batch_view_get, agnes_build_blocks  # noqa: F401
from ._binding import agnes_batch_finish, agnes_batch_wait, agnes_hyperbatch_begin  # noqa: F401
from ._binding import agnes_free, agnes_hyperbatch_prepare, agnes_last_error  # noqa: F401
from ._binding import agnes_hyperbatch_begin_device, agnes_hyperbatch_prepare_device  # noqa: F401
from ._binding import agnes_store_info, agnes_store_object_table, agnes_store_set_option  # noqa: F401
from ._binding import agnes_batch_tier_stats, agnes_build_blocks_staged, agnes_sage_forward  # noqa: F401
from ._binding import agnes_build_blocks_cached, agnes_philox4x64_10, agnes_set_device_allocator  # noqa: F401

_FEAT_DTYPES = {np.dtype(np.float32): B.AGNES_FLOAT32, np.dtype(np.float16): B.AGNES_FLOAT16}

_hip = None

# Every callback pair ever installed: a block keeps the release callback of the
# allocator it came from, so the ctypes objects must outlive every block.
_installed_callbacks = []


def use_torch_allocator(on: bool = True) -> None:
    """Let torch's caching allocator own the library's device memory (stores,
    batches, scratch space), or go back to hipMalloc / hipFree.  Blocks are
    allocated on the current device and stream; the stream is synchronised
    before a block is used, since the allocator may hand out memory whose last
    user's work is still pending on it.  Affects allocations made afterwards."""
    if not on:
        agnes_set_device_allocator(None, None)
        return

    def alloc(nbytes, user):
        try:
            dev = torch.cuda.current_device()
            stream = torch.cuda.current_stream(dev)
            ptr = torch.cuda.caching_allocator_alloc(int(nbytes), dev, stream)
            stream.synchronize()
            return ptr
        except Exception:          # the library reports AGNES_ERR_NOMEM
            return None

    def release(ptr, nbytes, user):
        torch.cuda.caching_allocator_delete(ptr)

    cbs = (B.DEVICE_ALLOC_FN(alloc), B.DEVICE_FREE_FN(release))
    _installed_callbacks.append(cbs)
    agnes_set_device_allocator(*cbs)


def _hiprt():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so.7")
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    return _hip


def device_to_host(ptr: int, count: int, dtype) -> np.ndarray:
    """Copy `count` elements of `dtype` from device memory to a new numpy array."""
    out = np.empty(count, dtype=dtype)
    if count:
        rc = _hiprt().hipMemcpy(out.ctypes.data, ctypes.c_void_p(ptr), out.nbytes, 2)
        if rc != 0:
            raise RuntimeError("hipMemcpy device->host failed with %d" % rc)
    return out


def _stream_handle(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else 0
    return int(getattr(stream, "cuda_stream", stream))


class Store:
    """HBM-resident topology and feature blocks (agnes_build_blocks), or with
    pool_blocks set, HBM-resident topology and a staged feature tier: features
    in pinned host memory, a pool of pool_blocks feature blocks in HBM
    (agnes_build_blocks_staged), and with cache_rows set also a feature cache
    of that many rows, admitting rows at cache_threshold accesses
    (agnes_build_blocks_cached)."""

    def __init__(self, offsets, indices, features, block_bytes: int, feat_dtype: str | None = None,
                 stream=None, pool_blocks: int | None = None, cache_rows: int | None = None,
                 cache_threshold: int = 2):
        off = np.ascontiguousarray(offsets)
        if off.dtype not in (np.int32, np.int64):
            raise TypeError("offsets must be int32 or int64")
        idx = np.ascontiguousarray(indices, dtype=np.int32)
        feat = np.ascontiguousarray(features)
        if feat.ndim != 2:
            raise ValueError("features must be 2-D [num_nodes, dim]")
        if feat_dtype == "bfloat16" or (feat_dtype is None and feat.dtype == np.uint16):
            fdt = B.AGNES_BFLOAT16
        elif feat.dtype in _FEAT_DTYPES:
            fdt = _FEAT_DTYPES[feat.dtype]
        else:
            raise TypeError("features must be float32, float16 or bfloat16 (as uint16)")
        csr = B.agnes_csr(len(off) - 1, len(idx), B.AGNES_INT64 if off.dtype == np.int64 else B.AGNES_INT32,
                          off.ctypes.data, idx.ctypes.data if len(idx) else None)
        fs = B.agnes_features(feat.ctypes.data, feat.shape[1], fdt)
        if pool_blocks is None:
            if cache_rows is not None:
                raise ValueError("a feature cache needs the staged tier (pool_blocks)")
            self.handle = agnes_build_blocks(csr, fs, block_bytes, _stream_handle(stream))
        elif cache_rows is None:
            self.handle = agnes_build_blocks_staged(csr, fs, block_bytes, int(pool_blocks), _stream_handle(stream))
        else:
            self.handle = agnes_build_blocks_cached(csr, fs, block_bytes, int(pool_blocks), int(cache_rows),
                                                    int(cache_threshold), _stream_handle(stream))
        self.pool_blocks = pool_blocks
        self.num_nodes = len(off) - 1
        self.row_bytes = feat.shape[1] * feat.itemsize
        self.block_bytes = block_bytes

    def info(self) -> dict:
        v = agnes_store_info(self.handle)
        keys = ["num_nodes", "num_edges", "topo_blocks", "edges_per_block", "feat_blocks",
                "rows_per_block", "row_bytes", "device_bytes"]
        return dict(zip(keys, v))

    def object_table(self):
        nblk = self.info()["topo_blocks"]
        first = np.empty(nblk, np.int32)
        last = np.empty(nblk, np.int32)
        agnes_store_object_table(self.handle, first.ctypes.data, last.ctypes.data)
        return first, last

    def set_profiling(self, on: bool) -> None:
        agnes_store_set_option(self.handle, B.AGNES_OPT_PROFILE, 1 if on else 0)

    def set_sampling_graph(self, mode) -> None:
        """True: replay the sampling kernels of a repeated hyperbatch shape
        from a captured HIP graph; False: launch them one by one; "auto" (the
        default): replay for shapes of at most 2^20 sampled edges."""
        v = 2 if mode == "auto" else (1 if mode else 0)
        agnes_store_set_option(self.handle, B.AGNES_OPT_SAMPLING_GRAPH, v)

    def set_join_path(self, buckets: bool = True, bucket_cap: int | None = None) -> None:
        """buckets=True: node-range buckets joined in workgroup memory;
        False: the device-wide radix sort and merge-path join (the store's
        default).  bucket_cap: entries of one sorted bucket before the
        hyperbatch is sampled again with the radix sort (never changes
        results)."""
        agnes_store_set_option(self.handle, B.AGNES_OPT_JOIN_PATH, 1 if buckets else 0)
        if bucket_cap is not None:
            agnes_store_set_option(self.handle, B.AGNES_OPT_BUCKET_CAP, int(bucket_cap))

    def set_sampling_groups(self, groups: int) -> None:
        """Most workgroups of each sampling-phase kernel that loops over its
        work, in [256, 4096], or 0 (the default) to choose per hop by its
        size (never changes results)."""
        agnes_store_set_option(self.handle, B.AGNES_OPT_SAMPLING_GROUPS, int(groups))

    def set_gather_shape(self, groups: int | None = None, unroll: int | None = None,
                         nontemporal: bool | None = None, chunks: int | None = None) -> None:
        """Launch shape and store kind of the row-copy kernel (never change results)."""
        if chunks is not None:
            agnes_store_set_option(self.handle, B.AGNES_OPT_GATHER_CHUNKS, int(chunks))
        if groups is not None:
            agnes_store_set_option(self.handle, B.AGNES_OPT_GATHER_GROUPS, int(groups))
        if unroll is not None:
            agnes_store_set_option(self.handle, B.AGNES_OPT_GATHER_UNROLL, int(unroll))
        if nontemporal is not None:
            agnes_store_set_option(self.handle, B.AGNES_OPT_GATHER_NONTEMPORAL, 1 if nontemporal else 0)

    def prepare(self, targets, fanouts, seed: int = 0, mb_base: int = 0,
                batch: "Batch | None" = None, stream=None) -> "Batch":
        """One hyperbatch, synchronously.  targets: int32 [H, B], a host numpy
        array (uploaded by the call) or a CUDA tensor (read in place)."""
        return self._start(agnes_hyperbatch_prepare, agnes_hyperbatch_prepare_device, targets, fanouts, seed,
                           mb_base, batch, stream)

    def begin(self, targets, fanouts, seed: int = 0, mb_base: int = 0,
              batch: "Batch | None" = None, stream=None) -> "Batch":
        """Enqueue the sampling hops of one hyperbatch and return (see Batch.finish)."""
        return self._start(agnes_hyperbatch_begin, agnes_hyperbatch_begin_device, targets, fanouts, seed,
                           mb_base, batch, stream)

    def _start(self, fn_host, fn_dev, targets, fanouts, seed, mb_base, batch, stream):
        if isinstance(targets, torch.Tensor):
            if not (targets.is_cuda and targets.dtype == torch.int32):
                raise TypeError("a targets tensor must be a CUDA int32 tensor [H, B]")
            t = targets.contiguous()
            fn, ptr = fn_dev, t.data_ptr()
        elif isinstance(targets, np.ndarray):
            if targets.dtype != np.int32:
                raise TypeError("a targets array must be int32 [H, B]")
            t = np.ascontiguousarray(targets)
            fn, ptr = fn_host, t.ctypes.data
        else:
            raise TypeError("targets must be an int32 numpy array or CUDA tensor [H, B]")
        if t.ndim != 2:
            raise ValueError("targets must be [H, B]")
        H, Bsz = t.shape
        fan = (ctypes.c_int32 * len(fanouts))(*[int(f) for f in fanouts])
        prev = batch.handle if batch is not None else None
        if batch is not None:
            batch.handle = None          # ownership passes to the call (released on error)
        h = fn(self.handle, ptr, H, Bsz, fan, len(fanouts), seed, mb_base, _stream_handle(stream), prev)
        if batch is None:
            batch = Batch(self)
        batch.handle = h
        batch._targets = t               # a device tensor is read until the hyperbatch is finished
        return batch

    def close(self) -> None:
        if getattr(self, "handle", None):
            agnes_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:       # interpreter shutdown: the process releases everything
            pass


class Batch:
    """Device outputs of one hyperbatch (agnes_batch)."""

    def __init__(self, store: Store):
        self.store = store
        self.handle = None

    def finish(self, stream=None) -> "Batch":
        """Wait for the output sizes and enqueue the gather (returns without waiting)."""
        agnes_batch_finish(self.handle, _stream_handle(stream))
        return self

    def wait(self) -> "Batch":
        agnes_batch_wait(self.handle)
        return self

    def stats(self) -> dict:
        s = agnes_batch_stats(self.handle)
        L = s.L
        return dict(requests=list(s.requests[:L]), sampled=list(s.sampled[:L]),
                    new_nodes=list(s.new_nodes[:L]), topo_blocks=list(s.topo_blocks[:L]),
                    rows=s.rows, distinct_rows=s.distinct_rows, feat_blocks=s.feat_blocks,
                    sample_ms=s.sample_ms, gather_ms=s.gather_ms, copy_ms=s.copy_ms)

    def sage_forward(self, weights, biases, out: torch.Tensor | None = None, stream=None,
                     noalloc: bool = False) -> torch.Tensor:
        """GraphSAGE forward over this batch (agnes_sage_forward, or with
        noalloc agnes_sage_forward_noalloc).  weights[i]: CUDA bf16 (or
        int16/uint16 bits) [dims[i+1], 2 dims[i]]; biases[i]: CUDA float32
        [dims[i+1]]; returns float32 [H*B, dims[L]] (enqueued on `stream`)."""
        L = len(weights)
        if L != len(biases) or L < 1 or L > B.AGNES_MAX_LAYERS:
            raise ValueError("one weight and one bias per layer")
        m = B.agnes_sage_model()
        m.L = L
        for i, (w, b) in enumerate(zip(weights, biases)):
            if not (w.is_cuda and w.dim() == 2 and w.element_size() == 2 and w.is_contiguous()):
                raise TypeError("weights must be contiguous 2-D CUDA bf16 tensors")
            if not (b.is_cuda and b.dtype == torch.float32 and b.is_contiguous()):
                raise TypeError("biases must be contiguous CUDA float32 tensors")
            if b.numel() != w.shape[0] or w.shape[1] % 2:
                raise ValueError("weight %d is [dims[i+1], 2 dims[i]] and bias %d [dims[i+1]]" % (i, i))
            if i > 0 and w.shape[1] // 2 != weights[i - 1].shape[0]:
                raise ValueError("layer %d's input dim is layer %d's output dim" % (i, i - 1))
            m.dims[i] = w.shape[1] // 2
            m.weight[i] = w.data_ptr()
            m.bias[i] = b.data_ptr()
        m.dims[L] = weights[-1].shape[0]
        v = self.view()
        rows = v.H * int(np.ctypeslib.as_array(v.layer_sizes, shape=(v.H * (v.L + 1),))[0])
        if out is None:
            out = torch.empty((rows, m.dims[L]), dtype=torch.float32, device="cuda")
        if not (out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and
                tuple(out.shape) == (rows, m.dims[L])):
            raise ValueError("out must be a contiguous CUDA float32 tensor [H*B, dims[L]]")
        fn = B.agnes_sage_forward_noalloc if noalloc else agnes_sage_forward
        fn(self.handle, m, out.data_ptr(), _stream_handle(stream))
        self._sage_keep = (weights, biases, out)
        return out

    def tier_stats(self) -> dict:
        """Staged-tier counters (all zero for HBM-resident features)."""
        t = agnes_batch_tier_stats(self.handle)
        return dict(needed_blocks=t.needed_blocks, staged_blocks=t.staged_blocks, hit_blocks=t.hit_blocks,
                    rounds=t.rounds, staged_bytes=t.staged_bytes, cache_hit_rows=t.cache_hit_rows,
                    admitted_rows=t.admitted_rows, cached_rows=t.cached_rows, gather_ms=t.gather_ms)

    def view(self) -> B.agnes_batch_view:
        return agnes_batch_view_get(self.handle)

    def to_host(self, minibatches=None, features: bool = True) -> list:
        """Per-minibatch host copies: dict(nodes, layer_sizes, row_ptr[l], col[l], features)."""
        self.wait()
        v = self.view()
        H, L = v.H, v.L
        node_off = np.ctypeslib.as_array(v.node_off, shape=(H + 1,)).copy()
        lsz = np.ctypeslib.as_array(v.layer_sizes, shape=(H * (L + 1),)).reshape(H, L + 1).copy()
        rows = int(node_off[H])
        nodes = device_to_host(v.nodes, rows, np.int32)
        rp, col, rpo, colo = [], [], [], []
        for l in range(L):
            ro = np.ctypeslib.as_array(v.rp_off[l], shape=(H + 1,)).copy()
            co = np.ctypeslib.as_array(v.col_off[l], shape=(H + 1,)).copy()
            rpo.append(ro)
            colo.append(co)
            rp.append(device_to_host(v.row_ptr[l], int(ro[H]), np.int32))
            col.append(device_to_host(v.col[l], int(co[H]), np.int32))
        rb = v.row_bytes
        out = []
        mbs = range(H) if minibatches is None else minibatches
        for j in mbs:
            a, b = int(node_off[j]), int(node_off[j + 1])
            d = dict(nodes=nodes[a:b], layer_sizes=lsz[j],
                     row_ptr=[rp[l][rpo[l][j]:rpo[l][j + 1]] for l in range(L)],
                     col=[col[l][colo[l][j]:colo[l][j + 1]] for l in range(L)])
            if features:
                d["features"] = device_to_host(v.features + a * rb, (b - a) * rb, np.uint8).reshape(b - a, rb)
            out.append(d)
        return out

    def close(self) -> None:
        if getattr(self, "handle", None):
            agnes_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:       # interpreter shutdown: the process releases everything
            pass
