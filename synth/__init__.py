"""Seeded synthetic workloads shared by the tests, the smoke check and the benchmark.

Graphs are R-MAT (Chakrabarti, Zhan, Faloutsos, SDM 2004) with unpermuted node
ids, stored as CSR with source rows; features are N(0,1); targets are distinct
node ids drawn by a partial Fisher-Yates shuffle.  The generator code lives in
``synth.c`` (SplitMix64 words, OpenMP); this module only builds and wraps it.

Nothing here implements any step of the data-preparation method: these are the
inputs both the GPU library and the CPU oracle consume.

The five workloads stand in for the paper's web-scale graphs (Table 2: IG, TW,
PA, FR, YH), which are not available: power-law R-MAT graphs of 2^14 to 2^26
nodes, average degree 16 to 30, fp32/fp16/bf16 features of 64 to 1024 dims.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from functools import lru_cache

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
# AGNES_SANITIZE (e.g. "address,undefined"): a separate build with LLVM's
# sanitizers, loaded only under their preloaded runtime
_SAN = os.environ.get("AGNES_SANITIZE", "")
_LIB = os.path.join(_HERE, "libsynth.san.so" if _SAN else "libsynth.so")

FEATURE_DTYPES = {"float32": (0, 4), "float16": (1, 2), "bfloat16": (2, 2)}


def build(force: bool = True) -> str:
    """Compile libsynth.so with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        if _SAN:
            clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
            cc = [clang, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=" + _SAN, "-fno-sanitize-recover=all"]
        else:
            cc = ["gcc", "-O3"]
        subprocess.check_call([*cc, "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i64, u64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
        L.synth_rmat_csr.restype = i64
        L.synth_rmat_csr.argtypes = [ctypes.c_int, i64, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, u64, vp, vp]
        L.synth_features.restype = None
        L.synth_features.argtypes = [i64, i64, ctypes.c_int, u64, vp]
        L.synth_targets.restype = ctypes.c_int
        L.synth_targets.argtypes = [i64, i64, u64, vp]
        L.synth_convert_f32.restype = None
        L.synth_convert_f32.argtypes = [vp, i64, ctypes.c_int, vp]
        L.synth_word.restype = u64
        L.synth_word.argtypes = [u64, u64, u64]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def rmat_csr(scale: int, edge_factor: int, abc=(0.57, 0.19, 0.19), seed: int = 0):
    """R-MAT graph with 2^scale nodes from 2^scale * edge_factor generated edges.

    Returns (offsets int64[N+1], indices int32[E]) after dropping duplicate
    edges and self-loops; rows are sorted by destination id.
    """
    n = 1 << scale
    m = n * edge_factor
    offsets = np.empty(n + 1, dtype=np.int64)
    indices = np.empty(max(m, 1), dtype=np.int32)
    e = lib().synth_rmat_csr(scale, m, abc[0], abc[1], abc[2], seed, _ptr(offsets), _ptr(indices))
    if e < 0:
        raise MemoryError("synth_rmat_csr: allocation failed")
    return offsets, indices[:e]


def features(n: int, dim: int, dtype: str = "float32", seed: int = 0) -> np.ndarray:
    """n x dim matrix ~ N(0,1), as float32 / float16 / bfloat16 (returned as uint16)."""
    code, size = FEATURE_DTYPES[dtype]
    npdt = {"float32": np.float32, "float16": np.float16, "bfloat16": np.uint16}[dtype]
    out = np.empty((n, dim), dtype=npdt)
    lib().synth_features(n, dim, code, seed, _ptr(out))
    return out


def targets(n: int, count: int, seed: int = 0) -> np.ndarray:
    """`count` distinct node ids in [0, n)."""
    out = np.empty(count, dtype=np.int32)
    if lib().synth_targets(n, count, seed, _ptr(out)) != 0:
        raise ValueError("targets: count > n or allocation failure")
    return out


def convert_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round-to-nearest-even conversion used for the fp16/bf16 features."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    code, _ = FEATURE_DTYPES[dtype]
    out = np.empty(x.shape, dtype=np.float32 if code == 0 else np.uint16)
    lib().synth_convert_f32(_ptr(x), x.size, code, _ptr(out))
    return out


@dataclass(frozen=True)
class Config:
    """One synthetic workload: graph, features, hyperbatch shape and sampler settings."""
    name: str
    scale: int
    edge_factor: int
    abc: tuple
    offsets_dtype: str          # "int32" | "int64"
    feat_dtype: str             # "float32" | "float16" | "bfloat16"
    dim: int
    fanouts: tuple
    H: int
    B: int
    block_bytes: int
    seed: int = 0               # sampling seed
    data_seed: int = 0          # graph / feature / target generator seed
    h_sweep: tuple = field(default=())

    @property
    def num_nodes(self) -> int:
        return 1 << self.scale

    @property
    def row_bytes(self) -> int:
        return self.dim * FEATURE_DTYPES[self.feat_dtype][1]

    def describe(self) -> str:
        return (f"rmat-2^{self.scale}-deg{self.edge_factor}-{self.feat_dtype}x{self.dim}"
                f"-fanout{list(self.fanouts)}-{self.H}x{self.B}-blk{self.block_bytes}")


CONFIGS = {
    # 2^14 nodes, avg degree 16, int32 CSR, fp32 dim 64, fanout [10,5], 8 x 256, 4 KiB blocks
    "c1": Config("c1", 14, 16, (0.57, 0.19, 0.19), "int32", "float32", 64, (10, 5), 8, 256, 4096),
    # 2^20 nodes, avg degree 20, int64 offsets, fp32 dim 128, fanout [15,10], 32 x 1024, 4 KiB
    "c2": Config("c2", 20, 20, (0.57, 0.19, 0.19), "int64", "float32", 128, (15, 10), 32, 1024, 4096),
    # 2^23 nodes, avg degree 30, fp32 dim 256, fanout [25,10], 64 x 1024, 64 KiB
    "c3": Config("c3", 23, 30, (0.57, 0.19, 0.19), "int64", "float32", 256, (25, 10), 64, 1024, 65536),
    # 2^26 nodes, avg degree 16, fp16 dim 128, fanout [15,10,5], 128 x 1024, 64 KiB
    "c4": Config("c4", 26, 16, (0.57, 0.19, 0.19), "int64", "float16", 128, (15, 10, 5), 128, 1024, 65536),
    # skew stress: (0.65,0.15,0.15), 2^23 nodes, avg degree 30, bf16 dim 1024, fanout [25,10],
    # hyperbatch swept over 1, 8, 64, 256 minibatches of 1024, 4 KiB
    "c5": Config("c5", 23, 30, (0.65, 0.15, 0.15), "int64", "bfloat16", 1024, (25, 10), 64, 1024, 4096,
                 h_sweep=(1, 8, 64, 256)),
}


@lru_cache(maxsize=2)
def graph(scale: int, edge_factor: int, abc: tuple, data_seed: int):
    return rmat_csr(scale, edge_factor, abc, data_seed)


@lru_cache(maxsize=2)
def feature_matrix(n: int, dim: int, dtype: str, data_seed: int):
    return features(n, dim, dtype, data_seed + 1)


def workload(cfg: Config, H: int | None = None, with_features: bool = True):
    """Materialise a config: dict with offsets (in the config's offset dtype),
    indices, features (or None), targets [H, B] and the sampler settings."""
    H = cfg.H if H is None else H
    off64, idx = graph(cfg.scale, cfg.edge_factor, tuple(cfg.abc), cfg.data_seed)
    offsets = off64.astype(np.int32) if cfg.offsets_dtype == "int32" else off64
    feat = feature_matrix(cfg.num_nodes, cfg.dim, cfg.feat_dtype, cfg.data_seed) if with_features else None
    tg = targets(cfg.num_nodes, H * cfg.B, cfg.data_seed + 2).reshape(H, cfg.B)
    return dict(cfg=cfg, num_nodes=cfg.num_nodes, offsets=offsets, offsets64=off64, indices=idx,
                features=feat, targets=tg, fanouts=list(cfg.fanouts), H=H, B=cfg.B,
                block_bytes=cfg.block_bytes, seed=cfg.seed, row_bytes=cfg.row_bytes)
