"""CPU oracle for hyperbatch GNN data preparation -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this package.  The GPU library never loads it, and the two share no code.

``oracle.c`` holds the arithmetic (Philox4x64-10, multiply-shift integer draws,
Floyd's subset algorithm, per-minibatch sampling and relabelling, the blocked
Alg. 1 order, the row gather); this module compiles it with gcc and marshals
numpy arrays.  Everything the oracle returns is plain numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# AGNES_SANITIZE (e.g. "address,undefined") selects a separate build with
# LLVM's sanitizers, loaded only under their preloaded runtime
# (tests/sanitized_cpu_suite.py)
_SAN = os.environ.get("AGNES_SANITIZE", "")
_LIB = os.path.join(_HERE, "liboracle.san.so" if _SAN else "liboracle.so")


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        if _SAN:
            clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
            cmd = [clang, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=" + _SAN,
                   "-fno-sanitize-recover=all", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC]
        else:
            cmd = ["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i32, i64, u64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
        L.oracle_philox4x64_10.restype = None
        L.oracle_philox4x64_10.argtypes = [vp, vp, vp]
        L.oracle_uniform_below.restype = u64
        L.oracle_uniform_below.argtypes = [u64, u64]
        L.oracle_draw_word.restype = u64
        L.oracle_draw_word.argtypes = [u64, i64, i64, i64, i64]
        L.oracle_floyd_from_draws.restype = i64
        L.oracle_floyd_from_draws.argtypes = [i64, i64, vp, vp]
        L.oracle_sample_positions.restype = i64
        L.oracle_sample_positions.argtypes = [i64, i64, u64, i64, i64, i64, vp]
        L.oracle_minibatch.restype = ctypes.c_int
        L.oracle_minibatch.argtypes = [i64, vp, vp, vp, i32, vp, i32, u64, i64, i64, vp, vp, vp,
                                       i64, vp, i64, vp, vp, vp]
        L.oracle_gather.restype = None
        L.oracle_gather.argtypes = [vp, i64, vp, i64, vp]
        L.oracle_hyperbatch_threads.restype = ctypes.c_int
        L.oracle_hyperbatch_threads.argtypes = [i64, vp, vp, vp, i64, vp, i32, i32, vp, i32, u64, i64, i32,
                                                vp, vp, vp, ctypes.c_uint32, vp, vp]
        L.oracle_hyperbatch_blocked.restype = ctypes.c_int
        L.oracle_hyperbatch_blocked.argtypes = [i64, vp, vp, i64, vp, i64, vp, i32, i32, vp, i32,
                                                u64, i64, i64, vp, vp, vp, i64, vp, i64, vp, vp, vp]
        _lib = L
    return _lib


def _p(a) -> int:
    return 0 if a is None else a.ctypes.data


# ------------------------------------------------------------------ primitives

def philox4x64_10(counter, key):
    c = np.asarray(counter, dtype=np.uint64)
    k = np.asarray(key, dtype=np.uint64)
    out = np.empty(4, dtype=np.uint64)
    lib().oracle_philox4x64_10(_p(c), _p(k), _p(out))
    return [int(x) for x in out]


def uniform_below(w: int, n: int) -> int:
    return int(lib().oracle_uniform_below(w, n))


def draw_word(seed: int, v: int, m: int, l: int, i: int) -> int:
    return int(lib().oracle_draw_word(seed, v, m, l, i))


def floyd_from_draws(n: int, k: int, draws) -> list:
    d = np.asarray(draws, dtype=np.uint64)
    out = np.empty(max(k, 1), dtype=np.int64)
    r = lib().oracle_floyd_from_draws(n, k, _p(d), _p(out))
    if r < 0:
        raise ValueError("draw out of range")
    return [int(x) for x in out[:k]]


def sample_positions(deg: int, f: int, seed: int, v: int, m: int, l: int) -> list:
    out = np.empty(max(min(deg, f), 1), dtype=np.int64)
    k = lib().oracle_sample_positions(deg, f, seed, v, m, l, _p(out))
    return [int(x) for x in out[:k]]


# ------------------------------------------------------------------ capacities

def capacities(num_nodes: int, B: int, fanouts) -> tuple:
    """Worst-case (nodes, row_ptr entries, edges) of one minibatch."""
    cap = B
    rp = 0
    edges = 0
    for f in fanouts:
        rp += cap + 1
        edges += cap * f
        cap = min(num_nodes, cap * (1 + f))
    return cap, rp, edges


def _as_i64_offsets(offsets) -> np.ndarray:
    return np.ascontiguousarray(offsets, dtype=np.int64)


class Minibatch:
    """Result of one minibatch: node list, per-hop CSR (local ids), global columns."""

    def __init__(self, nodes, layer_sizes, row_ptr, col, col_global):
        self.nodes = nodes                  # int32 [|N_j|], local-id order
        self.layer_sizes = layer_sizes      # int32 [L+1]
        self.row_ptr = row_ptr              # list of int32 [layer_sizes[l]+1]
        self.col = col                      # list of int32 [edges_l], local ids
        self.col_global = col_global        # list of int32 [edges_l], global ids


class Oracle:
    """Per-graph oracle context (keeps the -1-initialised id scratch)."""

    def __init__(self, offsets, indices, num_nodes=None):
        self.offsets = _as_i64_offsets(offsets)
        self.indices = np.ascontiguousarray(indices, dtype=np.int32)
        self.num_nodes = len(self.offsets) - 1 if num_nodes is None else num_nodes
        self._scratch = np.full(max(self.num_nodes, 1), -1, dtype=np.int32)

    def minibatch(self, targets, fanouts, seed: int, m: int) -> Minibatch:
        """Plain per-node sampling of one minibatch (global minibatch index m)."""
        t = np.ascontiguousarray(targets, dtype=np.int32)
        fan = np.ascontiguousarray(fanouts, dtype=np.int32)
        L = len(fan)
        B = len(t)
        cap_n, cap_rp, cap_e = capacities(self.num_nodes, B, fanouts)
        nodes = np.empty(max(cap_n, 1), np.int32)
        ls = np.empty(L + 1, np.int32)
        ec = np.empty(max(L, 1), np.int64)
        rp = np.empty(max(cap_rp, 1), np.int32)
        col = np.empty(max(cap_e, 1), np.int32)
        colg = np.empty(max(cap_e, 1), np.int32)
        rc = lib().oracle_minibatch(self.num_nodes, _p(self.offsets), _p(self.indices), _p(t), B,
                                    _p(fan), L, seed, m, cap_n, _p(nodes), _p(ls), _p(ec), cap_rp,
                                    _p(rp), cap_e, _p(col), _p(colg), _p(self._scratch))
        if rc == 1:
            raise ValueError("invalid targets (out of range or duplicate within the minibatch)")
        if rc != 0:
            raise RuntimeError("oracle_minibatch failed with code %d" % rc)
        rps, cols, colgs = [], [], []
        r0 = e0 = 0
        for l in range(L):
            n = int(ls[l])
            rps.append(rp[r0:r0 + n + 1].copy())
            cols.append(col[e0:e0 + ec[l]].copy())
            colgs.append(colg[e0:e0 + ec[l]].copy())
            r0 += n + 1
            e0 += int(ec[l])
        return Minibatch(nodes[:ls[L]].copy(), ls.copy(), rps, cols, colgs)

    def hyperbatch(self, targets, fanouts, seed: int, mb_base: int = 0, minibatches=None):
        """Plain order over a hyperbatch: a list with one Minibatch per row of targets
        (only the rows listed in `minibatches` when given; others are None)."""
        targets = np.asarray(targets)
        rows = range(targets.shape[0]) if minibatches is None else minibatches
        out = [None] * targets.shape[0]
        for j in rows:
            out[j] = self.minibatch(targets[j], fanouts, seed, mb_base + j)
        return out


class ThreadedRunner:
    """The plain order over whole hyperbatches on several threads
    (oracle_hyperbatch_threads): every minibatch runs oracle_minibatch and
    oracle_gather unchanged; used to time the CPU baseline on all cores."""

    def __init__(self, offsets, indices, features):
        self.offsets = _as_i64_offsets(offsets)
        self.indices = np.ascontiguousarray(indices, dtype=np.int32)
        self.num_nodes = len(self.offsets) - 1
        f = np.ascontiguousarray(features)
        self.feat = f.view(np.uint8).reshape(self.num_nodes, -1)
        self.seen = np.zeros(max(self.num_nodes, 1), np.uint32)
        self.stamp = 0

    def run(self, targets, fanouts, seed: int, mb_base: int, threads: int = 0) -> dict:
        t = np.ascontiguousarray(targets, dtype=np.int32)
        H, B = t.shape
        fan = np.ascontiguousarray(fanouts, dtype=np.int32)
        L = len(fan)
        ls = np.empty((H, L + 1), np.int32)
        ec = np.empty((H, max(L, 1)), np.int64)
        self.stamp += 1
        d = np.zeros(1, np.int64)
        used = np.zeros(1, np.int32)
        rc = lib().oracle_hyperbatch_threads(self.num_nodes, _p(self.offsets), _p(self.indices), _p(self.feat),
                                             self.feat.shape[1], _p(t), H, B, _p(fan), L, seed, mb_base, threads,
                                             _p(ls), _p(ec), _p(self.seen), self.stamp, _p(d), _p(used))
        if rc != 0:
            raise RuntimeError("oracle_hyperbatch_threads failed with code %d" % rc)
        return dict(layer_sizes=ls, edge_counts=ec[:, :L], distinct=int(d[0]), threads=int(used[0]))


def gather(features: np.ndarray, nodes) -> np.ndarray:
    """Byte copy of the feature rows of `nodes`: [len(nodes), row_bytes] uint8."""
    feat = np.ascontiguousarray(features)
    rb = feat.shape[1] * feat.itemsize if feat.ndim == 2 else feat.itemsize
    n = np.ascontiguousarray(nodes, dtype=np.int32)
    out = np.empty((len(n), rb), dtype=np.uint8)
    lib().oracle_gather(_p(feat), rb, _p(n), len(n), _p(out))
    return out


def hyperbatch_stats(offsets, block_bytes: int, row_bytes: int, mbs, L: int) -> dict:
    """Exact integer statistics of a hyperbatch computed from plain-order results:
    per hop requests R_l, sampled edges S_l, new nodes U_l, non-empty topology
    block rows T_l; rows (sum |N_j|), distinct rows, non-empty feature-block rows."""
    off = _as_i64_offsets(offsets)
    n = len(off) - 1
    E = int(off[-1])
    e_blk = block_bytes // 4
    nblk = max(1, -(-E // e_blk))
    rpb = max(1, block_bytes // row_bytes)
    st = dict(requests=[0] * L, sampled=[0] * L, new_nodes=[0] * L, topo_blocks=[0] * L)
    for l in range(L):
        homes = []
        for mb in mbs:
            st["requests"][l] += int(mb.layer_sizes[l])
            st["sampled"][l] += len(mb.col[l])
            st["new_nodes"][l] += int(mb.layer_sizes[l + 1] - mb.layer_sizes[l])
            fr = mb.nodes[:mb.layer_sizes[l]]
            homes.append(np.minimum(off[fr] // e_blk, nblk - 1))
        st["topo_blocks"][l] = int(np.unique(np.concatenate(homes)).size) if homes else 0
    alln = np.concatenate([mb.nodes for mb in mbs]) if mbs else np.zeros(0, np.int32)
    st["rows"] = int(alln.size)
    u = np.unique(alln)
    st["distinct_rows"] = int(u.size)
    st["feat_blocks"] = int(np.unique(u // rpb).size)
    del n
    return st


def hyperbatch_blocked(offsets, indices, block_bytes: int, features: np.ndarray, targets,
                       fanouts, seed: int, mb_base: int = 0):
    """The hyperbatch in Alg. 1's block-bucketed order (small inputs only).

    Returns (list of Minibatch, list of gathered feature arrays, stats dict)."""
    off = _as_i64_offsets(offsets)
    idx = np.ascontiguousarray(indices, dtype=np.int32)
    n = len(off) - 1
    tg = np.ascontiguousarray(targets, dtype=np.int32)
    H, B = tg.shape
    fan = np.ascontiguousarray(fanouts, dtype=np.int32)
    L = len(fan)
    feat = np.ascontiguousarray(features)
    rb = feat.shape[1] * feat.itemsize
    cap_n, cap_rp, cap_e = capacities(n, B, fanouts)
    nodes = np.empty(H * cap_n, np.int32)
    ls = np.empty(H * (L + 1), np.int32)
    ec = np.empty(H * L, np.int64)
    rp = np.empty(H * max(cap_rp, 1), np.int32)
    col = np.empty(H * max(cap_e, 1), np.int32)
    fout = np.empty((H * cap_n, rb), np.uint8)
    stats = np.empty(4 * L + 3, np.int64)
    rc = lib().oracle_hyperbatch_blocked(n, _p(off), _p(idx), block_bytes, _p(feat), rb, _p(tg), H,
                                         B, _p(fan), L, seed, mb_base, cap_n, _p(nodes), _p(ls),
                                         _p(ec), max(cap_rp, 1), _p(rp), max(cap_e, 1), _p(col),
                                         _p(fout), _p(stats))
    if rc == 1:
        raise ValueError("invalid targets")
    if rc != 0:
        raise RuntimeError("oracle_hyperbatch_blocked failed with code %d" % rc)
    mbs, feats = [], []
    for j in range(H):
        lsj = ls[j * (L + 1):(j + 1) * (L + 1)].copy()
        rps, cols = [], []
        r0 = j * max(cap_rp, 1)
        e0 = j * max(cap_e, 1)
        for l in range(L):
            k = int(lsj[l])
            rps.append(rp[r0:r0 + k + 1].copy())
            e = int(ec[j * L + l])
            cols.append(col[e0:e0 + e].copy())
            r0 += k + 1
            e0 += e
        nj = nodes[j * cap_n: j * cap_n + lsj[L]].copy()
        mbs.append(Minibatch(nj, lsj, rps, cols, None))
        feats.append(fout[j * cap_n: j * cap_n + lsj[L]].copy())
    st = dict(requests=[int(x) for x in stats[0:L]], sampled=[int(x) for x in stats[L:2 * L]],
              new_nodes=[int(x) for x in stats[2 * L:3 * L]],
              topo_blocks=[int(x) for x in stats[3 * L:4 * L]],
              rows=int(stats[4 * L]), distinct_rows=int(stats[4 * L + 1]),
              feat_blocks=int(stats[4 * L + 2]))
    return mbs, feats, st
