"""Small hand-built and random graphs for the tests (inputs only, no method code)."""
import numpy as np


def hand_graph():
    """0:[1,2], 1:[3], 2:[0,4,5], 3:[], 4:[5], 5:[1]"""
    offsets = np.array([0, 2, 3, 6, 6, 7, 8], dtype=np.int64)
    indices = np.array([1, 2, 3, 0, 4, 5, 5, 1], dtype=np.int32)
    return offsets, indices


def random_graph(n, avg_deg, seed, hubs=2, hub_deg=None, multi=False, zero_frac=0.2):
    """CSR with sorted rows: a few hubs, some isolated nodes, the rest Poisson-ish."""
    rng = np.random.default_rng(seed)
    deg = rng.poisson(avg_deg, size=n)
    deg[rng.random(n) < zero_frac] = 0
    hub_deg = hub_deg if hub_deg is not None else max(1, n // 2)
    for h in rng.choice(n, size=min(hubs, n), replace=False):
        deg[h] = hub_deg
    rows = []
    for v in range(n):
        if multi:
            r = np.sort(rng.integers(0, n, size=deg[v]))
        else:
            k = min(int(deg[v]), n - 1)
            cand = np.delete(np.arange(n), v)
            r = np.sort(rng.choice(cand, size=k, replace=False))
        rows.append(r.astype(np.int32))
    offsets = np.zeros(n + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(r) for r in rows])
    indices = np.concatenate(rows) if rows else np.zeros(0, np.int32)
    return offsets, indices.astype(np.int32)


def distinct_targets(n, H, B, seed):
    rng = np.random.default_rng(seed)
    return rng.permutation(n)[: H * B].reshape(H, B).astype(np.int32)


def features(n, dim, seed, dtype=np.float32):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, dim)).astype(dtype)


def star_graph(n, extra, seed):
    """Every node links to node 0 (first in its row) plus `extra` random others:
    node 0 is sampled by every request, so one (node, minibatch) run spans many
    tiles of the join."""
    rng = np.random.default_rng(seed)
    rows = [np.sort(rng.choice(np.arange(1, n), size=min(extra, n - 1), replace=False)).astype(np.int32)]
    for v in range(1, n):
        others = rng.choice(np.arange(1, n), size=extra, replace=False)
        rows.append(np.concatenate([[0], np.sort(others)]).astype(np.int32))
    offsets = np.zeros(n + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(r) for r in rows])
    return offsets, np.concatenate(rows).astype(np.int32)
