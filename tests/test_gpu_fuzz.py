"""Seeded random shapes through the C ABI, element by element against the
oracle: graph size, degree skew (hubs, isolated nodes, repeated edges), H, B,
hop count and fanouts (0, below and above typical degrees), int32 and int64
offsets (int64 also kept 64-bit on the device), row widths and dtypes, block
sizes, the sampling kernels' workgroup cap and graph replay.  Every case runs
twice on one batch with new targets, seed and minibatch base (the second call
replays the sampling kernels from a graph when the shape is small enough)."""
import os

import numpy as np
import pytest

import oracle
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu

# AGNES_FUZZ_CASES widens the sweep (the default suite runs 64)
N_CASES = int(os.environ.get("AGNES_FUZZ_CASES", "64"))


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(200, 6000))
    avg = float(rng.uniform(0.5, 20))
    hubs = int(rng.integers(0, 5))
    hub_deg = int(rng.integers(50, max(51, n // 2)))
    multi = bool(rng.random() < 0.2)
    H = int(rng.integers(1, 49))
    B = int(rng.integers(1, max(2, min(n // H, 300))))
    L = int(rng.integers(1, 4))
    fan = [int(x) for x in rng.choice([0, 1, 2, 3, 5, 7, 10, 15, 25, 30, 40], size=L)]
    o32 = bool(rng.random() < 0.4)
    wide = (not o32) and bool(rng.random() < 0.3)
    dtype = [np.float32, np.float16][int(rng.integers(0, 2))]
    dim = int(rng.choice([2, 4, 8, 24, 64, 128, 256, 300, 512]))
    if dtype == np.float16 and dim % 2:
        dim += 1
    row_bytes = dim * np.dtype(dtype).itemsize
    bb = 1 << int(rng.integers(max(6, int(np.ceil(np.log2(row_bytes)))), 17))
    groups = int(rng.choice([256, 512, 2048]))
    graph = ["auto", True, False][int(rng.integers(0, 3))]
    return dict(n=n, avg=avg, hubs=hubs, hub_deg=hub_deg, multi=multi, H=H, B=B, fan=fan, o32=o32, wide=wide,
                dtype=dtype, dim=dim, bb=bb, groups=groups, graph=graph)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_shape_matches_oracle(agnes, seed, monkeypatch):
    c = _case(seed)
    log("fuzz", seed, {k: (v.__name__ if isinstance(v, type) else v) for k, v in c.items()})
    off, idx = random_graph(c["n"], c["avg"], 2000 + seed, hubs=c["hubs"], hub_deg=c["hub_deg"], multi=c["multi"])
    if c["o32"]:
        off = off.astype(np.int32)
    if c["wide"]:
        monkeypatch.setenv("AGNES_WIDE_OFFSETS", "1")
    feat = features(c["n"], c["dim"], 3000 + seed, c["dtype"])
    store = agnes.Store(off, idx, feat, c["bb"])
    store.set_sampling_groups(c["groups"])
    store.set_sampling_graph(c["graph"])
    o = oracle.Oracle(off, idx)
    fb = feature_bytes(feat)
    b = None
    for rep in range(2):
        tg = distinct_targets(c["n"], c["H"], c["B"], 4000 + 10 * seed + rep)
        s, mb = 7 * seed + rep, 3 * rep
        b = store.prepare(tg, c["fan"], seed=s, mb_base=mb, batch=b)
        got = b.to_host()
        ref = o.hyperbatch(tg, c["fan"], s, mb)
        for j in range(c["H"]):
            compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("fuzz", seed, rep, j))
        st = b.stats()
        want = oracle.hyperbatch_stats(off, c["bb"], fb.shape[1], ref, len(c["fan"]))
        for k, v in want.items():
            assert st[k] == v, ("fuzz", seed, rep, k, st[k], v)
    b.close()
    store.close()


N_LARGE = int(os.environ.get("AGNES_FUZZ_LARGE_CASES", "6"))


def _large_case(seed):
    rng = np.random.default_rng(5000 + seed)
    scale = int(rng.integers(12, 18))
    ef = int(rng.integers(4, 24))
    abc = [(0.57, 0.19, 0.19), (0.65, 0.15, 0.15), (0.45, 0.25, 0.15)][int(rng.integers(0, 3))]
    n = 1 << scale
    H = int(rng.choice([16, 64, 128, 256]))
    bmax = max(1, min(n // H, 1024))                 # H * B <= n: distinct targets
    B = int(rng.integers(min(64, bmax), bmax + 1))
    L = int(rng.integers(1, 4))
    fan = [int(x) for x in rng.choice([2, 5, 10, 15, 25], size=L)]
    groups = int(rng.choice([0, 256, 512, 2048]))
    return dict(scale=scale, ef=ef, abc=abc, n=n, H=H, B=B, fan=fan, groups=groups)


@pytest.mark.parametrize("seed", range(N_LARGE))
def test_random_rmat_shape_matches_oracle(agnes, seed):
    """Larger R-MAT graphs (2^12 to 2^17 nodes, three skews) with hyperbatches
    of up to 256 x 1024 targets: join groups take several tiles each and the
    sampling kernels loop; every minibatch is compared with the oracle."""
    import synth
    c = _large_case(seed)
    log("fuzz large", seed, c)
    off, idx = synth.rmat_csr(c["scale"], c["ef"], c["abc"], 6000 + seed)
    feat = features(c["n"], 16, 7000 + seed)
    store = agnes.Store(off, idx, feat, 1024)
    if c["groups"]:
        store.set_sampling_groups(c["groups"])
    tg = synth.targets(c["n"], c["H"] * c["B"], 8000 + seed).reshape(c["H"], c["B"])
    b = store.prepare(tg, c["fan"], seed=seed, mb_base=11 * seed)
    got = b.to_host()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, c["fan"], seed, 11 * seed)
    fb = feature_bytes(feat)
    for j in range(c["H"]):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("fuzz large", seed, j))
    st = b.stats()
    want = oracle.hyperbatch_stats(off, 1024, fb.shape[1], ref, len(c["fan"]))
    for k, v in want.items():
        assert st[k] == v, ("fuzz large", seed, k, st[k], v)
    b.close()
    store.close()


@pytest.mark.parametrize("scale,abc", [(21, (0.57, 0.19, 0.19)), (22, (0.45, 0.25, 0.15))])
def test_rmat_large_sort_tiles_match_oracle(agnes, scale, abc):
    """2^21 and 2^22 nodes (three radix passes of 8-bit digits) with 64 x 1024
    targets and fanouts [25, 10]: the last hop's bound (about 17 M edges) is
    above 8 M keys, so its sort takes the 8192-key tiles; every minibatch is
    compared with the oracle, and every gathered row through the oracle's
    gather on four of them."""
    import synth
    off, idx = synth.rmat_csr(scale, 16, abc, 9000 + scale)
    n = 1 << scale
    feat = features(n, 16, 9100 + scale)
    store = agnes.Store(off, idx, feat, 1024)
    H, B, fan = 64, 1024, [25, 10]
    tg = synth.targets(n, H * B, 9200 + scale).reshape(H, B)
    b = store.prepare(tg, fan, seed=scale, mb_base=5)
    got = b.to_host()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, scale, 5)
    fb = feature_bytes(feat)
    for j in range(H):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes) if j % 16 == 0 else None,
                          tag=("large sort", scale, j))
    st = b.stats()
    want = oracle.hyperbatch_stats(off, 1024, fb.shape[1], ref, len(fan))
    for k, v in want.items():
        assert st[k] == v, ("large sort", scale, k, st[k], v)
    b.close()
    store.close()
