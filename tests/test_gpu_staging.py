"""The staged feature tier on the GPU: features in pinned host memory, a pool
of feature-block slots in HBM.

Outputs must be byte-identical to the oracle's (and so to a store with
HBM-resident features) for every pool size, including pools smaller than one
hyperbatch's blocks (several rounds), and the staged / hit / round counters
must equal the buffer-pool model's (oracle/staging.py) over a sequence of
hyperbatches that reuse blocks.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.staging import PoolModel, needed_blocks
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def check_sequence(ag, off, idx, feat, block_bytes, pool, hbs, fan, seed, streams=None):
    store = ag.Store(off, idx, feat, block_bytes, pool_blocks=pool)
    o = oracle.Oracle(off, idx)
    fb = feature_bytes(feat)
    rpb = block_bytes // fb.shape[1]
    model = PoolModel(pool)
    batches = []
    for s, (tg, mb_base) in enumerate(hbs):
        t = torch.from_numpy(np.ascontiguousarray(tg)).cuda()
        if streams is None:
            b = store.prepare(t, fan, seed=seed, mb_base=mb_base)
        else:
            b = store.begin(t, fan, seed=seed, mb_base=mb_base, stream=streams[s % len(streams)])
        batches.append((b, tg, mb_base, t))
        if streams is None:
            _check(b, o, fb, tg, fan, seed, mb_base, off, block_bytes, rpb, model, (pool, s))
    if streams is not None:
        # finish in order on a stream of its own, then check in the same order
        g = torch.cuda.Stream()
        for b, *_ in batches:
            b.finish(stream=g)
        for s, (b, tg, mb_base, _) in enumerate(batches):
            _check(b, o, fb, tg, fan, seed, mb_base, off, block_bytes, rpb, model, (pool, s, "streams"))
    for b, *_ in batches:
        b.close()
    store.close()


def _check(b, o, fb, tg, fan, seed, mb_base, off, block_bytes, rpb, model, tag):
    ref = o.hyperbatch(tg, fan, seed, mb_base)
    got = b.to_host()
    for j in range(tg.shape[0]):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=(tag, j))
    st = b.stats()
    want = oracle.hyperbatch_stats(off, block_bytes, fb.shape[1], ref, len(fan))
    for k, v in want.items():
        assert st[k] == v, (tag, k, st[k], v)
    ts = b.tier_stats()
    mc = model.hyperbatch(needed_blocks(ref, rpb))
    for k, v in mc.items():
        assert ts[k] == v, (tag, k, ts[k], v)
    assert ts["staged_bytes"] == mc["staged_blocks"] * rpb * fb.shape[1]
    log("tier", tag, ts)


@pytest.mark.parametrize("dim,dtype,block_bytes", [(256, np.float32, 4096), (20, np.float32, 256),
                                                   (3, np.float32, 64), (1024, np.float16, 4096)])
@pytest.mark.parametrize("pool", [1, 3, 40, 100000])
def test_staged_tier_matches_oracle_and_pool_model(agnes, dim, dtype, block_bytes, pool):
    off, idx = random_graph(2200, 9, 4, hubs=2, hub_deg=500)
    feat = features(2200, dim, 6, dtype)
    fan = [5, 3]
    hbs = [(distinct_targets(2200, 4, 30, 20 + s), 4 * s) for s in range(3)]
    hbs.append((hbs[0][0], 0))                  # the first hyperbatch again: its blocks may still be pooled
    check_sequence(agnes, off, idx, feat, block_bytes, pool, hbs, fan, seed=7)


def test_staged_tier_batches_in_flight_on_several_streams(agnes):
    off, idx = random_graph(3000, 10, 9, hubs=3, hub_deg=700)
    feat = features(3000, 64, 2)
    fan = [6, 4]
    hbs = [(distinct_targets(3000, 5, 25, 50 + s), 5 * s) for s in range(4)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    check_sequence(agnes, off, idx, feat, 1024, 12, hbs, fan, seed=11, streams=streams)


def test_staged_store_rejects_empty_pool(agnes):
    off, idx = random_graph(100, 4, 1)
    feat = features(100, 8, 1)
    with pytest.raises(agnes.AgnesError):
        agnes.Store(off, idx, feat, 256, pool_blocks=0)


@pytest.mark.parametrize("cache_rows,threshold", [(0, 1), (7, 2), (300, 1), (100000, 3)])
@pytest.mark.parametrize("dim,dtype,block_bytes", [(256, np.float32, 4096), (3, np.float32, 64),
                                                   (20, np.float32, 256)])
def test_feature_cache_matches_oracle_and_model(agnes, cache_rows, threshold, dim, dtype, block_bytes):
    """Hyperbatches that repeat earlier targets make rows hot: rows reaching the
    threshold enter the cache and are served from it, their blocks are no
    longer staged, and every counter equals the model's."""
    from oracle.staging import CachedPoolModel
    off, idx = random_graph(2200, 9, 4, hubs=2, hub_deg=500)
    feat = features(2200, dim, 6, dtype)
    fan = [5, 3]
    base = [distinct_targets(2200, 4, 30, 20 + s) for s in range(3)]
    hbs = [(base[0], 0), (base[1], 4), (base[0], 0), (base[2], 8), (base[0], 0), (base[1], 4)]
    pool = 20
    store = agnes.Store(off, idx, feat, block_bytes, pool_blocks=pool, cache_rows=cache_rows,
                        cache_threshold=threshold)
    o = oracle.Oracle(off, idx)
    fb = feature_bytes(feat)
    rpb = block_bytes // fb.shape[1]
    model = CachedPoolModel(pool, cache_rows, threshold, rpb)
    b = None
    for s, (tg, mb_base) in enumerate(hbs):
        t = torch.from_numpy(np.ascontiguousarray(tg)).cuda()
        b = store.prepare(t, fan, seed=7, mb_base=mb_base, batch=b)
        ref = o.hyperbatch(tg, fan, 7, mb_base)
        got = b.to_host()
        for j in range(tg.shape[0]):
            compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("cache", s, j))
        ts = b.tier_stats()
        want = model.hyperbatch(ref)
        log("cache", cache_rows, threshold, s, ts)
        for k, v in want.items():
            assert ts[k] == v, (s, k, ts[k], v)
    if cache_rows:
        assert ts["cached_rows"] > 0
    b.close()
    store.close()
