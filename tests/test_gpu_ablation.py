"""The paper's hyperbatch ablation (AGNES-No: every minibatch prepared alone) on
the GPU.

A minibatch prepared alone with mb_base j gives exactly its part of the
hyperbatch (the random streams are keyed by the global minibatch index), and
its statistics equal the oracle's for that minibatch alone.  Block reads of the
one-at-a-time mode are the per-minibatch sums, which are never below the
hyperbatch's once-per-block reads (Sec. 3.3: a block loaded for the hyperbatch
serves every minibatch that needs it).
"""
import json

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def test_minibatches_alone_match_hyperbatch_and_oracle(agnes):
    off, idx = random_graph(3000, 12, 5, hubs=3, hub_deg=800)
    H, B = 6, 40
    tg = distinct_targets(3000, H, B, 8)
    feat = features(3000, 16, 1)
    fan = [6, 4]
    bb = 128
    store = agnes.Store(off, idx, feat, bb)
    t = torch.from_numpy(np.ascontiguousarray(tg)).cuda()
    hb = store.prepare(t, fan, seed=3, mb_base=0)
    got_hb = hb.to_host()
    st_hb = hb.stats()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, 3, 0)
    fb = feature_bytes(feat)
    sums = {"topo": [0] * len(fan), "feat": 0, "distinct": 0}
    for j in range(H):
        b = store.prepare(t[j:j + 1], fan, seed=3, mb_base=j)
        g = b.to_host()[0]
        compare_minibatch(g, ref[j], oracle.gather(fb, ref[j].nodes), tag=("alone", j))
        for k in ("nodes", "layer_sizes"):
            assert np.array_equal(g[k], got_hb[j][k])
        want = oracle.hyperbatch_stats(off, bb, fb.shape[1], [ref[j]], len(fan))
        st = b.stats()
        for k, v in want.items():
            assert st[k] == v, (j, k, st[k], v)
        for l in range(len(fan)):
            sums["topo"][l] += st["topo_blocks"][l]
        sums["feat"] += st["feat_blocks"]
        sums["distinct"] += st["distinct_rows"]
        b.close()
    for l in range(len(fan)):
        assert sums["topo"][l] >= st_hb["topo_blocks"][l]
    assert sums["feat"] >= st_hb["feat_blocks"]
    assert sums["distinct"] >= st_hb["distinct_rows"]
    assert sum(sums["topo"]) > sum(st_hb["topo_blocks"])       # minibatches share blocks here
    hb.close()
    store.close()


def test_bench_ablation_line(agnes):
    """bench.py --ablation on the 2^14-node workload: one JSON line whose counts
    agree with the batch statistics and whose ratios are at least 1."""
    import bench
    cfg = synth.CONFIGS["c1"]
    w = synth.workload(cfg, H=4)
    store = agnes.Store(w["offsets"], w["indices"], w["features"], cfg.block_bytes)
    t = torch.from_numpy(np.ascontiguousarray(w["targets"])).cuda()
    out = bench.ablation(store, cfg, t, 4, 2, 4, cfg.row_bytes, torch)
    log(json.dumps(out))
    assert out["block_read_ratio"] >= 1.0 and out["feature_row_read_ratio"] >= 1.0
    assert out["hyperbatch"]["rows"] == out["one_at_a_time"]["rows"]
    assert out["hyperbatch"]["sampled_edges"] == out["one_at_a_time"]["sampled_edges"]
    o = oracle.Oracle(w["offsets64"], w["indices"])
    ref = o.hyperbatch(w["targets"], cfg.fanouts, cfg.seed, 0)
    want = oracle.hyperbatch_stats(w["offsets64"], cfg.block_bytes, cfg.row_bytes, ref, len(cfg.fanouts))
    assert out["hyperbatch"]["topo_block_reads"] == sum(want["topo_blocks"])
    assert out["hyperbatch"]["feat_block_reads"] == want["feat_blocks"]
    per = [oracle.hyperbatch_stats(w["offsets64"], cfg.block_bytes, cfg.row_bytes, [m], len(cfg.fanouts)) for m in ref]
    assert out["one_at_a_time"]["topo_block_reads"] == sum(sum(p["topo_blocks"]) for p in per)
    assert out["one_at_a_time"]["feat_block_reads"] == sum(p["feat_blocks"] for p in per)
    store.close()
