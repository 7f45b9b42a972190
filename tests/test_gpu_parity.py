"""GPU parity on small inputs: the HIP library against the CPU oracle, element by
element (node ids, per-hop CSR, feature bytes) and the exact statistics.

Sizes span many blocks, several minibatches and ragged tails; cases cover int32
and int64 offsets, fp32/fp16/bf16 and 4-byte-multiple rows, fanout 0, fanouts
above every degree (take-all rows), fanouts above 32 (the sampler's memory
path), isolated targets, multigraph rows and batch reuse with growing shapes.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.graphs import distinct_targets, features, hand_graph, random_graph, star_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def run_case(ag, off, idx, feat, tg, fan, seed, mb_base, block_bytes, batch=None, check_stats=True,
             tag=""):
    store = ag.Store(off, idx, feat, block_bytes)
    t = torch.from_numpy(np.ascontiguousarray(tg, dtype=np.int32)).cuda()
    b = store.prepare(t, fan, seed=seed, mb_base=mb_base, batch=batch)
    got = b.to_host()
    o = oracle.Oracle(off, idx)
    ref = o.hyperbatch(tg, fan, seed, mb_base)
    fb = feature_bytes(feat)
    for j in range(tg.shape[0]):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=(tag, j))
    if check_stats:
        st = b.stats()
        want = oracle.hyperbatch_stats(off, block_bytes, fb.shape[1], ref, len(fan))
        for k, v in want.items():
            assert st[k] == v, (tag, k, st[k], v)
    return store, b


def test_hand_example_on_gpu(agnes):
    off, idx = hand_graph()
    feat = features(6, 4, 0)
    store, b = run_case(agnes, off, idx, feat, np.array([[2, 5]]), [3, 3], 0, 0, 16, tag="hand")
    g = b.to_host()[0]
    assert g["nodes"].tolist() == [2, 5, 0, 1, 4, 3]
    assert g["col"][1].tolist() == [2, 4, 1, 3, 3, 0, 5, 1]
    first, last = store.object_table()
    # 4 edges per block: homes 0,0,0,1,1,1 -> block 0 holds nodes 0..2, block 1 nodes 3..5
    assert first.tolist() == [0, 3] and last.tolist() == [2, 5]


def test_stored_fixture_on_gpu(agnes):
    """The HIP path against values stored under tests/golden/ (written by the
    oracle's fixture script), not against a fresh oracle run."""
    import json
    import os
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_small.json")) as fh:
        fx = json.load(fh)
    off = np.array(fx["offsets"], np.int64)
    idx = np.array(fx["indices"], np.int32)
    feat = np.array(fx["features"], np.float32)
    tg = np.array(fx["targets"], np.int32)
    log("golden oracle_small", tg.shape, fx["fanouts"])
    store = agnes.Store(off, idx, feat, fx["block_bytes"])
    b = store.prepare(torch.from_numpy(tg).cuda(), fx["fanouts"], seed=fx["seed"], mb_base=fx["mb_base"])
    got = b.to_host()
    fb = feature_bytes(feat)
    for j, want in enumerate(fx["expected"]["minibatches"]):
        g = got[j]
        assert g["nodes"].tolist() == want["nodes"], j
        assert g["layer_sizes"].tolist() == want["layer_sizes"], j
        assert [r.tolist() for r in g["row_ptr"]] == want["row_ptr"], j
        assert [c.tolist() for c in g["col"]] == want["col"], j
        assert np.array_equal(g["features"], fb[np.array(want["nodes"], np.int64)]), j
    st = b.stats()
    for k, v in fx["expected"]["stats"].items():
        assert st[k] == v, (k, st[k], v)
    b.close()
    store.close()


@pytest.mark.parametrize("seed", range(4))
def test_random_graphs_int64(agnes, seed):
    off, idx = random_graph(3000, 14, seed, hubs=4, hub_deg=900)
    H, B = 5, 37
    tg = distinct_targets(3000, H, B, seed + 10)
    feat = features(3000, 20, seed)                     # 80-byte rows: 16-byte lanes
    log("random int64", seed)
    run_case(agnes, off, idx, feat, tg, [7, 3, 2], seed=seed, mb_base=3 * seed, block_bytes=256,
             tag=("rand64", seed))


@pytest.mark.parametrize("seed", range(2))
def test_random_graphs_int64_kept_wide_on_device(agnes, seed, monkeypatch):
    """int64 offsets of a graph below 2^31 edges are narrowed to int32 on the
    device; AGNES_WIDE_OFFSETS=1 keeps them 64-bit, so the int64 sampling
    kernels run here too, with the same results."""
    monkeypatch.setenv("AGNES_WIDE_OFFSETS", "1")
    off, idx = random_graph(3000, 14, seed + 20, hubs=4, hub_deg=900)
    tg = distinct_targets(3000, 5, 37, seed + 30)
    feat = features(3000, 20, seed)
    log("random int64 kept wide", seed)
    run_case(agnes, off, idx, feat, tg, [7, 3, 2], seed=seed, mb_base=3 * seed, block_bytes=256,
             tag=("wide64", seed))


def test_random_graph_int32_offsets_fp16(agnes):
    off, idx = random_graph(2000, 9, 7, hubs=3, hub_deg=700)
    tg = distinct_targets(2000, 3, 64, 1)
    feat = features(2000, 24, 2, np.float16)            # 48-byte rows
    run_case(agnes, off.astype(np.int32), idx, feat, tg, [10, 4], 5, 0, 64, tag="int32-fp16")


def test_rows_not_multiple_of_16_bytes(agnes):
    off, idx = random_graph(1500, 6, 3)
    tg = distinct_targets(1500, 2, 50, 2)
    feat = features(1500, 3, 1)                         # 12-byte rows: 4-byte lanes
    run_case(agnes, off, idx, feat, tg, [5, 5], 1, 0, 32, tag="rows12")


def test_bfloat16_rows(agnes):
    off, idx = random_graph(1000, 8, 4)
    tg = distinct_targets(1000, 4, 30, 3)
    rng = np.random.default_rng(0)
    feat = rng.integers(0, 65536, size=(1000, 64), dtype=np.uint16)   # arbitrary bf16 bit patterns
    store = agnes.Store(off, idx, feat, 4096, feat_dtype="bfloat16")
    t = torch.from_numpy(tg).cuda()
    got = store.prepare(t, [6, 2], seed=9).to_host()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, [6, 2], 9, 0)
    for j in range(4):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes), tag=("bf16", j))


def test_zero_fanout_and_take_all(agnes):
    off, idx = random_graph(800, 5, 5, hubs=1, hub_deg=30)
    tg = distinct_targets(800, 3, 20, 4)
    feat = features(800, 8, 3)
    run_case(agnes, off, idx, feat, tg, [0, 40, 0], 2, 0, 128, tag="fan0-all")


def test_large_fanout_memory_path(agnes):
    off, idx = random_graph(1200, 60, 6, hubs=5, hub_deg=1000)
    tg = distinct_targets(1200, 2, 40, 5)
    feat = features(1200, 4, 4)
    run_case(agnes, off, idx, feat, tg, [100, 33], 3, 1, 1024, tag="fanout>32")


@pytest.mark.parametrize("fan", [[1], [4, 4, 4, 4], [3, 8, 16, 32]])
def test_fanout_register_paths(agnes, fan):
    off, idx = random_graph(2500, 30, 8, hubs=3, hub_deg=2000)
    tg = distinct_targets(2500, 3, 25, 6)
    feat = features(2500, 4, 5)
    run_case(agnes, off, idx, feat, tg, fan, 4, 7, 512, tag=("regs", tuple(fan)))


def test_multigraph_rows(agnes):
    off, idx = random_graph(600, 12, 2, multi=True)
    tg = distinct_targets(600, 3, 15, 7)
    feat = features(600, 4, 6)
    run_case(agnes, off, idx, feat, tg, [5, 3], 8, 0, 64, tag="multi")


def test_isolated_and_single_node_graph(agnes):
    off = np.zeros(11, np.int64)
    idx = np.zeros(0, np.int32)
    feat = features(10, 4, 0)
    run_case(agnes, off, idx, feat, np.array([[3, 1], [0, 9]]), [5, 5], 0, 0, 16, tag="no-edges")


def test_determinism_reuse_and_grouping(agnes):
    off, idx = random_graph(2000, 12, 11, hubs=3, hub_deg=600)
    feat = features(2000, 16, 7)
    tg = distinct_targets(2000, 6, 40, 8)
    store = agnes.Store(off, idx, feat, 256)
    t = torch.from_numpy(tg).cuda()
    b = store.prepare(t, [6, 4], seed=3, mb_base=20)
    first = b.to_host()
    b = store.prepare(t, [6, 4], seed=3, mb_base=20, batch=b)        # reuse the batch
    second = b.to_host()
    for x, y in zip(first, second):
        for k in ("nodes", "features"):
            assert np.array_equal(x[k], y[k])
        for l in range(2):
            assert np.array_equal(x["col"][l], y["col"][l])
    # minibatch j alone, with mb_base + j, equals its place in the hyperbatch
    for j in range(6):
        alone = store.prepare(t[j:j + 1], [6, 4], seed=3, mb_base=20 + j).to_host()[0]
        for k in ("nodes", "features"):
            assert np.array_equal(alone[k], first[j][k])
        for l in range(2):
            assert np.array_equal(alone["row_ptr"][l], first[j]["row_ptr"][l])
            assert np.array_equal(alone["col"][l], first[j]["col"][l])
    # a bigger hyperbatch reusing the smaller batch's buffers
    tg2 = distinct_targets(2000, 9, 100, 9)
    b = store.prepare(torch.from_numpy(tg2).cuda(), [8, 5, 2], seed=4, batch=b)
    ref = oracle.Oracle(off, idx).hyperbatch(tg2, [8, 5, 2], 4, 0)
    got = b.to_host()
    for j in range(9):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes), tag=("grow", j))


def test_invalid_targets_are_rejected_and_store_stays_usable(agnes):
    off, idx = random_graph(500, 6, 1)
    feat = features(500, 4, 1)
    store = agnes.Store(off, idx, feat, 64)
    bad_dup = torch.tensor([[1, 2, 1]], dtype=torch.int32).cuda()
    with pytest.raises(agnes.AgnesError) as e:
        store.prepare(bad_dup, [3])
    assert e.value.status == 1
    bad_range = torch.tensor([[1, 500]], dtype=torch.int32).cuda()
    with pytest.raises(agnes.AgnesError) as e:
        store.prepare(bad_range, [3])
    assert e.value.status == 1
    with pytest.raises(agnes.AgnesError):
        store.prepare(torch.tensor([[1, -3]], dtype=torch.int32).cuda(), [3])
    with pytest.raises(agnes.AgnesError):
        store.prepare(torch.tensor([[1, 2]], dtype=torch.int32).cuda(), [2000])
    tg = distinct_targets(500, 2, 10, 0)
    got = store.prepare(torch.from_numpy(tg).cuda(), [3, 3], seed=1).to_host()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, [3, 3], 1, 0)
    for j in range(2):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes))


def test_object_table_matches_offsets(agnes):
    off, idx = random_graph(4000, 10, 12, hubs=2, hub_deg=3000)
    store = agnes.Store(off, idx, features(4000, 4, 0), 1024)
    first, last = store.object_table()
    e_blk = 1024 // 4
    nblk = max(1, -(-int(off[-1]) // e_blk))
    home = np.minimum(off[:-1] // e_blk, nblk - 1)
    for blk in range(nblk):
        vs = np.nonzero(home == blk)[0]
        if len(vs):
            assert first[blk] == vs[0] and last[blk] == vs[-1]
        else:
            assert first[blk] == -1 and last[blk] == -1


def test_two_batches_in_flight_on_two_streams(agnes):
    """begin/finish interleaved over two batches and two streams, as a loader
    overlapping the sampling of one hyperbatch with the gather of another."""
    off, idx = random_graph(3000, 12, 21, hubs=3, hub_deg=900)
    feat = features(3000, 32, 9)
    store = agnes.Store(off, idx, feat, 512)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    fan = [6, 3]
    tgs = [distinct_targets(3000, 5, 40, 100 + k) for k in range(6)]
    dev = [torch.from_numpy(t).cuda() for t in tgs]
    o = oracle.Oracle(off, idx)
    fb = feature_bytes(feat)
    slots = [None, None]
    done = []
    slots[0] = store.begin(dev[0], fan, seed=5, mb_base=0, batch=None, stream=streams[0])
    for k in range(6):
        if k + 1 < 6:
            n = (k + 1) % 2
            if k >= 1:
                done.append((k - 1, slots[n].to_host()))
            slots[n] = store.begin(dev[k + 1], fan, seed=5, mb_base=(k + 1) * 5, batch=slots[n],
                                   stream=streams[n])
        slots[k % 2].finish(stream=streams[k % 2])
    for k in range(4, 6):
        done.append((k, slots[k % 2].to_host()))
    assert sorted(k for k, _ in done) == list(range(6))
    for k, got in done:
        ref = o.hyperbatch(tgs[k], fan, 5, k * 5)
        for j in range(5):
            compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("async", k, j))


def test_three_batches_two_sampling_streams_one_gather_stream(agnes):
    """The loader schedule of bench.py: hyperbatches t+1 and t+2 sample on two
    streams (alternating) while t gathers on a third; every batch is checked."""
    off, idx = random_graph(4000, 10, 31, hubs=3, hub_deg=1200)
    feat = features(4000, 16, 12)
    store = agnes.Store(off, idx, feat, 256)
    s_streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    g_stream = torch.cuda.Stream()
    fan = [5, 4]
    n, D = 8, 2
    tgs = [distinct_targets(4000, 4, 50, 200 + k) for k in range(n)]
    dev = [torch.from_numpy(t).cuda() for t in tgs]
    o = oracle.Oracle(off, idx)
    fb = feature_bytes(feat)
    slots = [None] * (D + 1)
    done = []

    def begin(s):
        k = s % (D + 1)
        slots[k] = store.begin(dev[s], fan, seed=7, mb_base=s * 4, batch=slots[k], stream=s_streams[s % 2])

    for s in range(D):
        begin(s)
    for s in range(n):
        if s >= 1:
            done.append((s - 1, slots[(s - 1) % (D + 1)].to_host()))
        if s + D < n:
            begin(s + D)
        slots[s % (D + 1)].finish(stream=g_stream)
    done.append((n - 1, slots[(n - 1) % (D + 1)].to_host()))
    assert sorted(k for k, _ in done) == list(range(n))
    for k, got in done:
        ref = o.hyperbatch(tgs[k], fan, 7, k * 4)
        for j in range(4):
            compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("3slot", k, j))


def test_finish_on_other_stream_and_errors(agnes):
    off, idx = random_graph(800, 8, 3)
    feat = features(800, 8, 1)
    store = agnes.Store(off, idx, feat, 256)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    tg = distinct_targets(800, 3, 20, 1)
    b = store.begin(torch.from_numpy(tg).cuda(), [4, 4], seed=2, stream=s1)
    b.finish(stream=s2)
    got = b.to_host()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, [4, 4], 2, 0)
    for j in range(3):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes))
    with pytest.raises(agnes.AgnesError):
        b.finish()                          # nothing begun
    bad = torch.tensor([[1, 1]], dtype=torch.int32).cuda()
    b2 = store.begin(bad, [2], seed=0)
    with pytest.raises(agnes.AgnesError):
        b2.finish()                         # duplicate target is reported at finish
    b2 = store.begin(torch.from_numpy(tg).cuda(), [4, 4], seed=2, batch=b2)   # the batch stays usable
    got = b2.finish().to_host()
    for j in range(3):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes))


@pytest.mark.parametrize("rows_dim,dtype", [(20, np.float32), (3, np.float32), (64, np.float32),
                                            (256, np.float32), (384, np.float32), (1024, np.float16),
                                            (1280, np.float32)])
def test_gather_launch_shapes_do_not_change_results(agnes, rows_dim, dtype):
    """Every row-copy launch shape (workgroups, rows in flight) gives the same
    bytes; small workgroup counts force many rows per lane group and ragged ends.
    Rows of 12, 80 and 256 bytes take the lane-group copy; 1 KiB, 1.5 KiB, 2 KiB
    and 5 KiB rows take the wave-per-row copy (one or two units per lane, one to
    three chunks per row, a partial last chunk for 1.5 and 5 KiB)."""
    off, idx = random_graph(2500, 8, 21, hubs=2, hub_deg=600)
    tg = distinct_targets(2500, 4, 45, 3)
    feat = features(2500, rows_dim, 4, dtype)
    fan = [6, 3]
    row_bytes = feat.shape[1] * feat.itemsize
    block = 256
    while block < row_bytes:
        block *= 2
    store = agnes.Store(off, idx, feat, block)
    t = torch.from_numpy(np.ascontiguousarray(tg, dtype=np.int32)).cuda()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, 9, 0)
    fb = feature_bytes(feat)
    want = oracle.hyperbatch_stats(off, block, fb.shape[1], ref, len(fan))
    for groups, unroll, nt, chunks in [(8, 4, True, 1), (8, 16, False, 3), (24, 8, True, 1),
                                       (2048, 4, False, 7), (65536, 8, True, 64), (1000, 16, True, 2),
                                       (1 << 22, 4, True, 1), (1 << 22, 16, False, 5), (1 << 22, 0, True, 1),
                                       (64, 0, False, 3)]:
        log("gather shape", rows_dim, groups, unroll, nt, chunks)
        store.set_gather_shape(groups, unroll, nt, chunks)
        b = store.prepare(t, fan, seed=9, mb_base=0)
        got = b.to_host()
        for j in range(tg.shape[0]):
            compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=(groups, unroll, j))
        st = b.stats()
        for k, v in want.items():
            assert st[k] == v, (groups, unroll, k, st[k], v)
        b.close()
    for bad in [(7, None), ((1 << 22) + 1, None), (None, 3), (None, 2), (None, 32)]:
        with pytest.raises(agnes.AgnesError):
            store.set_gather_shape(*bad)
    for bad_chunks in [0, 65]:
        with pytest.raises(agnes.AgnesError):
            store.set_gather_shape(chunks=bad_chunks)
    store.close()


def test_runs_spanning_join_tiles(agnes):
    """Node 0 is a neighbour of every request: with take-all rows, minibatch j
    holds a run of thousands of equal (0, j) edges, longer than a join tile, and
    the long runs of hop 1 continue across tile and group boundaries."""
    off, idx = star_graph(9000, 2, 3)
    tg = (np.random.default_rng(9).permutation(8999)[:6000] + 1).reshape(2, 3000).astype(np.int32)
    feat = features(9000, 8, 8)
    run_case(agnes, off, idx, feat, tg, [4, 3], 5, 0, 512, tag="star")


def test_many_minibatches(agnes):
    """H = 4096 minibatches of 2 targets: the widest per-minibatch LDS tables."""
    off, idx = random_graph(20000, 6, 12, hubs=2, hub_deg=3000)
    tg = distinct_targets(20000, 4096, 2, 10)
    feat = features(20000, 4, 9)
    run_case(agnes, off, idx, feat, tg, [3, 2], 6, 11, 256, tag="H4096")


def test_single_minibatch_many_targets(agnes):
    """H = 1: minibatch ranking without minibatch bits; ragged last tile."""
    off, idx = random_graph(30000, 9, 13, hubs=3, hub_deg=5000)
    tg = distinct_targets(30000, 1, 7001, 11)
    feat = features(30000, 8, 10)
    run_case(agnes, off, idx, feat, tg, [6, 4], 7, 2, 1024, tag="H1")


def _same_outputs(a, b, tag):
    for key in ("nodes", "layer_sizes", "features"):
        assert np.array_equal(a[key], b[key]), (tag, key)
    for key in ("row_ptr", "col"):
        assert len(a[key]) == len(b[key]), (tag, key)
        for l, (x, y) in enumerate(zip(a[key], b[key])):
            assert np.array_equal(x, y), (tag, key, l)


def test_sampling_graph_replays_equal_launches(agnes):
    """The sampling kernels replayed from a captured HIP graph give what they
    give launched one by one, on every replay: new targets, seeds and minibatch
    bases each call, torch work and synchronizations between replays, shape
    changes (a new capture) and growing buffers.  The last replay is also
    checked against the oracle."""
    n = 3000
    off, idx = random_graph(n, 12, seed=21)
    feat = features(n, 16, 5)
    one_by_one = agnes.Store(off, idx, feat, 256)
    one_by_one.set_sampling_graph(False)
    replayed = agnes.Store(off, idx, feat, 256)
    replayed.set_sampling_graph(True)
    shapes = [(4, 64, [5, 3])] * 4 + [(2, 32, [7])] * 3 + [(4, 64, [5, 3])] * 2 + [(8, 128, [5, 3])] * 3
    b1 = b2 = None
    side = torch.cuda.Stream()
    for i, (H, B, fan) in enumerate(shapes):
        tg = distinct_targets(n, H, B, 100 + i)
        log("graph replay", i, H, B, fan)
        t = torch.from_numpy(tg).cuda()
        b1 = one_by_one.prepare(t, fan, seed=9 + i, mb_base=10 * i, batch=b1)
        b2 = replayed.prepare(t, fan, seed=9 + i, mb_base=10 * i, batch=b2, stream=side if i % 2 else None)
        got1, got2 = b1.to_host(), b2.to_host()
        for j in range(H):
            _same_outputs(got1[j], got2[j], (i, j))
        assert b1.stats()["rows"] == b2.stats()["rows"]
        # unrelated eager work and a synchronization before the next replay
        x = torch.randn(4096, device="cuda")
        assert torch.isfinite((x * 2).sum()).item()
        torch.cuda.synchronize()
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, 9 + i, 10 * i)
    fb = feature_bytes(feat)
    for j in range(H):
        compare_minibatch(got2[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("graph", j))
    for b in (b1, b2):
        b.close()
    one_by_one.close()
    replayed.close()


def test_torch_allocator_owns_device_memory(agnes):
    """With torch's caching allocator installed, the library's device memory
    is torch's (memory_allocated grows), results stay bit-exact, and every
    block goes back when the store and batch close.  A store built before the
    switch keeps freeing through hipFree."""
    off, idx = random_graph(2000, 10, seed=31)
    feat = features(2000, 32, 6)
    tg = distinct_targets(2000, 6, 48, 44)
    old_store = agnes.Store(off, idx, feat, 512)       # hipMalloc
    t_dev = torch.from_numpy(tg).cuda()
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    agnes.use_torch_allocator(True)
    try:
        store = agnes.Store(off, idx, feat, 512)
        assert torch.cuda.memory_allocated() > base
        b = None
        for rep in range(3):
            log("torch allocator", rep)
            b = store.prepare(t_dev, [6, 4], seed=3 + rep, mb_base=rep, batch=b)
            got = b.to_host()
            ref = oracle.Oracle(off, idx).hyperbatch(tg, [6, 4], 3 + rep, rep)
            fb = feature_bytes(feat)
            for j in range(tg.shape[0]):
                compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("torch-alloc", rep, j))
        # a batch of the hipMalloc store, allocated while torch's allocator is installed
        b2 = old_store.prepare(t_dev, [6, 4], seed=3, mb_base=0)
        ref0 = oracle.Oracle(off, idx).hyperbatch(tg, [6, 4], 3, 0)
        assert b2.to_host()[0]["nodes"].tolist() == ref0[0].nodes.tolist()
        b.close()
        b2.close()
        store.close()
    finally:
        agnes.use_torch_allocator(False)
    import gc
    gc.collect()
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() <= base
    old_store.close()


def test_argument_limits_are_rejected_and_store_stays_usable(agnes):
    from paper_2601_01473_amd import _binding as B
    off, idx = random_graph(300, 6, seed=61)
    feat = features(300, 8, 2)
    store = agnes.Store(off, idx, feat, 256)
    good = distinct_targets(300, 2, 8, 3)
    cases = [
        (np.zeros((0, 8), np.int32), [3]),            # H = 0
        (np.zeros((2, 0), np.int32), [3]),            # B = 0
        (good, []),                                   # L = 0
        (good, [1] * 9),                              # L = 9
        (good, [-1]),                                 # negative fanout
        (good, [1025]),                               # fanout above 1024
    ]
    for tg, fan in cases:
        log("limit", tg.shape, fan)
        t = torch.from_numpy(np.ascontiguousarray(tg)).cuda() if tg.size else torch.zeros(tg.shape, dtype=torch.int32, device="cuda")
        with pytest.raises((B.AgnesError, ValueError)) as e:
            store.prepare(t, fan, seed=0)
        if isinstance(e.value, B.AgnesError):
            assert e.value.status == B.AGNES_ERR_INVALID, (tg.shape, fan, str(e.value))
    with pytest.raises(B.AgnesError) as e:
        store.prepare(torch.from_numpy(good).cuda(), [3], seed=0, mb_base=-1)
    assert e.value.status == B.AGNES_ERR_INVALID
    # H above 4096
    big = np.arange(300, dtype=np.int32)[np.arange(4097) % 300].reshape(4097, 1)
    with pytest.raises(B.AgnesError) as e:
        store.prepare(torch.from_numpy(big).cuda(), [1], seed=0)
    assert e.value.status == B.AGNES_ERR_INVALID
    b = store.prepare(torch.from_numpy(good).cuda(), [3, 2], seed=4)
    ref = oracle.Oracle(off, idx).hyperbatch(good, [3, 2], 4, 0)
    got = b.to_host()
    for j in range(good.shape[0]):
        compare_minibatch(got[j], ref[j], oracle.gather(feature_bytes(feat), ref[j].nodes), tag=("after limits", j))
    b.close()
    store.close()


def test_largest_fanout_against_a_hub(agnes):
    """Fanout 1024 (the largest accepted) where a hub has 3000 neighbours, so
    Floyd draws 1024 of 3000 positions in the sampler's staged-position path."""
    n = 4000
    rng = np.random.default_rng(71)
    rows = [np.sort(rng.choice(np.arange(1, n), size=3000, replace=False)).astype(np.int32)]
    for v in range(1, n):
        k = int(rng.integers(0, 12))
        cand = np.delete(np.arange(n), v)
        rows.append(np.sort(rng.choice(cand, size=k, replace=False)).astype(np.int32))
    off = np.zeros(n + 1, np.int64)
    off[1:] = np.cumsum([len(r) for r in rows])
    idx = np.concatenate(rows).astype(np.int32)
    feat = features(n, 8, 3)
    tg = np.array([[0, 5, 17, 900], [0, 2, 3, 4]], np.int32)
    run_case(agnes, off, idx, feat, tg, [1024], 9, 2, 4096, tag="fanout 1024")


def test_eight_hops(agnes):
    """The largest hop count: eight hops of small fanouts, frontiers capped by
    the graph's size."""
    off, idx = random_graph(600, 5, seed=81)
    feat = features(600, 4, 5)
    tg = distinct_targets(600, 3, 4, 8)
    run_case(agnes, off, idx, feat, tg, [2, 2, 1, 2, 1, 1, 2, 1], 13, 3, 256, tag="eight hops")
