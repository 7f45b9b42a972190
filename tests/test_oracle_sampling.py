"""Pins of the oracle's sampling, relabelling and gathering.

Nothing in the paper prints a worked example with values, so the oracle is
pinned by:
- a hand-derived example (every fanout >= every degree, so no randomness);
- the full-fanout special case, where sampling reduces to the L-hop nested
  neighbourhood expansion, computed independently with scipy.sparse row slicing
  and numpy set routines;
- the invariants every sample must satisfy (true neighbours, min(deg, f)
  distinct positions, ascending rows, distinct nodes with the targets first,
  new nodes of a hop ascending, local ids consistent with the node list);
- the block-bucketed order of Alg. 1 producing exactly the plain order's result;
- independence from how minibatches are grouped into hyperbatches;
- the gathered rows equal numpy fancy indexing of the feature matrix.
"""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from tests.graphs import distinct_targets, features, hand_graph, random_graph


# ------------------------------------------------------------------ hand example

def test_hand_example():
    """Graph 0:[1,2] 1:[3] 2:[0,4,5] 3:[] 4:[5] 5:[1]; targets [2,5]; fanouts [3,3].

    Hop 0: frontier [2,5]; 2 -> {0,4,5}, 5 -> {1}; new = {0,1,4} (5 already in),
      nodes [2,5,0,1,4]; local ids 0->2, 4->4, 5->1, 1->3:
      row_ptr [0,3,4], col [2,4,1,3].
    Hop 1: frontier [2,5,0,1,4]; 2 -> {0,4,5}, 5 -> {1}, 0 -> {1,2}, 1 -> {3},
      4 -> {5}; new = {3}; nodes [2,5,0,1,4,3]:
      row_ptr [0,3,4,6,7,8], col [2,4,1,3,3,0,5,1].
    """
    off, idx = hand_graph()
    mb = oracle.Oracle(off, idx).minibatch([2, 5], [3, 3], seed=0, m=0)
    assert mb.nodes.tolist() == [2, 5, 0, 1, 4, 3]
    assert mb.layer_sizes.tolist() == [2, 5, 6]
    assert mb.row_ptr[0].tolist() == [0, 3, 4]
    assert mb.col[0].tolist() == [2, 4, 1, 3]
    assert mb.row_ptr[1].tolist() == [0, 3, 4, 6, 7, 8]
    assert mb.col[1].tolist() == [2, 4, 1, 3, 3, 0, 5, 1]
    st = oracle.hyperbatch_stats(off, 16, 4, [mb], 2)
    assert st["requests"] == [2, 5] and st["sampled"] == [4, 8] and st["new_nodes"] == [3, 1]
    # 16-byte blocks hold 4 edges: homes of nodes 0..5 are blocks 0,0,0,1,1,1
    # hop 0 frontier {2,5} -> blocks {0,1}; hop 1 frontier adds 0,1,4 -> still {0,1}
    assert st["topo_blocks"] == [2, 2]
    assert st["rows"] == 6 and st["distinct_rows"] == 6


def test_hand_example_zero_fanout_and_isolated_target():
    off, idx = hand_graph()
    mb = oracle.Oracle(off, idx).minibatch([3, 2], [0, 2], seed=0, m=0)
    # hop 0 samples nothing; node 3 has no neighbours; hop 1 takes 2 of {0,4,5}
    assert mb.layer_sizes[:2].tolist() == [2, 2]
    assert mb.row_ptr[0].tolist() == [0, 0, 0]
    assert mb.col[0].size == 0
    assert mb.row_ptr[1].tolist()[:2] == [0, 0]
    assert mb.row_ptr[1][2] == 2


def test_invalid_targets_rejected():
    off, idx = hand_graph()
    o = oracle.Oracle(off, idx)
    with pytest.raises(ValueError):
        o.minibatch([2, 2], [1], 0, 0)
    with pytest.raises(ValueError):
        o.minibatch([6], [1], 0, 0)
    # the scratch map is restored after a failure
    assert o.minibatch([2, 5], [3, 3], 0, 0).nodes.tolist() == [2, 5, 0, 1, 4, 3]


# ------------------------------------------------------------------ full fanout

def scipy_expansion(offsets, indices, targets, L):
    n = len(offsets) - 1
    A = sp.csr_matrix((np.ones(len(indices), dtype=np.int8), indices, offsets), shape=(n, n))
    nodes = np.asarray(targets, dtype=np.int64)
    out = []
    for _ in range(L):
        sub = A[nodes]
        cg = sub.indices.astype(np.int64)
        new = np.setdiff1d(np.unique(cg), nodes)
        nxt = np.concatenate([nodes, new])
        order = np.argsort(nxt, kind="stable")
        local = order[np.searchsorted(nxt[order], cg)]
        out.append((sub.indptr.astype(np.int64), local, cg, len(nodes)))
        nodes = nxt
    return nodes, out


@pytest.mark.parametrize("seed", range(6))
def test_full_fanout_equals_scipy_expansion(seed):
    off, idx = random_graph(300, 4, seed, hubs=2, hub_deg=40)
    maxdeg = int(np.diff(off).max())
    tg = distinct_targets(300, 1, 7, seed)[0]
    L = 3
    mb = oracle.Oracle(off, idx).minibatch(tg, [maxdeg] * L, seed=seed, m=seed)
    nodes, hops = scipy_expansion(off, idx, tg, L)
    assert mb.nodes.tolist() == nodes.tolist()
    for l, (rp, col, cg, nd) in enumerate(hops):
        assert mb.layer_sizes[l] == nd
        assert mb.row_ptr[l].tolist() == rp.tolist()
        assert mb.col[l].tolist() == col.tolist()
        assert mb.col_global[l].tolist() == cg.tolist()


# ------------------------------------------------------------------ invariants

def check_invariants(off, idx, tg, fanouts, mb, simple=True):
    L = len(fanouts)
    nodes = mb.nodes
    assert len(set(nodes.tolist())) == len(nodes)                         # I4 distinct
    assert nodes[: len(tg)].tolist() == list(tg)                          # I4 targets first
    for l, f in enumerate(fanouts):
        nd = int(mb.layer_sizes[l])
        rp, col, cg = mb.row_ptr[l], mb.col[l], mb.col_global[l]
        assert rp[0] == 0 and len(rp) == nd + 1 and np.all(np.diff(rp) >= 0)
        assert nodes[col].tolist() == cg.tolist()                         # local ids
        assert np.all(col < mb.layer_sizes[l + 1])
        seg = nodes[nd: mb.layer_sizes[l + 1]]
        assert np.all(np.diff(seg) > 0)                                   # new nodes ascending
        for r in range(nd):
            v = nodes[r]
            nbrs = idx[off[v]: off[v + 1]]
            row = cg[rp[r]: rp[r + 1]]
            assert len(row) == min(len(nbrs), f)                          # I2
            assert np.all(np.isin(row, nbrs))                             # I1
            if simple:
                assert np.all(np.diff(row) > 0)                           # I3 (+ distinct)


@pytest.mark.parametrize("seed", range(4))
def test_invariants_random_graphs(seed):
    off, idx = random_graph(400, 12, seed, hubs=3, hub_deg=150)
    tg = distinct_targets(400, 1, 16, seed)[0]
    fan = [5, 3, 2]
    mb = oracle.Oracle(off, idx).minibatch(tg, fan, seed=11, m=seed)
    check_invariants(off, idx, tg, fan, mb)


def test_invariants_multigraph_positions_distinct():
    off, idx = random_graph(200, 10, 3, multi=True)
    tg = distinct_targets(200, 1, 10, 3)[0]
    fan = [4, 4]
    mb = oracle.Oracle(off, idx).minibatch(tg, fan, seed=1, m=0)
    check_invariants(off, idx, tg, fan, mb, simple=False)


def test_sampled_rows_are_positions_of_the_key():
    """Each row equals the neighbours at the positions the sampler draws for that key."""
    off, idx = random_graph(300, 20, 9, hubs=2, hub_deg=200)
    tg = distinct_targets(300, 1, 12, 9)[0]
    fan = [6, 4]
    m = 5
    mb = oracle.Oracle(off, idx).minibatch(tg, fan, seed=3, m=m)
    for l, f in enumerate(fan):
        for r in range(int(mb.layer_sizes[l])):
            v = int(mb.nodes[r])
            deg = int(off[v + 1] - off[v])
            pos = oracle.sample_positions(deg, f, 3, v, m, l)
            row = mb.col_global[l][mb.row_ptr[l][r]: mb.row_ptr[l][r + 1]]
            assert row.tolist() == idx[off[v] + np.array(pos, dtype=np.int64)].tolist()


# ------------------------------------------------------------------ Alg. 1 order

def compare_results(a, b):
    assert a.nodes.tolist() == b.nodes.tolist()
    assert a.layer_sizes.tolist() == b.layer_sizes.tolist()
    for x, y in zip(a.row_ptr, b.row_ptr):
        assert x.tolist() == y.tolist()
    for x, y in zip(a.col, b.col):
        assert x.tolist() == y.tolist()


@pytest.mark.parametrize("block_bytes", [16, 64, 4096])
def test_blocked_order_equals_plain_order(block_bytes):
    off, idx = random_graph(500, 10, 21, hubs=3, hub_deg=300)
    H, B = 6, 9
    tg = distinct_targets(500, H, B, 4)
    fan = [6, 3]
    feat = features(500, 8, 1)
    mbs, feats, st = oracle.hyperbatch_blocked(off, idx, block_bytes, feat, tg, fan, seed=2, mb_base=10)
    plain = oracle.Oracle(off, idx).hyperbatch(tg, fan, seed=2, mb_base=10)
    for j in range(H):
        compare_results(mbs[j], plain[j])
        assert np.array_equal(feats[j], oracle.gather(feat, plain[j].nodes))
    assert st == oracle.hyperbatch_stats(off, block_bytes, feat.shape[1] * 4, plain, len(fan))


def test_hand_example_blocked_stats():
    off, idx = hand_graph()
    feat = features(6, 1, 0)
    mbs, feats, st = oracle.hyperbatch_blocked(off, idx, 16, feat, np.array([[2, 5]]), [3, 3], 0)
    assert st["topo_blocks"] == [2, 2]
    # one row per 16-byte feature block of 4-byte rows: 4 rows per block, nodes 0..5 -> blocks 0,1
    assert st["feat_blocks"] == 2 and st["distinct_rows"] == 6 and st["rows"] == 6


def test_grouping_into_hyperbatches_does_not_matter():
    off, idx = random_graph(400, 8, 5, hubs=2, hub_deg=120)
    H, B = 4, 10
    tg = distinct_targets(400, H, B, 8)
    fan = [4, 4]
    feat = features(400, 4, 2)
    whole, _, _ = oracle.hyperbatch_blocked(off, idx, 64, feat, tg, fan, seed=9, mb_base=100)
    for j in range(H):
        alone, _, _ = oracle.hyperbatch_blocked(off, idx, 64, feat, tg[j:j + 1], fan, seed=9,
                                                mb_base=100 + j)
        compare_results(whole[j], alone[0])


def test_determinism():
    off, idx = random_graph(300, 9, 6)
    tg = distinct_targets(300, 1, 20, 6)[0]
    o = oracle.Oracle(off, idx)
    a = o.minibatch(tg, [7, 3], 4, 2)
    b = o.minibatch(tg, [7, 3], 4, 2)
    compare_results(a, b)
    c = o.minibatch(tg, [7, 3], 5, 2)
    assert any(x.tolist() != y.tolist() for x, y in zip(a.col_global, c.col_global))


# ------------------------------------------------------------------ gather

@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_gather_equals_fancy_indexing(dtype):
    feat = features(100, 24, 3, dtype)
    feat[5, 3] = np.array(-0.0, dtype=dtype)
    feat[7, 0] = np.array(np.nan, dtype=dtype)
    nodes = np.array([7, 5, 0, 99, 5, 42], dtype=np.int32)
    got = oracle.gather(feat, nodes)
    want = feat[nodes].view(np.uint8).reshape(len(nodes), -1)
    assert np.array_equal(got, want)
