"""The oracle against the stored fixtures under tests/golden/.

- hand_example.json: values derived by hand from the definitions (Alg. 1's
  sampling loop with every fanout at least every degree, so no random draw is
  involved), with the derivation written out in the fixture.
- oracle_small.json: the oracle's own output on one small hyperbatch with
  random draws, written by tests/golden/make_oracle_fixtures.py.  It locks the
  oracle's arithmetic: a change that alters it must be justified by the paper
  and the fixture rewritten by that script.
"""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def check_minibatch(mb, want):
    assert mb.nodes.tolist() == want["nodes"]
    assert mb.layer_sizes.tolist() == want["layer_sizes"]
    assert [r.tolist() for r in mb.row_ptr] == want["row_ptr"]
    assert [c.tolist() for c in mb.col] == want["col"]
    if mb.col_global is not None:          # the blocked order returns local ids only
        assert [c.tolist() for c in mb.col_global] == want["col_global"]


def test_hand_fixture_is_the_stated_graph():
    fx = load("hand_example.json")
    g = fx["graph"]
    off, idx = g["offsets"], g["indices"]
    for v, row in g["adjacency"].items():
        v = int(v)
        assert idx[off[v]:off[v + 1]] == row


def test_oracle_matches_hand_derived_fixture():
    fx = load("hand_example.json")
    off = np.array(fx["graph"]["offsets"], np.int64)
    idx = np.array(fx["graph"]["indices"], np.int32)
    tg = np.array(fx["targets"], np.int32)
    mbs = oracle.Oracle(off, idx).hyperbatch(tg, fx["fanouts"], fx["seed"], fx["mb_base"])
    check_minibatch(mbs[0], fx["expected"])
    st = oracle.hyperbatch_stats(off, fx["block_bytes"], fx["row_bytes"], mbs, len(fx["fanouts"]))
    assert st == fx["expected"]["stats"]
    feat = np.arange(6, dtype=np.float32).reshape(6, 1)
    blocked, feats, bst = oracle.hyperbatch_blocked(off, idx, fx["block_bytes"], feat, tg, fx["fanouts"],
                                                    fx["seed"], fx["mb_base"])
    check_minibatch(blocked[0], fx["expected"])
    assert bst == fx["expected"]["stats"]
    assert feats[0].view(np.float32).ravel().tolist() == [float(v) for v in fx["expected"]["nodes"]]


def test_oracle_reproduces_stored_fixture():
    fx = load("oracle_small.json")
    off = np.array(fx["offsets"], np.int64)
    idx = np.array(fx["indices"], np.int32)
    tg = np.array(fx["targets"], np.int32)
    mbs = oracle.Oracle(off, idx).hyperbatch(tg, fx["fanouts"], fx["seed"], fx["mb_base"])
    for mb, want in zip(mbs, fx["expected"]["minibatches"]):
        check_minibatch(mb, want)
    feat = np.array(fx["features"], np.float32)
    st = oracle.hyperbatch_stats(off, fx["block_bytes"], feat.shape[1] * 4, mbs, len(fx["fanouts"]))
    assert st == fx["expected"]["stats"]


def test_stored_fixture_exercises_random_draws():
    """At least one request of every hop takes fewer neighbours than its degree."""
    fx = load("oracle_small.json")
    off = np.array(fx["offsets"], np.int64)
    deg = np.diff(off)
    for l, f in enumerate(fx["fanouts"]):
        partial = 0
        for want in fx["expected"]["minibatches"]:
            frontier = want["nodes"][:want["layer_sizes"][l]]
            partial += sum(1 for v in frontier if deg[v] > f)
        assert partial > 0, l
