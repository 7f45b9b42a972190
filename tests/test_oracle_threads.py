"""The all-cores runner of the CPU baseline (oracle_hyperbatch_threads) runs the
plain per-minibatch oracle unchanged: its per-minibatch layer sizes and edge
counts, and the distinct nodes of the hyperbatch, equal those of the plain
order run one minibatch at a time, for any thread count."""
import numpy as np
import pytest

import oracle
from tests.graphs import distinct_targets, features, random_graph


@pytest.mark.parametrize("threads", [1, 3, 8])
def test_threaded_runner_equals_plain_order(threads):
    n = 1500
    off, idx = random_graph(n, 7, seed=81)
    feat = features(n, 12, 2)
    tg = distinct_targets(n, 9, 30, 82)
    fan = [4, 3]
    run = oracle.ThreadedRunner(off, idx, feat)
    for rep in range(2):
        got = run.run(tg, fan, seed=5, mb_base=10 * rep, threads=threads)
        ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, 5, 10 * rep)
        assert got["threads"] == threads
        for j in range(tg.shape[0]):
            assert got["layer_sizes"][j].tolist() == ref[j].layer_sizes.tolist()
            assert got["edge_counts"][j].tolist() == [len(c) for c in ref[j].col]
        assert got["distinct"] == len(np.unique(np.concatenate([m.nodes for m in ref])))


def test_threaded_runner_rejects_duplicate_targets():
    n = 200
    off, idx = random_graph(n, 5, seed=83)
    run = oracle.ThreadedRunner(off, idx, features(n, 4, 3))
    tg = distinct_targets(n, 2, 10, 84)
    tg[1, 3] = tg[1, 2]
    with pytest.raises(RuntimeError):
        run.run(tg, [3], seed=0, mb_base=0, threads=2)
