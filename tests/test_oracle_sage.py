"""Pins of the GraphSAGE oracle (oracle/sage.py), the reference for the GPU
forward pass: a hand-worked example, the two special cases that reduce to a
plain matrix product, an independent dense formulation (mean aggregation as
D^-1 A X over the full neighbourhood, from scipy), and a check that the error
bound covers an emulation of the kernels' low-precision arithmetic."""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from oracle import sage
from tests.graphs import distinct_targets, hand_graph, random_graph
from tests.test_oracle_sampling import scipy_expansion


def bf16_bits(x):
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def test_hand_example():
    # Hand graph, targets [2, 5], one hop with fanout 3 (every neighbour):
    # local ids 0..4 = nodes 2, 5, 0, 1, 4; node 2's neighbours 0, 4, 5 and
    # node 5's neighbour 1.  X[v] = [v, 1], W = [[1, 0, 10, 0], [0, 1, 0, 100]],
    # b = [0.5, 0]:  row 0: self [2, 1], mean [3, 1] -> [32.5, 101];
    # row 1: self [5, 1], mean [1, 1] -> [15.5, 101].
    off, idx = hand_graph()
    mb = oracle.Oracle(off, idx).minibatch(np.array([2, 5]), [3], seed=0, m=0)
    X = np.stack([np.arange(6, dtype=np.float64), np.ones(6)], axis=1)
    W = bf16_bits([[1, 0, 10, 0], [0, 1, 0, 100]])
    out, bound = sage.forward(mb, X, [W], [np.array([0.5, 0.0], np.float32)])
    assert out.tolist() == [[32.5, 101.0], [15.5, 101.0]]
    assert (bound >= 0).all()


def test_relu_between_layers():
    # Two hops on the hand graph.  Layer weights pick single coordinates so the values can be
    # followed: layer 0 maps [h, m] -> [-h0 + m0, h1] (ReLU clips the first
    # coordinate), layer 1 maps [h, m] -> [h0 + m0, h1 + m1].
    off, idx = hand_graph()
    mb = oracle.Oracle(off, idx).minibatch(np.array([2, 5]), [3, 3], seed=0, m=0)
    X = np.stack([np.arange(6, dtype=np.float64), np.ones(6)], axis=1)
    W0 = bf16_bits([[-1, 0, 1, 0], [0, 1, 0, 0]])
    W1 = bf16_bits([[1, 0, 1, 0], [0, 1, 0, 1]])
    z = [np.zeros(2, np.float32)] * 2
    out, _ = sage.forward(mb, X, [W0, W1], z)
    # by hand, layer 0 over hop 1 (nodes 2, 5, 0, 1, 4 with neighbours
    # {0,4,5}, {1}, {1,2}, {3}, {5}):  h' = [max(-v + mean_v, 0), 1]
    h1 = {2: [max(-2 + 3, 0), 1], 5: [max(-5 + 1, 0), 1], 0: [max(0 + 1.5, 0), 1],
          1: [max(-1 + 3, 0), 1], 4: [max(-4 + 5, 0), 1]}
    # layer 1 over hop 0: node 2's neighbours 0, 4, 5; node 5's neighbour 1
    want = [[h1[2][0] + (h1[0][0] + h1[4][0] + h1[5][0]) / 3, 2.0], [h1[5][0] + h1[1][0], 2.0]]
    assert np.allclose(out, want, rtol=0, atol=0)


@pytest.mark.parametrize("seed", range(3))
def test_zero_neighbour_weights_reduce_to_a_matrix_product(seed):
    rng = np.random.default_rng(seed)
    off, idx = random_graph(200, 5, seed)
    tg = distinct_targets(200, 1, 9, seed)[0]
    mb = oracle.Oracle(off, idx).minibatch(tg, [4], seed=seed, m=0)
    X = rng.standard_normal((200, 8))
    Wf = np.concatenate([rng.standard_normal((6, 8)), np.zeros((6, 8))], axis=1)
    W = bf16_bits(Wf)
    b = rng.standard_normal(6).astype(np.float32)
    out, _ = sage.forward(mb, X, [W], [b])
    ref = X[tg] @ sage.bf16_bits_to_f64(W)[:, :8].T + b
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_zero_fanout_gives_zero_mean(seed):
    # fanout 0: every row is empty, the mean is the zero vector, and only the
    # self half of W acts
    rng = np.random.default_rng(seed + 3)
    off, idx = random_graph(200, 5, seed)
    tg = distinct_targets(200, 1, 9, seed)[0]
    mb = oracle.Oracle(off, idx).minibatch(tg, [0], seed=seed, m=0)
    X = rng.standard_normal((200, 8))
    W = bf16_bits(rng.standard_normal((6, 16)))
    b = rng.standard_normal(6).astype(np.float32)
    out, _ = sage.forward(mb, X, [W], [b])
    assert np.allclose(out, X[tg] @ sage.bf16_bits_to_f64(W)[:, :8].T + b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_full_neighbourhood_equals_dense_mean_aggregation(seed):
    # With every fanout >= every degree, hop l's CSR is the full neighbourhood:
    # layer outputs equal relu(H_self Ws^T + (D^-1 A H) Wn^T + b) built from the
    # dense adjacency of scipy's nested expansion, independent of the oracle's
    # sampling and relabelling.
    rng = np.random.default_rng(seed)
    off, idx = random_graph(150, 4, seed, hubs=1, hub_deg=20)
    tg = distinct_targets(150, 1, 6, seed)[0]
    maxdeg = int(np.diff(off).max())
    L = 2
    mb = oracle.Oracle(off, idx).minibatch(tg, [maxdeg] * L, seed=seed, m=0)
    nodes, hops = scipy_expansion(off, idx, tg, L)
    dims = [5, 7, 3]
    X = rng.standard_normal((150, dims[0]))
    Ws = [bf16_bits(rng.standard_normal((dims[i + 1], 2 * dims[i]))) for i in range(L)]
    bs = [rng.standard_normal(dims[i + 1]).astype(np.float32) for i in range(L)]
    out, _ = sage.forward(mb, X, Ws, bs)
    h = X[nodes]
    for i in range(L):
        l = L - 1 - i
        rp, local, _, nd = hops[l]
        A = sp.csr_matrix((np.ones(len(local)), local, rp), shape=(nd, h.shape[0])).toarray()
        deg = A.sum(axis=1, keepdims=True)
        mean = np.divide(A @ h, deg, out=np.zeros((nd, h.shape[1])), where=deg > 0)
        W = sage.bf16_bits_to_f64(Ws[i])
        z = h[:nd] @ W[:, :dims[i]].T + mean @ W[:, dims[i]:].T + bs[i]
        h = np.maximum(z, 0) if i + 1 < L else z
    assert np.allclose(out, h, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("seed", range(3))
def test_bound_covers_low_precision_arithmetic(seed):
    rng = np.random.default_rng(seed + 7)
    off, idx = random_graph(300, 8, seed, hubs=2, hub_deg=60)
    tg = distinct_targets(300, 1, 12, seed)[0]
    mb = oracle.Oracle(off, idx).minibatch(tg, [6, 4], seed=seed, m=0)
    dims = [32, 32, 32]
    X = rng.standard_normal((300, dims[0])).astype(np.float32).astype(np.float64)
    Ws = [bf16_bits(rng.standard_normal((dims[i + 1], 2 * dims[i])) / np.sqrt(2 * dims[i])) for i in range(2)]
    bs = [rng.standard_normal(dims[i + 1]).astype(np.float32) for i in range(2)]
    out, bound = sage.forward(mb, X, Ws, bs)
    sim = sage.simulate_low_precision(mb, X, Ws, bs)
    err = np.abs(sim - out)
    assert (err <= bound).all(), float((err - bound).max())
    assert err.max() > 0                       # the emulation does round
    assert bound.max() < 0.1 * np.abs(out).max() + 0.1     # and the bound stays informative
