"""The device generator against numpy's Philox, and allocation failures at every
allocation point of build, prepare and growth (through the C ABI)."""
import numpy as np
import pytest
import torch

import oracle
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import compare_minibatch, feature_bytes, log
from tests.test_oracle_rng import numpy_philox

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def test_device_philox_matches_numpy(agnes):
    """The device Philox4x64-10 (the sampler's own code) against numpy's
    implementation of the published generator: random counters and keys,
    zero words (borrow chains in numpy's counter), and the sampler's keying
    (counter (i / 4, v, m, l), key (seed, 0))."""
    rng = np.random.default_rng(12)
    ctr = rng.integers(0, 2**63, size=(300, 4), dtype=np.uint64) * 2 + rng.integers(0, 2, size=(300, 4), dtype=np.uint64)
    key = rng.integers(0, 2**63, size=(300, 2), dtype=np.uint64) * 2 + 1
    ctr[::4, 0] = 0
    ctr[::8, 1] = 0
    ctr[0] = 0
    key[0] = 0
    extra_c, extra_k = [], []
    for seed in (0, 7):
        for v in (0, 1, 123456, 2**31 - 2):
            for i in range(0, 40, 4):
                extra_c.append([i >> 2, v, 5, 1])
                extra_k.append([seed, 0])
    ctr = np.concatenate([ctr, np.array(extra_c, np.uint64)])
    key = np.concatenate([key, np.array(extra_k, np.uint64)])
    log("device philox", len(ctr))
    got = agnes.agnes_philox4x64_10(ctr, key)
    for n in range(len(ctr)):
        want = numpy_philox([int(x) for x in ctr[n]], [int(x) for x in key[n]])
        assert [int(x) for x in got[n]] == want, n


# Callback pairs stay alive for the whole process: a block keeps the release
# callback of the allocator it came from.
_KEEP = []


def _failing_allocator(agnes, state):
    from paper_2601_01473_amd import _binding as B

    def alloc(nbytes, user):
        k = state["calls"]
        state["calls"] += 1
        if k == state["fail_at"]:
            return None
        dev = torch.cuda.current_device()
        stream = torch.cuda.current_stream(dev)
        ptr = torch.cuda.caching_allocator_alloc(int(nbytes), dev, stream)
        stream.synchronize()
        return ptr

    def release(ptr, nbytes, user):
        torch.cuda.caching_allocator_delete(ptr)

    cbs = (B.DEVICE_ALLOC_FN(alloc), B.DEVICE_FREE_FN(release))
    _KEEP.append(cbs)
    return cbs


def _workload():
    n = 1500
    off, idx = random_graph(n, 8, seed=51)
    feat = features(n, 16, 7)
    small = distinct_targets(n, 4, 32, 9)
    large = distinct_targets(n, 8, 64, 10)
    return off, idx, feat, small, large


def _run(agnes, off, idx, feat, t_small, t_large):
    """build, two prepares of one shape, one larger prepare on the same batch"""
    store = agnes.Store(off, idx, feat, 256)
    b = None
    try:
        b = store.prepare(t_small, [4, 3], seed=1, mb_base=0)
        b = store.prepare(t_small, [4, 3], seed=2, mb_base=4, batch=b)
        b = store.prepare(t_large, [4, 3], seed=3, mb_base=8, batch=b)
        return b.to_host()
    finally:
        if b is not None:
            b.close()
        store.close()


def test_every_allocation_failure_is_reported_and_recoverable(agnes):
    from paper_2601_01473_amd import _binding as B
    off, idx, feat, small, large = _workload()
    t_small = torch.from_numpy(small).cuda()
    t_large = torch.from_numpy(large).cuda()
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    state = {"calls": 0, "fail_at": -1}
    agnes.agnes_set_device_allocator(*_failing_allocator(agnes, state))
    try:
        _run(agnes, off, idx, feat, t_small, t_large)
        total = state["calls"]
        log("allocations in build + 3 prepares:", total)
        assert total >= 20
        for k in range(total):
            state.update(calls=0, fail_at=k)
            with pytest.raises(B.AgnesError) as e:
                _run(agnes, off, idx, feat, t_small, t_large)
            assert e.value.status == B.AGNES_ERR_NOMEM, (k, str(e.value))
            assert "device allocator" in str(e.value)
        state.update(calls=0, fail_at=-1)
        got = _run(agnes, off, idx, feat, t_small, t_large)
    finally:
        agnes.agnes_set_device_allocator(None, None)
    ref = oracle.Oracle(off, idx).hyperbatch(large, [4, 3], 3, 8)
    fb = feature_bytes(feat)
    for j in range(large.shape[0]):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=("after failures", j))
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() <= base
