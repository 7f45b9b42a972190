"""The boundary's contracts on the GPU, through the C ABI.

- Targets in host memory (agnes_hyperbatch_prepare / _begin, Alg. 1's input N)
  and in device memory (the _device variants) give identical outputs, equal to
  the oracle's; host targets are copied by the call, so the caller may
  overwrite them as soon as it returns.
- A hop whose requests plus sampled edges can reach 2^32 is refused with
  AGNES_ERR_RANGE before any device allocation or launch.
- A GraphSAGE forward enqueued on one stream is not overwritten by the next
  hyperbatch begun on the same batch from another stream.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from oracle import sage
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu

_KEEP = []


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def _check(got, off, idx, feat, tg, fan, seed, mb_base, tag):
    ref = oracle.Oracle(off, idx).hyperbatch(tg, fan, seed, mb_base)
    fb = feature_bytes(feat)
    for j in range(tg.shape[0]):
        compare_minibatch(got[j], ref[j], oracle.gather(fb, ref[j].nodes), tag=(tag, j))


def test_host_and_device_targets_agree(agnes):
    n = 3000
    off, idx = random_graph(n, 9, seed=61)
    feat = features(n, 24, 3)
    tg = distinct_targets(n, 6, 50, 62)
    fan = [5, 4]
    log("host vs device targets", tg.shape, fan)
    store = agnes.Store(off, idx, feat, 512)
    bh = store.prepare(tg, fan, seed=7, mb_base=3)
    bd = store.prepare(torch.from_numpy(tg).cuda(), fan, seed=7, mb_base=3)
    gh, gd = bh.to_host(), bd.to_host()
    for j in range(tg.shape[0]):
        for k in ("nodes", "features"):
            assert np.array_equal(gh[j][k], gd[j][k]), (j, k)
        for l in range(len(fan)):
            assert np.array_equal(gh[j]["row_ptr"][l], gd[j]["row_ptr"][l]), (j, l)
            assert np.array_equal(gh[j]["col"][l], gd[j]["col"][l]), (j, l)
    _check(gh, off, idx, feat, tg, fan, 7, 3, "host")
    # two-phase with host targets on a stream of its own
    s = torch.cuda.Stream()
    b2 = store.begin(tg, fan, seed=7, mb_base=3, stream=s).finish(stream=s).wait()
    _check(b2.to_host(), off, idx, feat, tg, fan, 7, 3, "host begin")
    for b in (bh, bd, b2):
        b.close()
    store.close()


def test_host_targets_are_copied_by_the_call(agnes):
    n = 2500
    off, idx = random_graph(n, 8, seed=63)
    feat = features(n, 16, 4)
    tg = distinct_targets(n, 4, 40, 64)
    keep = tg.copy()
    fan = [4, 3]
    store = agnes.Store(off, idx, feat, 256)
    s = torch.cuda.Stream()
    b = store.begin(tg, fan, seed=2, mb_base=0, stream=s)
    tg[:] = 0                         # the caller reuses its array at once
    b.finish(stream=s).wait()
    _check(b.to_host(), off, idx, feat, keep, fan, 2, 0, "copied")
    b.close()
    store.close()


def test_hop_bound_of_2_32_refused_before_any_allocation(agnes):
    """H = 4096, B = 1024, fanout 1024 is a legal call whose hop bound
    (4096 * 1024 * 1025 requests plus edges) reaches 2^32."""
    from paper_2601_01473_amd import _binding as B
    n = 1200
    off, idx = random_graph(n, 6, seed=65)
    feat = features(n, 8, 5)
    store = agnes.Store(off, idx, feat, 256)
    calls = {"n": 0}

    def alloc(nbytes, user):
        calls["n"] += 1
        return None

    def release(ptr, nbytes, user):
        pass

    cbs = (B.DEVICE_ALLOC_FN(alloc), B.DEVICE_FREE_FN(release))
    _KEEP.append(cbs)
    H, Bsz = 4096, 1024
    tg = (np.arange(H * Bsz, dtype=np.int64) % n).astype(np.int32).reshape(H, Bsz)
    for fan in ([1024], [2, 1024], [1024, 1024]):
        log("2^32 bound", H, Bsz, fan)
        agnes.agnes_set_device_allocator(*cbs)
        try:
            with pytest.raises(B.AgnesError) as e:
                store.prepare(tg, fan, seed=0)
        finally:
            agnes.agnes_set_device_allocator(None, None)
        assert e.value.status == B.AGNES_ERR_RANGE, str(e.value)
        assert "2^32" in str(e.value)
    assert calls["n"] == 0
    # the store is still usable
    small = distinct_targets(n, 3, 20, 66)
    b = store.prepare(small, [3, 2], seed=1)
    _check(b.to_host(), off, idx, feat, small, [3, 2], 1, 0, "after refusal")
    b.close()
    store.close()


def test_forward_is_not_overwritten_by_the_next_hyperbatch(agnes):
    n = 40000
    off, idx = random_graph(n, 12, seed=67)
    X = features(n, 256, 6)
    fan = [10, 8]
    t1 = distinct_targets(n, 16, 256, 68)
    t2 = distinct_targets(n, 16, 256, 69)
    store = agnes.Store(off, idx, X, 4096)
    dims = [256, 256, 128]
    rng = np.random.default_rng(70)

    def bits(x):
        u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
        return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)

    Ws = [bits(rng.standard_normal((dims[i + 1], 2 * dims[i])) / np.sqrt(dims[i])) for i in range(2)]
    bs = [(rng.standard_normal(dims[i + 1]) * 0.1).astype(np.float32) for i in range(2)]
    tw = [torch.from_numpy(w.view(np.int16)).cuda() for w in Ws]
    tb = [torch.from_numpy(x).cuda() for x in bs]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    b = store.prepare(t1, fan, seed=11, mb_base=0, stream=sa)
    log("forward on stream A, next hyperbatch on stream B")
    with torch.cuda.stream(sa):
        out = torch.empty((16 * 256, dims[-1]), dtype=torch.float32, device="cuda")
    out = b.sage_forward(tw, tb, out=out, stream=sa)
    b = store.begin(t2, fan, seed=11, mb_base=16, batch=b, stream=sb).finish(stream=sb).wait()
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    mbs = oracle.Oracle(off, idx).hyperbatch(t1, fan, 11, 0)
    ref, bound = sage.forward_hyperbatch(mbs, X.astype(np.float64), Ws, bs)
    err = np.abs(got - ref)
    log("max err", float(err.max()), "max bound", float(bound.max()))
    assert not np.any(err > bound)
    _check(b.to_host(), off, idx, X, t2, fan, 11, 16, "second hyperbatch")
    b.close()
    store.close()
