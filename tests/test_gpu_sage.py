"""GraphSAGE forward on the GPU (agnes_sage_forward) against the float64 oracle
(oracle/sage.py): every output element within the oracle's error bound for
bf16 operands, float32 sums and bf16 hidden storage.

Cases: fp32 / fp16 / bf16 feature rows; one to three layers; output dims that
are and are not multiples of the 128-wide tile; row widths that give the
aggregation every lane-group size (4 to 64 lanes of 16 bytes per row, with a
partial last chunk, and rows of more than 64 pieces); zero fanout (empty rows) and
fanouts above every degree; a batch with many minibatches; and the 2^14-node
workload at full size.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import sage
from tests.graphs import distinct_targets, features, random_graph
from tests.parity import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def agnes():
    import paper_2601_01473_amd as ag
    return ag


def bf16_bits(x):
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def model(dims, seed):
    rng = np.random.default_rng(seed)
    Ws = [bf16_bits(rng.standard_normal((dims[i + 1], 2 * dims[i])) / np.sqrt(dims[i])) for i in range(len(dims) - 1)]
    bs = [rng.standard_normal(dims[i + 1]).astype(np.float32) * 0.1 for i in range(len(dims) - 1)]
    return Ws, bs


def run(ag, off, idx, feat, feat_dtype, X64, tg, fan, dims, seed, block_bytes=256):
    store = ag.Store(off, idx, feat, block_bytes, feat_dtype=feat_dtype)
    t = torch.from_numpy(np.ascontiguousarray(tg, dtype=np.int32)).cuda()
    b = store.prepare(t, fan, seed=seed, mb_base=0)
    Ws, bs = model(dims, seed)
    tw = [torch.from_numpy(w.view(np.int16)).cuda() for w in Ws]
    tb = [torch.from_numpy(x).cuda() for x in bs]
    out = b.sage_forward(tw, tb)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    mbs = oracle.Oracle(off, idx).hyperbatch(tg, fan, seed, 0)
    ref, bound = sage.forward_hyperbatch(mbs, X64, Ws, bs)
    err = np.abs(got - ref)
    log("sage", dims, fan, "max err", float(err.max()), "max bound", float(bound.max()),
        "max |ref|", float(np.abs(ref).max()))
    assert got.shape == ref.shape
    bad = err > bound
    assert not bad.any(), (np.argwhere(bad)[:5], err[bad][:5], bound[bad][:5])
    b.close()
    store.close()
    return got, ref


@pytest.mark.parametrize("dims,fan", [([32, 64, 32], [5, 3]), ([64, 96], [7]), ([32, 32, 160, 32], [4, 3, 2]),
                                      ([128, 256, 64], [6, 4]), ([256, 64], [5]), ([512, 1024, 32], [4, 3])])
def test_fp32_features(agnes, dims, fan):
    off, idx = random_graph(2000, 9, 3, hubs=2, hub_deg=400)
    tg = distinct_targets(2000, 3, 40, 5)
    feat = features(2000, dims[0], 1)
    run(agnes, off, idx, feat, None, feat.astype(np.float64), tg, fan, dims, seed=4,
        block_bytes=max(256, 1 << int(np.ceil(np.log2(dims[0] * 4)))))


@pytest.mark.parametrize("dims", [[64, 64, 32], [128, 256, 96]])
def test_fp16_features(agnes, dims):
    off, idx = random_graph(1500, 8, 6, hubs=2, hub_deg=300)
    tg = distinct_targets(1500, 4, 25, 2)
    feat = features(1500, dims[0], 3, np.float16)
    run(agnes, off, idx, feat, None, feat.astype(np.float64), tg, [5, 5], dims, seed=2)


def test_bf16_features(agnes):
    off, idx = random_graph(1500, 8, 7)
    tg = distinct_targets(1500, 2, 33, 9)
    f32 = features(1500, 96, 5)
    bits = bf16_bits(f32)
    run(agnes, off, idx, bits, "bfloat16", sage.bf16_bits_to_f64(bits), tg, [6, 2], [96, 64, 32], seed=5)


def test_zero_fanout_and_take_all(agnes):
    off, idx = random_graph(1200, 6, 8, hubs=1, hub_deg=100)
    tg = distinct_targets(1200, 2, 30, 1)
    feat = features(1200, 32, 2)
    X = feat.astype(np.float64)
    run(agnes, off, idx, feat, None, X, tg, [0], [32, 32], seed=6)
    run(agnes, off, idx, feat, None, X, tg, [1000, 0], [32, 64, 32], seed=7)


def test_many_minibatches(agnes):
    off, idx = random_graph(3000, 10, 9)
    tg = distinct_targets(3000, 40, 20, 4)
    feat = features(3000, 64, 6)
    run(agnes, off, idx, feat, None, feat.astype(np.float64), tg, [5, 3], [64, 64, 64], seed=8)


def test_workload_2_14_full_size(agnes):
    cfg = synth.CONFIGS["c1"]
    w = synth.workload(cfg)
    run(agnes, w["offsets"], w["indices"], w["features"], None, w["features"].astype(np.float64), w["targets"],
        list(cfg.fanouts), [64, 128, 64], seed=0, block_bytes=cfg.block_bytes)


def test_rejects_wrong_dims(agnes):
    off, idx = random_graph(300, 4, 1)
    feat = features(300, 32, 1)
    store = agnes.Store(off, idx, feat, 256)
    t = torch.from_numpy(distinct_targets(300, 1, 8, 1)).cuda()
    b = store.prepare(t, [3, 3], seed=0)
    Ws, bs = model([32, 32, 32], 1)
    tw = [torch.from_numpy(w.view(np.int16)).cuda() for w in Ws]
    tb = [torch.from_numpy(x).cuda() for x in bs]
    with pytest.raises(agnes.AgnesError):
        b.sage_forward(tw[:1], tb[:1])             # one layer for a two-hop batch
    Ws2, bs2 = model([64, 32, 32], 1)                # dims[0] is not the feature dim
    with pytest.raises(agnes.AgnesError):
        b.sage_forward([torch.from_numpy(w.view(np.int16)).cuda() for w in Ws2],
                       [torch.from_numpy(x).cuda() for x in bs2])
    # misaligned weight and output pointers are refused before any launch
    rows = 8
    big = torch.empty(rows * 32 + 1, dtype=torch.float32, device="cuda")
    with pytest.raises(agnes.AgnesError):
        b.sage_forward(tw, tb, out=big[1:].view(rows, 32))
    wbig = torch.empty(tw[0].numel() + 1, dtype=torch.int16, device="cuda")
    wbig[1:].copy_(tw[0].view(-1))
    with pytest.raises(agnes.AgnesError):
        b.sage_forward([wbig[1:].view(tw[0].shape), tw[1]], tb)
    out = b.sage_forward(tw, tb)                     # the batch is still usable
    torch.cuda.synchronize()
    assert out.shape == (rows, 32) and bool(torch.isfinite(out).all())
    b.close()
    store.close()
