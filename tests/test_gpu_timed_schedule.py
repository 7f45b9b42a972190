"""Parity under the schedule the benchmark times, at the 2^23-node workload.

bench.py's own Pipeline runs consecutive fresh hyperbatches with its default
launch configuration: three sampling streams taking turns, three hyperbatches
sampling ahead of the one gathering on the default stream, the "ahead" order,
five batch slots reused, profiling events on.  After a warm-up (every slot
allocated), 8 timed steps are retired one by one while later steps are still
in flight; for each of them:
  - two of its minibatches are compared with the oracle element by element
    (node ids, every hop's row_ptr and col, feature bytes);
  - every gathered row is checked on the device through out[i] == X[nodes[i]]
    (torch's index_select);
and for the first and last timed step the exact statistics of the whole
hyperbatch equal the oracle's.
"""
import ctypes
import os
import sys
import time

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import compare_minibatch, feature_bytes, log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_pipeline_schedule_c3():
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import bench
    import paper_2601_01473_amd as ag

    cfg = synth.CONFIGS["c3"]
    t0 = time.time()
    w = synth.workload(cfg)
    H, B = w["H"], w["B"]
    log(f"[c3 schedule] inputs ready in {time.time() - t0:.1f}s")
    warm, steps = 5, 8
    n_steps = warm + steps
    perm = synth.targets(cfg.num_nodes, n_steps * H * B, cfg.data_seed + 7)
    step_targets = [perm[s * H * B:(s + 1) * H * B].reshape(H, B) for s in range(n_steps)]
    dev_targets = [torch.from_numpy(np.ascontiguousarray(t)).cuda() for t in step_targets]
    store = ag.Store(w["offsets"], w["indices"], w["features"], cfg.block_bytes, feat_dtype=cfg.feat_dtype)
    store.set_profiling(True)
    log("[c3 schedule] store built")
    o = oracle.Oracle(w["offsets64"], w["indices"])
    fb = feature_bytes(w["features"])
    words = cfg.row_bytes // 4
    X = torch.from_numpy(fb.view(np.int32).reshape(-1, words)).cuda()
    hip = ag._hiprt()
    checked = []

    def check(s, batch, record):
        batch.wait()
        if not record:
            return
        v = batch.view()
        rows = int(np.ctypeslib.as_array(v.node_off, shape=(H + 1,))[H])
        nodes = torch.empty(rows, dtype=torch.int32, device="cuda")
        out = torch.empty((rows, words), dtype=torch.int32, device="cuda")
        assert hip.hipMemcpy(ctypes.c_void_p(nodes.data_ptr()), ctypes.c_void_p(v.nodes), rows * 4, 3) == 0
        assert hip.hipMemcpy(ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(v.features), rows * cfg.row_bytes,
                             3) == 0
        chunk = 1 << 20
        for a in range(0, rows, chunk):
            ref = torch.index_select(X, 0, nodes[a:a + chunk].long())
            assert torch.equal(ref, out[a:a + chunk]), ("step", s, "feature rows differ in chunk", a)
        del nodes, out
        sample = sorted({s % H, (7 * s + 3) % H})
        got = batch.to_host(minibatches=sample)
        for k, j in enumerate(sample):
            ref = o.minibatch(step_targets[s][j], cfg.fanouts, cfg.seed, s * H + j)
            compare_minibatch(got[k], ref, oracle.gather(fb, ref.nodes), tag=("step", s, j))
        if s in (warm, warm + steps - 1):
            st = batch.stats()
            ref_all = o.hyperbatch(step_targets[s], cfg.fanouts, cfg.seed, s * H)
            want = oracle.hyperbatch_stats(w["offsets64"], cfg.block_bytes, cfg.row_bytes, ref_all,
                                           len(cfg.fanouts))
            for key, val in want.items():
                assert st[key] == val, ("step", s, key, st[key], val)
        checked.append(s)
        log(f"[c3 schedule] step {s}: {rows} rows and minibatches {sample} ok")

    pipe = bench.Pipeline(store, cfg, H, dev_targets, on_retire=check)
    assert (pipe.D, pipe.NSLOT, len(pipe.s_streams), pipe.schedule) == (3, 5, 3, "ahead")
    pipe.run(0, warm, record=False)
    torch.cuda.synchronize()
    pipe.run(warm, steps, record=True)
    torch.cuda.synchronize()
    assert checked == list(range(warm, warm + steps))
    pipe.close()
    store.close()
    del X
    torch.cuda.empty_cache()
