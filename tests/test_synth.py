"""Checks of the synthetic input generators (inputs only)."""
import numpy as np
import pytest
import torch

import synth


def test_rmat_csr_structure():
    off, idx = synth.rmat_csr(12, 8, (0.57, 0.19, 0.19), seed=3)
    n = 1 << 12
    assert off.shape == (n + 1,) and off[0] == 0 and off[-1] == len(idx)
    assert np.all(np.diff(off) >= 0)
    assert idx.min() >= 0 and idx.max() < n
    src = np.repeat(np.arange(n), np.diff(off))
    assert not np.any(src == idx)                                   # no self-loops
    key = src.astype(np.int64) * n + idx
    assert np.all(np.diff(key) > 0)                                 # sorted, no duplicates
    assert len(idx) > 0.8 * n * 8


def test_rmat_deterministic_and_seeded():
    a = synth.rmat_csr(10, 4, seed=1)
    b = synth.rmat_csr(10, 4, seed=1)
    c = synth.rmat_csr(10, 4, seed=2)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert not np.array_equal(a[1][: min(len(a[1]), len(c[1]))], c[1][: min(len(a[1]), len(c[1]))])


def test_rmat_skew_low_ids_are_hubs():
    off, idx = synth.rmat_csr(14, 16, (0.57, 0.19, 0.19), seed=0)
    deg = np.diff(off)
    assert deg[0] == deg.max()
    assert deg[:64].mean() > 20 * deg.mean()


def test_features_normal_and_seeded():
    x = synth.features(2000, 64, "float32", seed=5)
    assert abs(float(x.mean())) < 0.01 and abs(float(x.std()) - 1.0) < 0.01
    assert np.array_equal(x, synth.features(2000, 64, "float32", seed=5))


@pytest.mark.parametrize("dtype,tdt", [("float16", torch.float16), ("bfloat16", torch.bfloat16)])
def test_half_conversions_match_torch(dtype, tdt):
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(200000).astype(np.float32),
        (rng.standard_normal(20000) * 1e-6).astype(np.float32),     # fp16 subnormal range
        (rng.standard_normal(2000) * 7e4).astype(np.float32),       # fp16 overflow range
        np.array([0.0, -0.0, np.inf, -np.inf, 65504.0, 65519.0, 65520.0, 6.1e-5, 5.96e-8,
                  2.98e-8, 2.99e-8, 1e-45], dtype=np.float32),
    ])
    got = synth.convert_f32(vals, dtype)
    want = torch.from_numpy(vals).to(tdt).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    x = synth.features(1000, 16, dtype, seed=4)
    ref = synth.convert_f32(synth.features(1000, 16, "float32", seed=4), dtype)
    assert np.array_equal(x.view(np.uint16), ref)


def test_targets_distinct_in_range():
    t = synth.targets(5000, 4096, seed=9)
    assert len(np.unique(t)) == 4096 and t.min() >= 0 and t.max() < 5000
    assert np.array_equal(t, synth.targets(5000, 4096, seed=9))
    with pytest.raises(ValueError):
        synth.targets(10, 11)


def test_config_table():
    c = synth.CONFIGS
    assert c["c1"].num_nodes == 1 << 14 and c["c1"].row_bytes == 256
    assert c["c3"].row_bytes == 1024 and c["c3"].fanouts == (25, 10)
    assert c["c4"].row_bytes == 256 and c["c4"].fanouts == (15, 10, 5)
    assert c["c5"].row_bytes == 2048 and c["c5"].h_sweep == (1, 8, 64, 256)


def test_workload_c1():
    w = synth.workload(synth.CONFIGS["c1"])
    assert w["offsets"].dtype == np.int32 and w["targets"].shape == (8, 256)
    assert w["features"].shape == (1 << 14, 64)
