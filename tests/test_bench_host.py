"""bench.py's host-side bookkeeping (no GPU): the committed traffic summary is
used only for the workload and kernel it was measured on, the copy kernel is
named by row width, and graph replay follows the library's rule."""
import os
import sys

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_traffic_summary_only_for_its_workload():
    c3 = synth.CONFIGS["c3"]
    got = bench.measured_traffic(ROOT, f"{c3.describe()}|H={c3.H}")
    assert got is not None
    traffic, algorithmic = got
    assert 1.0 < traffic / algorithmic < 1.1
    assert bench.measured_traffic(ROOT, f"{c3.describe()}|H=8") is None
    c4 = synth.CONFIGS["c4"]
    assert bench.measured_traffic(ROOT, f"{c4.describe()}|H={c4.H}") is None


def test_copy_kernel_named_by_row_width():
    assert bench.copy_kernel_name(1024).startswith("k_gather_rows")
    assert bench.copy_kernel_name(2048).startswith("k_gather_rows")
    assert bench.copy_kernel_name(512).startswith("k_gather ")
    assert bench.copy_kernel_name(1020).startswith("k_gather ")


def test_graph_replay_rule():
    # C1's hops can sample 8*256*10 + 8*2816*5 = 133,120 edges: replayed
    c1 = synth.CONFIGS["c1"]
    assert bench.sampling_replayed(2, c1.H, c1.B, c1.fanouts, c1.num_nodes)
    for name in ("c2", "c3", "c4", "c5"):
        c = synth.CONFIGS[name]
        assert not bench.sampling_replayed(2, c.H, c.B, c.fanouts, c.num_nodes), name
    assert bench.sampling_replayed(1, 64, 1024, (25, 10), 1 << 23)
    assert not bench.sampling_replayed(0, 8, 256, (10, 5), 1 << 14)
    # exactly at the bound: 2^20 edges
    assert bench.sampling_replayed(2, 1, 1 << 20, (1,), 1 << 22)
    assert not bench.sampling_replayed(2, 1, (1 << 20) + 1, (1,), 1 << 22)


def test_offset_width_counted_as_the_device_keeps_it(monkeypatch):
    import numpy as np
    small64 = {"offsets": np.zeros(4, np.int64), "indices": np.zeros(10, np.int32)}
    small32 = {"offsets": np.zeros(4, np.int32), "indices": np.zeros(10, np.int32)}
    assert bench.offset_bytes(small64) == 4
    assert bench.offset_bytes(small32) == 4
    monkeypatch.setenv("AGNES_WIDE_OFFSETS", "1")
    assert bench.offset_bytes(small64) == 8
    assert bench.offset_bytes(small32) == 4


def test_algorithmic_bytes_split_between_sampling_and_copy():
    # one hop: 10 requests, 30 sampled edges, 20 new nodes; 100 output rows
    # of 1 KiB, 40 of them distinct; 4-byte offsets
    st = {"requests": [10], "sampled": [30], "new_nodes": [20], "rows": 100, "distinct_rows": 40}
    bs, bg, copy = bench.algorithmic_bytes(st, 4, 1024)
    assert bs == 10 * (4 + 2 * 4 + 4) + 8 * 30 + 4 * 20
    assert bg == 100 * (4 + 1024) + 40 * 1024
    # the sampling phase packs the output node ids, so the row copy moves rows only
    assert copy == 100 * 1024 + 40 * 1024
    # on the node-range bucket path the row copy also stores the ids
    assert bench.algorithmic_bytes(st, 4, 1024, ids_in_copy=True)[2] == bg
