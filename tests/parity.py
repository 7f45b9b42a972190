"""Helpers that compare the GPU library's outputs with the CPU oracle."""
import sys

import numpy as np

import oracle


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare_minibatch(gpu: dict, ref: "oracle.Minibatch", feat_ref=None, tag=""):
    """Element-by-element equality of one minibatch (ids, CSR, feature bytes)."""
    L = len(ref.row_ptr)
    assert np.array_equal(gpu["layer_sizes"], ref.layer_sizes), (tag, "layer_sizes",
                                                                 gpu["layer_sizes"], ref.layer_sizes)
    assert np.array_equal(gpu["nodes"], ref.nodes), (tag, "nodes", first_diff(gpu["nodes"], ref.nodes))
    for l in range(L):
        assert np.array_equal(gpu["row_ptr"][l], ref.row_ptr[l]), (tag, "row_ptr", l,
                                                                   first_diff(gpu["row_ptr"][l], ref.row_ptr[l]))
        assert np.array_equal(gpu["col"][l], ref.col[l]), (tag, "col", l, first_diff(gpu["col"][l], ref.col[l]))
    if feat_ref is not None:
        got = gpu["features"]
        assert got.shape == feat_ref.shape, (tag, got.shape, feat_ref.shape)
        if not np.array_equal(got, feat_ref):
            bad = np.nonzero(np.any(got != feat_ref, axis=1))[0]
            raise AssertionError((tag, "feature rows differ", bad[:10], len(bad)))


def first_diff(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    if a.shape != b.shape:
        return ("shape", a.shape, b.shape)
    d = np.nonzero(a != b)[0]
    return ("first", int(d[0]), a[d[0]], b[d[0]]) if len(d) else None


def feature_bytes(features: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(features)
    return f.view(np.uint8).reshape(f.shape[0], -1)
