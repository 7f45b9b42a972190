"""Writes tests/golden/oracle_small.json from the oracle alone.

The fixture locks the oracle's output on one small hyperbatch whose fanouts are
below most degrees, so every Philox word, Floyd draw and relabelling step of the
sampling hops (Alg. 1, sampling loop; Eq. 1's neighbour subsets) shows in it.
A later change of the oracle's arithmetic that alters these values has to name
the passage of the paper that justifies it and rerun this script:

    python tests/golden/make_oracle_fixtures.py

Inputs are built here from numpy's seeded generator and stored in the fixture,
so the test does not depend on any generator staying the same.
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_small.json")


def graph(n=40, seed=3):
    """Sorted rows without self-loops; two hubs, a few isolated nodes."""
    rng = np.random.default_rng(seed)
    deg = rng.poisson(6, size=n)
    deg[rng.random(n) < 0.15] = 0
    deg[rng.choice(n, size=2, replace=False)] = 25
    rows = []
    for v in range(n):
        cand = np.delete(np.arange(n), v)
        rows.append(np.sort(rng.choice(cand, size=min(int(deg[v]), n - 1), replace=False)))
    off = np.zeros(n + 1, np.int64)
    off[1:] = np.cumsum([len(r) for r in rows])
    return off, np.concatenate(rows).astype(np.int32)


def main():
    off, idx = graph()
    n = len(off) - 1
    H, B = 3, 4
    targets = np.random.default_rng(5).permutation(n)[:H * B].reshape(H, B).astype(np.int32)
    fanouts, seed, mb_base = [3, 2], 11, 5
    row_dim = 2
    feat = np.arange(n * row_dim, dtype=np.float32).reshape(n, row_dim) * 0.5 - 3.0
    mbs = oracle.Oracle(off, idx).hyperbatch(targets, fanouts, seed=seed, mb_base=mb_base)
    stats = oracle.hyperbatch_stats(off, 64, row_dim * 4, mbs, len(fanouts))
    fix = {
        "about": "oracle output on one small hyperbatch; written by make_oracle_fixtures.py, "
                 "which calls only the oracle",
        "offsets": off.tolist(), "indices": idx.tolist(),
        "features": feat.tolist(),
        "targets": targets.tolist(), "fanouts": fanouts, "seed": seed, "mb_base": mb_base,
        "block_bytes": 64,
        "expected": {
            "minibatches": [{
                "nodes": mb.nodes.tolist(),
                "layer_sizes": mb.layer_sizes.tolist(),
                "row_ptr": [r.tolist() for r in mb.row_ptr],
                "col": [c.tolist() for c in mb.col],
                "col_global": [c.tolist() for c in mb.col_global],
            } for mb in mbs],
            "stats": stats,
        },
    }
    with open(OUT, "w") as fh:
        json.dump(fix, fh, separators=(",", ":"))
        fh.write("\n")
    print("wrote", OUT)


if __name__ == "__main__":
    main()
