"""Buffer-pool model of the staged feature tier -- TEST INFRASTRUCTURE ONLY.

Only the tests may import this module; the GPU library never loads it.

The paper keeps blocks in a main-memory buffer: blocks already there are
pinned until the current iteration has processed them, and replacement is
least-recently-used (Sec. 3.4(1)).  The staged feature tier applies this to
feature blocks held in an HBM pool of P slots.  This module is the plain
definition of that policy, written for small inputs (linear scans, no heap):

- a hyperbatch needs the feature blocks of its gather bucket, ascending;
- they are taken in rounds of at most P blocks;
- every use of a slot gets the next access number (counting over the life of
  the pool);
- in a round, first every needed block already in the pool is a hit and its
  slot is used (ascending block order), which pins it for the round;
- then every other block of the round, ascending, is a miss: it takes the
  lowest slot that never held a block, else the least recently used slot
  among the slots not used in this round (access numbers are distinct, so
  there are no ties); the block that slot held leaves the pool; the slot is
  used.
"""
from __future__ import annotations

import numpy as np


class PoolModel:
    def __init__(self, pool_blocks: int):
        assert pool_blocks >= 1
        self.P = pool_blocks
        self.slot_block = [-1] * pool_blocks
        self.last_use = [-1] * pool_blocks
        self.where: dict[int, int] = {}
        self.t = 0

    def _use(self, s: int) -> None:
        self.t += 1
        self.last_use[s] = self.t

    def hyperbatch(self, needed_blocks) -> dict:
        """Counters for one hyperbatch whose gather needs `needed_blocks`
        (distinct ids, any order: they are taken ascending)."""
        need = sorted(int(b) for b in set(int(x) for x in needed_blocks))
        staged = hits = rounds = 0
        for i0 in range(0, len(need), self.P):
            t0 = self.t                            # uses after t0 belong to this round
            rounds += 1
            chunk = need[i0:i0 + self.P]
            for b in chunk:
                if b in self.where:
                    self._use(self.where[b])
                    hits += 1
            for b in chunk:
                if b in self.where:
                    continue
                never = [s for s in range(self.P) if self.slot_block[s] == -1]
                if never:
                    s = min(never)
                else:
                    cand = [(self.last_use[s], s) for s in range(self.P) if self.last_use[s] <= t0]
                    assert cand, "every slot is pinned in this round"
                    s = min(cand)[1]
                    del self.where[self.slot_block[s]]
                self.slot_block[s] = b
                self.where[b] = s
                self._use(s)
                staged += 1
            for b in chunk:                       # pinned: every block of the round is present
                assert self.slot_block[self.where[b]] == b
        return dict(needed_blocks=len(need), staged_blocks=staged, hit_blocks=hits, rounds=rounds)


def needed_blocks(minibatches, rows_per_block: int) -> np.ndarray:
    """Feature blocks a hyperbatch's gather touches: the distinct blocks of all
    its minibatches' node lists, ascending."""
    if not minibatches:
        return np.zeros(0, np.int64)
    nodes = np.concatenate([np.asarray(m.nodes, dtype=np.int64) for m in minibatches])
    return np.unique(nodes // rows_per_block)


class CachedPoolModel:
    """The staged tier with a feature cache (Sec. 3.4(2): access counts per
    feature vector; vectors whose count reaches a threshold are kept in a
    feature cache; the others are loaded with their blocks when needed).

    Per hyperbatch:
    - its rows are the distinct nodes of its minibatches; a row's multiplicity
      is the number of minibatches holding it;
    - rows in the cache are served from it; the needed blocks are the blocks
      of the other rows, and go through the block pool (PoolModel);
    - then every row's access count grows by its multiplicity, and rows not
      in the cache whose count reaches the threshold enter it, ascending by
      node id, while it has fewer than `cache_rows` rows; rows never leave it.
    """

    def __init__(self, pool_blocks: int, cache_rows: int, threshold: int, rows_per_block: int):
        self.pool = PoolModel(pool_blocks)
        self.C = cache_rows
        self.T = threshold
        self.rpb = rows_per_block
        self.cache: dict[int, int] = {}
        self.count: dict[int, int] = {}

    def hyperbatch(self, minibatches) -> dict:
        mult: dict[int, int] = {}
        for m in minibatches:
            for u in set(int(x) for x in np.asarray(m.nodes)):
                mult[u] = mult.get(u, 0) + 1
        rows = sorted(mult)
        hits = [u for u in rows if u in self.cache]
        unc = [u for u in rows if u not in self.cache]
        out = self.pool.hyperbatch(sorted(set(u // self.rpb for u in unc)))
        for u in rows:
            self.count[u] = min(0xFFFFFFFF, self.count.get(u, 0) + mult[u])
        admitted = 0
        for u in unc:
            if self.count[u] >= self.T and len(self.cache) < self.C:
                self.cache[u] = len(self.cache)
                admitted += 1
        out.update(cache_hit_rows=len(hits), admitted_rows=admitted, cached_rows=len(self.cache))
        return out
