"""Pins of the buffer-pool model (oracle/staging.py) used as the reference for
the staged feature tier's counters: a hand-worked LRU example, and the two
cases with closed forms (a pool larger than everything ever needed; a pool of
one block)."""
import numpy as np
import pytest

from oracle.staging import PoolModel, needed_blocks


def test_hand_example_lru_with_pinning():
    # P = 2.  hb1 [0, 1]: 0 -> slot 0 (use 1), 1 -> slot 1 (use 2).
    # hb2 [1, 2]: 1 hits (slot 1, use 3); 2 evicts block 0 (slot 0, last use 1).
    # hb3 [0, 2]: 2 hits (slot 0, use 5); 0 evicts block 1 (slot 1, last use 3).
    m = PoolModel(2)
    assert m.hyperbatch([1, 0]) == dict(needed_blocks=2, staged_blocks=2, hit_blocks=0, rounds=1)
    assert m.hyperbatch([2, 1]) == dict(needed_blocks=2, staged_blocks=1, hit_blocks=1, rounds=1)
    assert m.slot_block == [2, 1]
    assert m.hyperbatch([0, 2]) == dict(needed_blocks=2, staged_blocks=1, hit_blocks=1, rounds=1)
    assert m.slot_block == [2, 0]


def test_rounds_and_least_recently_used_slot():
    # P = 2, one hyperbatch of 3 blocks: round 0 stages 0 (slot 0, use 1) and
    # 1 (slot 1, use 2); round 1 stages 2 into slot 0, the least recently used.
    m = PoolModel(2)
    assert m.hyperbatch([0, 1, 2]) == dict(needed_blocks=3, staged_blocks=3, hit_blocks=0, rounds=2)
    assert m.slot_block == [2, 1]
    # the next hyperbatch needs 1 and 2: both hit in one round
    assert m.hyperbatch([2, 1]) == dict(needed_blocks=2, staged_blocks=0, hit_blocks=2, rounds=1)


@pytest.mark.parametrize("seed", range(5))
def test_pool_larger_than_everything_stages_each_block_once(seed):
    rng = np.random.default_rng(seed)
    hbs = [rng.choice(200, size=rng.integers(1, 60), replace=False) for _ in range(12)]
    m = PoolModel(1000)
    staged = hits = 0
    for hb in hbs:
        c = m.hyperbatch(hb)
        assert c["rounds"] == 1
        staged += c["staged_blocks"]
        hits += c["hit_blocks"]
    assert staged == len(set(np.concatenate(hbs).tolist()))
    assert staged + hits == sum(len(set(h.tolist())) for h in hbs)


@pytest.mark.parametrize("seed", range(5))
def test_pool_of_one_block_keeps_only_the_last(seed):
    rng = np.random.default_rng(seed + 100)
    hbs = [rng.choice(20, size=rng.integers(1, 8), replace=False) for _ in range(10)]
    m = PoolModel(1)
    prev = None
    for hb in hbs:
        need = sorted(set(hb.tolist()))
        c = m.hyperbatch(hb)
        assert c["rounds"] == len(need)
        # only the first block of a hyperbatch can hit: the one left by the previous
        assert c["hit_blocks"] == (1 if prev is not None and need[0] == prev else 0)
        assert c["staged_blocks"] == len(need) - c["hit_blocks"]
        prev = need[-1]


def test_hits_refresh_recency():
    # P = 3: [0, 1, 2] fills slots 0-2 (uses 1-3); [0, 3]: 0 hits (use 4), 3
    # evicts block 1 (slot 1, use 2), not block 0 whose slot was used again.
    m = PoolModel(3)
    m.hyperbatch([0, 1, 2])
    assert m.hyperbatch([3, 0]) == dict(needed_blocks=2, staged_blocks=1, hit_blocks=1, rounds=1)
    assert m.slot_block == [0, 3, 2]


def test_needed_blocks_are_the_distinct_blocks_of_all_node_lists():
    class M:
        def __init__(self, nodes):
            self.nodes = np.asarray(nodes)
    got = needed_blocks([M([9, 3, 4]), M([4, 15, 0])], 4)
    assert got.tolist() == [0, 1, 2, 3]


class _MB:
    def __init__(self, nodes):
        self.nodes = np.asarray(nodes)


def test_cache_hand_example():
    # rows_per_block 2, pool 4 blocks, cache 1 row, threshold 2.
    # hb1: minibatches [0, 5] and [0]: rows 0 (x2), 5; blocks 0, 2 staged; counts
    #      0:2, 5:1; row 0 reaches 2 and enters the cache.
    # hb2: [0, 1]: row 0 from the cache; row 1's block 0 is still pooled (hit);
    #      counts 0:3, 1:1; nothing new reaches 2.
    # hb3: [1] and [1, 5]: rows 1 (x2), 5 not cached; blocks 0, 2 pooled; counts
    #      1:3, 5:2 reach 2 but the cache is full.
    from oracle.staging import CachedPoolModel
    m = CachedPoolModel(4, 1, 2, 2)
    assert m.hyperbatch([_MB([0, 5]), _MB([0])]) == dict(
        needed_blocks=2, staged_blocks=2, hit_blocks=0, rounds=1, cache_hit_rows=0, admitted_rows=1, cached_rows=1)
    assert m.hyperbatch([_MB([0, 1])]) == dict(
        needed_blocks=1, staged_blocks=0, hit_blocks=1, rounds=1, cache_hit_rows=1, admitted_rows=0, cached_rows=1)
    assert m.hyperbatch([_MB([1]), _MB([1, 5])]) == dict(
        needed_blocks=2, staged_blocks=0, hit_blocks=2, rounds=1, cache_hit_rows=0, admitted_rows=0, cached_rows=1)


def test_cache_threshold_one_serves_a_repeated_hyperbatch_entirely():
    from oracle.staging import CachedPoolModel
    rng = np.random.default_rng(3)
    mbs = [_MB(rng.choice(500, size=40, replace=False)) for _ in range(3)]
    m = CachedPoolModel(8, 10 ** 6, 1, 4)
    first = m.hyperbatch(mbs)
    distinct = len(set(np.concatenate([x.nodes for x in mbs]).tolist()))
    assert first["admitted_rows"] == distinct and first["cache_hit_rows"] == 0
    again = m.hyperbatch(mbs)
    assert again == dict(needed_blocks=0, staged_blocks=0, hit_blocks=0, rounds=0, cache_hit_rows=distinct,
                         admitted_rows=0, cached_rows=distinct)


def test_no_cache_reduces_to_the_pool_model():
    from oracle.staging import CachedPoolModel
    rng = np.random.default_rng(5)
    a, b = CachedPoolModel(5, 0, 1, 3), PoolModel(5)
    for _ in range(6):
        mbs = [_MB(rng.choice(100, size=12, replace=False)) for _ in range(2)]
        got = a.hyperbatch(mbs)
        want = b.hyperbatch(needed_blocks(mbs, 3))
        assert {k: got[k] for k in want} == want
        assert got["cache_hit_rows"] == got["admitted_rows"] == got["cached_rows"] == 0
