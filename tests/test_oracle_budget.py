"""Pins of the oracle's fixed-budget tier (section 6.5: eviction under a fixed budget).

Generational eviction: with E* the smallest epoch such that at most `budget` pairs were last used
at or after E*, every pair used before E* is removed.  Pins: hand-computed cases, the defining
properties on random indexes (the survivors fit, they are exactly the pairs at or after E*, and
E* is minimal: keeping one more generation would exceed the budget), the touch semantics of
lookup and store, and the capacity an eviction frees."""

import numpy as np
import pytest

import oracle


def _keys(rng, n):
    return rng.integers(0, 256, size=(n, 16), dtype=np.uint8)


def _index_with_epochs(epochs, rng, cap=1024):
    """One pair per epoch value given, stored by a touching store at that epoch."""
    idx = oracle.Index(cap)
    k = _keys(rng, len(epochs))
    for i, e in enumerate(epochs):
        assert idx.store_touch(k[i:i + 1], np.array([0, 1], np.int64), np.zeros(1, np.int32),
                               np.array([i], np.uint64), int(e)) == 0
    return idx, k


@pytest.mark.parametrize("budget,left", [(6, 6), (5, 5), (4, 3), (3, 3), (2, 0), (0, 0), (100, 6)])
def test_hand_computed_generations(budget, left):
    # epochs 5,5,5,3,3,1: budget 4 keeps only the three newest (the epoch-3 generation does not fit)
    idx, _ = _index_with_epochs([5, 3, 5, 1, 5, 3], np.random.default_rng(1))
    assert idx.evict(budget) == 6 - left
    assert len(idx) == left
    kept = sorted(idx.dump_epochs().tolist())
    assert kept == sorted([5, 3, 5, 1, 5, 3], reverse=True)[:left][::-1] or left == 0


@pytest.mark.parametrize("seed", range(6))
def test_eviction_properties(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    epochs = rng.integers(0, int(rng.integers(1, 40)), size=n)
    budget = int(rng.integers(0, n + 5))
    idx, _ = _index_with_epochs(epochs, rng)
    before = idx.dump_epochs()
    idx.evict(budget)
    after = idx.dump_epochs()
    assert len(after) <= budget
    if len(after) < n:
        cut = after.min() if len(after) else before.max() + 1
        # survivors are exactly the pairs at or after the cut ...
        assert (before >= cut).sum() == len(after)
        # ... and the cut is minimal: the next older generation would not fit
        older = before[before < cut]
        assert (before >= older.max()).sum() > budget
    else:
        assert n <= budget


def test_touch_semantics():
    rng = np.random.default_rng(7)
    k = _keys(rng, 6)
    ko = np.array([0, 6], np.int64)
    idx = oracle.Index(64)
    assert idx.store_touch(k[:4], np.array([0, 4], np.int64), np.zeros(1, np.int32),
                           np.arange(4, dtype=np.uint64), 1) == 0
    # the lookup of k0..k5 hits 4 blocks and touches exactly those
    assert idx.lookup_touch(k, ko, 2).tolist() == [4]
    assert sorted(idx.dump_epochs().tolist()) == [2, 2, 2, 2]
    # a store with hit length 2 inserts k4, k5 at epoch 3 and refreshes the candidates k2, k3 only
    assert idx.store_touch(k, ko, np.array([2], np.int32), np.arange(6, dtype=np.uint64) + 100, 3) == 0
    keys, locs = idx.dump()
    ep = dict(zip([bytes(x) for x in keys], idx.dump_epochs().tolist()))
    lc = dict(zip([bytes(x) for x in keys], locs.tolist()))
    assert [ep[bytes(x)] for x in k] == [2, 2, 3, 3, 3, 3]
    assert [lc[bytes(x)] for x in k] == [0, 1, 2, 3, 104, 105]      # old locations unchanged
    # the plain lookup touches nothing
    idx.lookup(k, ko)
    assert [ep[bytes(x)] for x in k] == [2, 2, 3, 3, 3, 3]


def test_eviction_frees_capacity():
    """Evicted entries stop counting against the capacity: a full index refuses a new key until an
    eviction to a smaller budget removes the least recently used ones."""
    rng = np.random.default_rng(81)
    k = rng.integers(0, 256, size=(3, 16), dtype=np.uint8)
    one = np.array([0, 1], np.int64)
    idx = oracle.Index(2)
    for i in range(2):
        assert idx.store_touch(k[i:i + 1], one, np.zeros(1, np.int32), np.zeros(1, np.uint64), i + 1) == 0
    assert idx.store_touch(k[2:3], one, np.zeros(1, np.int32), np.zeros(1, np.uint64), 3) == oracle.EFULL
    assert len(idx) == 2
    assert idx.evict(1) == 1 and len(idx) == 1
    assert idx.store_touch(k[2:3], one, np.zeros(1, np.int32), np.zeros(1, np.uint64), 3) == 0
    kk, _ = idx.dump()
    assert sorted(bytes(x) for x in kk) == sorted([bytes(k[1]), bytes(k[2])])
    assert idx.evict(0) == 2 and len(idx) == 0
