"""Pins of the oracle's index semantics (lookup = longest stored prefix of block keys; store =
insert-if-absent, section 3.4: an entry already present is never replaced).  Checked against a
brute-force Python dict on small random inputs with planted overlaps."""

import numpy as np
import pytest

import oracle


def _rand_keys(rng, n, pool):
    """n keys drawn from a small pool so that overlaps are frequent."""
    return pool[rng.integers(0, pool.shape[0], size=n)]


def _brute_lookup(table, keys, key_off):
    out = []
    for r in range(len(key_off) - 1):
        h = 0
        while h < key_off[r + 1] - key_off[r] and bytes(keys[key_off[r] + h]) in table:
            h += 1
        out.append(h)
    return np.array(out, np.int32)


def _brute_store(table, keys, key_off, hits, locs):
    new = {}
    for r in range(len(key_off) - 1):
        for j in range(int(hits[r]), int(key_off[r + 1] - key_off[r])):
            k = bytes(keys[key_off[r] + j])
            if k in table:
                continue
            loc = int(locs[key_off[r] + j])
            new[k] = min(loc, new.get(k, loc))
    out = dict(table)
    out.update(new)
    return out


@pytest.mark.parametrize("seed", range(12))
def test_lookup_and_store_against_brute_force(seed):
    rng = np.random.default_rng(seed)
    pool = rng.integers(0, 256, size=(40, 16), dtype=np.uint8)
    n_req = int(rng.integers(1, 12))
    lens = rng.integers(0, 9, size=n_req)
    key_off = np.zeros(n_req + 1, np.int64)
    key_off[1:] = np.cumsum(lens)
    keys = _rand_keys(rng, int(key_off[-1]), pool)
    locs = rng.permutation(10_000)[: int(key_off[-1])].astype(np.uint64)
    # a pre-existing table
    pre_keys = _rand_keys(rng, 15, pool)
    pre_off = np.array([0, 15], np.int64)
    idx = oracle.Index(1024)
    assert idx.store(pre_keys, pre_off, np.zeros(1, np.int32), np.arange(15, dtype=np.uint64) + 50_000) == 0
    table = _brute_store({}, pre_keys, pre_off, [0], np.arange(15, dtype=np.uint64) + 50_000)
    dk, dl = idx.dump()
    assert {bytes(k): int(v) for k, v in zip(dk, dl)} == table

    hits = idx.lookup(keys, key_off)
    assert (hits == _brute_lookup(table, keys, key_off)).all()
    # store with arbitrary (not necessarily lookup-derived) hits
    h2 = np.minimum(hits, rng.integers(0, 9, size=n_req)).astype(np.int32)
    assert idx.store(keys, key_off, h2, locs) == 0
    table = _brute_store(table, keys, key_off, h2, locs)
    dk, dl = idx.dump()
    assert {bytes(k): int(v) for k, v in zip(dk, dl)} == table
    # dump is sorted by unsigned byte order
    assert [bytes(k) for k in dk] == sorted(bytes(k) for k in dk)


def test_store_is_idempotent_and_lookup_after_store_hits_everything():
    rng = np.random.default_rng(99)
    keys = rng.integers(0, 256, size=(50, 16), dtype=np.uint8)
    key_off = np.array([0, 10, 10, 35, 50], np.int64)
    locs = np.arange(50, dtype=np.uint64)
    idx = oracle.Index(64)
    hits = idx.lookup(keys, key_off)
    assert (hits == 0).all()
    assert idx.store(keys, key_off, hits, locs) == 0
    first = idx.dump()
    assert (idx.lookup(keys, key_off) == np.diff(key_off)).all()
    assert idx.store(keys, key_off, np.zeros(4, np.int32), locs + 7) == 0
    second = idx.dump()
    assert (first[0] == second[0]).all() and (first[1] == second[1]).all()   # never overwritten


def test_duplicates_in_one_batch_keep_the_smallest_location():
    k = np.arange(16, dtype=np.uint8)[None].repeat(3, 0)
    idx = oracle.Index(8)
    assert idx.store(k, np.array([0, 1, 2, 3], np.int64), np.zeros(3, np.int32),
                     np.array([30, 10, 20], np.uint64)) == 0
    keys, locs = idx.dump()
    assert keys.shape[0] == 1 and int(locs[0]) == 10


def test_capacity_is_exact():
    rng = np.random.default_rng(5)
    keys = rng.integers(0, 256, size=(9, 16), dtype=np.uint8)
    off = np.array([0, 8], np.int64)
    idx = oracle.Index(8)
    assert idx.store(keys[:8], off, np.zeros(1, np.int32), np.arange(8, dtype=np.uint64)) == 0
    assert len(idx) == 8
    before = idx.dump()
    # one more distinct key does not fit; the index is left unchanged
    assert idx.store(keys[1:9], off, np.zeros(1, np.int32), np.arange(8, dtype=np.uint64)) == oracle.EFULL
    after = idx.dump()
    assert (before[0] == after[0]).all()
    # keys already present cost nothing
    assert idx.store(keys[:8], off, np.zeros(1, np.int32), np.arange(8, dtype=np.uint64)) == 0


def test_reserved_locations_rejected():
    keys = np.zeros((1, 16), np.uint8)
    idx = oracle.Index(8)
    assert idx.store(keys, np.array([0, 1], np.int64), np.zeros(1, np.int32),
                     np.array([1 << 62], np.uint64)) == oracle.ERESERVED
    assert len(idx) == 0
    assert idx.store(keys, np.array([0, 1], np.int64), np.zeros(1, np.int32),
                     np.array([(1 << 62) - 1], np.uint64)) == 0


@pytest.mark.parametrize("seed", range(8))
def test_efull_exactly_when_distinct_keys_exceed_capacity(seed):
    """Store is all or nothing against the capacity: it fails with EFULL iff the index would hold more
    distinct keys than its capacity (section 3.4 store; any 128-bit value is an ordinary key), and a
    failed store leaves the index as it was.  Checked against a Python set over random batches whose
    keys repeat within and across batches."""
    rng = np.random.default_rng(700 + seed)
    cap = int(rng.integers(1, 12))
    pool = rng.integers(0, 256, size=(20, 16), dtype=np.uint8)
    idx = oracle.Index(cap)
    model = set()
    for _ in range(12):
        n = int(rng.integers(0, 6))
        k = pool[rng.integers(0, pool.shape[0], size=n)]
        off = np.array([0, n], np.int64)
        want_full = len(model | {bytes(x) for x in k}) > cap
        before = idx.dump()
        rc = idx.store(k, off, np.zeros(1, np.int32), np.arange(n, dtype=np.uint64))
        if want_full:
            assert rc == oracle.EFULL
            after = idx.dump()
            assert (before[0] == after[0]).all() and (before[1] == after[1]).all()
        else:
            assert rc == 0
            model |= {bytes(x) for x in k}
        assert len(idx) == len(model) <= cap


@pytest.mark.parametrize("seed", range(6))
def test_store_skips_keys_below_the_given_hits(seed):
    """The store path inserts only keys j >= hits[r], whatever the hits say: a caller that already holds
    a prefix (for instance from a local cache) passes its length and those keys stay out of the index."""
    rng = np.random.default_rng(300 + seed)
    pool = rng.integers(0, 256, size=(50, 16), dtype=np.uint8)
    n_req = int(rng.integers(1, 10))
    lens = rng.integers(0, 9, size=n_req)
    key_off = np.zeros(n_req + 1, np.int64)
    key_off[1:] = np.cumsum(lens)
    keys = _rand_keys(rng, int(key_off[-1]), pool)
    locs = rng.permutation(10_000)[: int(key_off[-1])].astype(np.uint64)
    hits = np.array([int(rng.integers(0, n + 2)) for n in lens], np.int32)     # may exceed the true hits
    idx = oracle.Index(1024)
    assert idx.store(keys, key_off, hits, locs) == 0
    dk, dl = idx.dump()
    assert {bytes(k): int(v) for k, v in zip(dk, dl)} == _brute_store({}, keys, key_off, hits, locs)


def test_clone_is_an_independent_copy():
    idx = oracle.Index(64)
    k = np.random.default_rng(5).integers(0, 256, size=(10, 16), dtype=np.uint8)
    ko = np.array([0, 10], np.int64)
    assert idx.store(k[:6], np.array([0, 6], np.int64), np.zeros(1, np.int32), np.arange(6, dtype=np.uint64)) == 0
    c = idx.clone()
    a0, b0 = idx.dump()
    a1, b1 = c.dump()
    assert (a0 == a1).all() and (b0 == b1).all() and c.capacity == idx.capacity
    assert c.store(k, ko, np.zeros(1, np.int32), np.arange(10, dtype=np.uint64) + 100) == 0
    assert len(c) == 10 and len(idx) == 6
    a2, b2 = idx.dump()
    assert (a0 == a2).all() and (b0 == b2).all()


@pytest.mark.parametrize("threads", [3, 17])
def test_threaded_store_and_lookup_match_brute_force(threads):
    """The index's store sorts its candidates on several threads and its lookup splits requests over
    threads: on batches large enough for the threaded sort (2^16 candidates and more), with
    duplicates spread across the slices, the dump equals a Python dict model (smallest location per
    new key, present keys untouched) and the hits equal a brute-force set scan, for every thread
    count."""
    rng = np.random.default_rng(900 + threads)
    pool = rng.integers(0, 256, size=(60000, 16), dtype=np.uint8)
    model = {}
    idx = oracle.Index(1 << 20, threads=threads)
    for rnd in range(3):
        n_req = 700
        lens = rng.integers(0, 200, size=n_req)
        ko = np.zeros(n_req + 1, np.int64)
        ko[1:] = np.cumsum(lens)
        keys = pool[rng.integers(0, pool.shape[0], size=int(ko[-1]))]
        locs = rng.permutation(1 << 24)[: keys.shape[0]].astype(np.uint64)
        hits = idx.lookup(keys, ko)
        want = []
        for r in range(n_req):
            h = 0
            while h < lens[r] and bytes(keys[ko[r] + h]) in model:
                h += 1
            want.append(h)
        assert hits.tolist() == want, rnd
        new = {}
        for r in range(n_req):
            for j in range(int(hits[r]), int(lens[r])):
                k = bytes(keys[ko[r] + j])
                if k not in model:
                    new[k] = min(new.get(k, 1 << 63), int(locs[ko[r] + j]))
        assert idx.store(keys, ko, hits, locs) == 0
        model.update(new)
        gk, gl = idx.dump()
        assert [bytes(x) for x in gk] == sorted(model)
        assert gl.tolist() == [model[k] for k in sorted(model)]
