"""GPU parity of the fused derive-and-lookup call (pkv_derive_lookup) against the oracle: keys bit for
bit and hit lengths exactly, on indexes prepared so that requests hit anywhere from none to all of
their keys, at loads where probes continue into following buckets, on a completely full index, and
at every kernel shape the call switches between (one or two lane-pair workgroups per compute unit,
and the two-kernel path for more requests or other block sizes)."""

import numpy as np
import pytest

import oracle
from tests.gpu_util import THREADS, announce, gpu_available, gpu_batch, oracle_keys
from workloads import Batch, locations, make_workload

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()       # the HIP library must be built; no fallback exists
    return m


def _batch(rng, n_req, max_blocks, block, n_desc=6):
    """Requests of 0..max_blocks blocks (plus a partial block now and then) under a few descriptors."""
    lens = rng.integers(0, max_blocks + 1, size=n_req) * block
    lens += np.where(rng.random(n_req) < 0.3, rng.integers(0, block, size=n_req), 0)
    lens[rng.random(n_req) < 0.05] = 0
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = rng.integers(0, 128256, size=int(off[-1]), dtype=np.int64).astype(np.int32)
    descs = [[(b"model_id", b"m%d" % i), (b"salt", rng.bytes(8))] for i in range(n_desc)]
    return Batch(toks, off, block, descs, rng.integers(0, n_desc, size=n_req).astype(np.int32))


def _prefixes(rng, b):
    """The same requests cut to a random number of whole blocks (the prefixes the index holds)."""
    n = np.diff(b.tok_off) // b.block
    keep = np.minimum(n, rng.integers(0, n + 2))            # 0..n blocks
    whole = rng.random(n.shape[0]) < 0.25                   # and every block for a quarter of them
    keep[whole] = n[whole]
    lens = keep * b.block
    off = np.zeros(lens.shape[0] + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = np.concatenate([b.tokens[b.tok_off[r]: b.tok_off[r] + lens[r]] for r in range(lens.shape[0])] or
                          [np.zeros(0, np.int32)]).astype(np.int32)
    return Batch(toks, off, b.block, b.descs, b.desc_idx, tag=2)


def _filler(rng, n_keys, block):
    """Chains under a descriptor no request carries, n_keys keys in all."""
    per = 64
    n_req = (n_keys + per - 1) // per
    if n_req <= 0:
        return Batch(np.zeros(0, np.int32), np.zeros(1, np.int64), block, [[(b"model_id", b"filler")]],
                     np.zeros(0, np.int32), tag=3)
    lens = np.full(n_req, per * block, np.int64)
    lens[-1] = (n_keys - per * (n_req - 1)) * block
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = rng.integers(0, 128256, size=int(off[-1]), dtype=np.int64).astype(np.int32)
    return Batch(toks, off, block, [[(b"model_id", b"filler")]], np.zeros(n_req, np.int32), tag=3)


def _fill_both(pkv, capacity, batches):
    """An oracle index and a device index holding every key of the given batches."""
    idx = oracle.Index(capacity, threads=THREADS)
    table = pkv.Table(capacity)
    for fb in batches:
        if fb.n_req == 0:
            continue
        keys, ko = oracle_keys(fb)
        assert idx.store(keys, ko, np.zeros(fb.n_req, np.int32), locations(ko, fb.tag)) == 0
        db = gpu_batch(fb)
        db.digest()
        db.derive()
        db.hits.zero_()
        db.store(table)
        assert db.host_status() == 0
    return idx, table


def _check_fused(pkv, b, idx, table):
    okeys, ko = oracle_keys(b)
    ohits = idx.lookup(okeys, ko)
    db = gpu_batch(b)
    db.hits.fill_(-7)
    db.digest()
    db.derive_lookup(table)
    assert db.host_status() == 0
    assert (db.host_keys() == okeys).all()
    hits = db.host_hits()
    assert (hits == ohits).all(), np.flatnonzero(hits != ohits)[:10]
    return ohits


@pytest.mark.parametrize("n_req", [1, 31, 33, 1000, 8192, 8193, 12000, 16384, 16385])
def test_fused_matches_oracle(pkv, n_req):
    """Every kernel shape: up to 8192 requests one lane-pair pair per workgroup, up to 16384 two,
    beyond that the derive and lookup kernels one after the other; request counts that end inside a
    row or a wavefront; an index at load 0.6 holding random prefixes of the requests."""
    rng = np.random.default_rng(n_req)
    b = _batch(rng, n_req, 40, 16)
    pre = _prefixes(rng, b)
    n_pre = int(np.sum(np.diff(pre.tok_off) // 16))
    capacity = 1 << max(10, int(np.ceil(np.log2((n_pre + 64) / 0.6))))
    fill = _filler(rng, int(0.6 * capacity) - n_pre, 16) if int(0.6 * capacity) > n_pre else None
    announce(f"fused n_req={n_req} capacity={capacity}")
    idx, table = _fill_both(pkv, capacity, [pre] + ([fill] if fill is not None else []))
    ohits = _check_fused(pkv, b, idx, table)
    if n_req >= 1000:                    # misses on the first key, whole chains and partial hits all occur
        n = np.diff(oracle.key_offsets(b.tok_off, 16))
        assert (ohits == 0).any() and ((ohits == n) & (n > 0)).any() and ((ohits > 0) & (ohits < n)).any()


@pytest.mark.parametrize("load", [0.9, 0.97])
def test_fused_at_high_load(pkv, load):
    """Most probes continue into following buckets, so a chain's probes fall behind its keys and
    catch up later; long chains whose keys are all present end with probes still open."""
    rng = np.random.default_rng(int(load * 100))
    b = _batch(rng, 3000, 100, 16)
    pre = _prefixes(rng, b)
    n_pre = int(np.sum(np.diff(pre.tok_off) // 16))
    capacity = 1 << int(np.ceil(np.log2(n_pre / load)))
    fill = _filler(rng, int(load * capacity) - n_pre, 16)
    announce(f"fused load={load} capacity={capacity}")
    idx, table = _fill_both(pkv, capacity, [pre, fill])
    _check_fused(pkv, b, idx, table)


def test_fused_on_a_full_index(pkv):
    """No never-used slot anywhere: a probe for an absent key checks every bucket before it ends."""
    rng = np.random.default_rng(5)
    b = _batch(rng, 40, 6, 16)
    pre = _prefixes(rng, b)
    n_pre = int(np.sum(np.diff(pre.tok_off) // 16))
    capacity = 1 << int(np.ceil(np.log2(n_pre + 1)))
    fill = _filler(rng, capacity - n_pre, 16)
    idx, table = _fill_both(pkv, capacity, [pre, fill])
    assert len(idx) == capacity
    _check_fused(pkv, b, idx, table)


@pytest.mark.parametrize("block", [1, 7, 32, 256])
def test_fused_other_block_sizes(pkv, block):
    """Block sizes without the fused kernel run the derive and lookup kernels: same results."""
    rng = np.random.default_rng(block)
    b = _batch(rng, 300, 12, block)
    pre = _prefixes(rng, b)
    idx, table = _fill_both(pkv, 1 << 14, [pre])
    _check_fused(pkv, b, idx, table)


def test_fused_empty_index_and_empty_requests(pkv):
    """An empty index (every hit 0), requests shorter than one block, and no requests at all."""
    import torch
    rng = np.random.default_rng(9)
    b = _batch(rng, 500, 30, 16)
    idx, table = _fill_both(pkv, 1 << 12, [])
    hits = _check_fused(pkv, b, idx, table)
    assert (hits == 0).all()
    short = Batch(np.arange(15, dtype=np.int32), np.array([0, 5, 5, 15, 15, 15], np.int64), 16, b.descs,
                  np.zeros(5, np.int32))
    _check_fused(pkv, short, idx, table)
    z = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_derive_lookup(z[:0], torch.zeros(1, dtype=torch.int64, device="cuda"),
                          torch.zeros((1, 16), dtype=torch.uint8, device="cuda"), 16,
                          torch.zeros(1, dtype=torch.int64, device="cuda"),
                          torch.zeros((1, 16), dtype=torch.uint8, device="cuda"), table, z, z)
    torch.cuda.synchronize()
    assert int(z.item()) == 0


def test_fused_inconsistent_offsets(pkv):
    """A request whose key offsets disagree with its tokens gets PKV_ELAYOUT, no key and hit 0; the
    other requests are unaffected."""
    rng = np.random.default_rng(11)
    b = _batch(rng, 200, 20, 16)
    pre = _prefixes(rng, b)
    idx, table = _fill_both(pkv, 1 << 13, [pre])
    okeys, ko = oracle_keys(b)
    ohits = idx.lookup(okeys, ko)
    db = gpu_batch(b)
    bad = int(np.flatnonzero(np.diff(ko) > 2)[0])
    koff = db.key_off.clone()
    koff[bad + 1] -= 1                                    # request `bad` one key short, `bad+1` one long
    db.key_off.copy_(koff)
    db.hits.fill_(-7)
    db.digest()
    db.derive_lookup(table)
    assert db.host_status() == pkv.PKV_ELAYOUT
    hits = db.host_hits()
    assert hits[bad] == 0 and hits[bad + 1] == 0
    others = np.setdiff1d(np.arange(b.n_req), [bad, bad + 1])
    assert (hits[others] == ohits[others]).all()


def test_fused_step_c2(pkv):
    """The c2 configuration at full size through the fused step (keys and hits in one call, then the
    store): every key, every hit length and the index after the store equal the oracle's."""
    from tests.test_gpu_parity import _compare_dump
    from tests.gpu_util import check_structure, gpu_fill, oracle_fill
    w = make_workload("c2")
    announce("fused c2: oracle")
    idx = oracle.Index(w.capacity, threads=THREADS)
    oracle_fill(idx, w.fill)
    okeys, ko = oracle_keys(w.batch)
    ohits = idx.lookup(okeys, ko)
    assert idx.store(okeys, ko, ohits, locations(ko, w.batch.tag)) == 0
    announce("fused c2: gpu")
    table = pkv.Table(w.capacity)
    assert gpu_fill(table, w.fill).host_status() == 0
    db = gpu_batch(w.batch)
    db.step_fused(table)
    assert db.host_status() == 0
    assert (db.host_keys() == okeys).all()
    assert (db.host_hits() == ohits).all()
    _compare_dump(table, idx)
    check_structure(table)


def test_fused_through_removed_slots(pkv):
    """An index whose eviction left removed slots on probe paths (the fixed-budget tier): the fused
    probes run through them as the lookup does, and give the oracle's hit lengths."""
    import torch
    from tests.test_gpu_pipeline import _batches
    cap, budget = 1024, 300
    table = pkv.Table(cap, epochs=True)
    idx = oracle.Index(cap)
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")
    batches = _batches(10, seed=77, n_req=20)
    for epoch, b in enumerate(batches[:8], start=1):
        db = gpu_batch(b)
        db.digest()
        db.derive()
        db.n_new.zero_()
        pkv.pkv_lookup_prefix_touch(table, db.keys, db.key_off, epoch, db.hits[: max(1, db.n_req)], db.status)
        pkv.pkv_store_touch(table, db.keys, db.key_off, db.hits[: max(1, db.n_req)], db.locs, db.n_new, db.status,
                            epoch, db.new_slots)
        k, ko = oracle_keys(b)
        hits = idx.lookup_touch(k, ko, epoch)
        assert idx.store_touch(k, ko, hits, locations(ko, b.tag), epoch) == 0
        pkv.pkv_table_evict(table, budget, n_ev)
        assert int(n_ev.item()) == idx.evict(budget)
        assert db.host_status() == 0
    from tests.gpu_util import TOMB, raw_table
    assert (raw_table(table)[1] == TOMB).sum() > 0           # removed slots exist
    for b in batches:                                        # evicted, kept and never stored prefixes
        ohits = _check_fused(pkv, b, idx, table)
        assert ohits.shape[0] == b.n_req
