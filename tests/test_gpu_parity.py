"""GPU parity: the HIP path through the C ABI against the oracle, element by element and bit-exact
(keys, hit lengths, index contents), plus error handling and index invariants."""

import numpy as np
import pytest

import oracle
from tests.gpu_util import (THREADS, announce, check_structure, gpu_available, gpu_batch, gpu_fill, oracle_fill,
                            oracle_keys)
from workloads import Batch, locations, make_workload

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()       # the HIP library must be built; no fallback exists
    return m


def _ragged_batch(rng, n_req, max_len, block, n_desc=5, vocab=1 << 31):
    lens = rng.integers(0, max_len + 1, size=n_req)
    lens[rng.integers(0, n_req)] = 0
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = rng.integers(-vocab, vocab, size=int(off[-1]), dtype=np.int64).astype(np.int32)
    descs = [[(b"model_id", b"m%d" % i), (b"salt", rng.bytes(8))] for i in range(n_desc)]
    return Batch(toks, off, block, descs, rng.integers(0, n_desc, size=n_req).astype(np.int32))


# ---- digests and keys ---------------------------------------------------------------------------

def test_digest_batch_matches_oracle(pkv):
    import torch
    rng = np.random.default_rng(0)
    descs = []
    for w in ("tiny", "c3"):
        descs += make_workload(w).batch.descs
    for _ in range(150):   # binary values, odd lengths, descriptors crossing several SHA blocks
        n = int(rng.integers(0, 12))
        descs.append([(b"x%03d" % i, rng.bytes(int(rng.integers(0, 200)))) for i in range(n)])
    idx = np.concatenate([np.arange(len(descs)), rng.integers(0, len(descs), size=60)]).astype(np.int32)
    b = Batch(np.zeros(0, np.int32), np.zeros(idx.shape[0] + 1, np.int64), 16, descs, idx)
    announce(f"digest_batch n={idx.shape[0]}")
    db = gpu_batch(b)
    db.digest()
    got = db.digests[: idx.shape[0]].cpu().numpy()
    torch.cuda.synchronize()
    assert db.host_status() == 0
    assert (got == oracle.batch_digests(b)).all()


def test_expand_digests(pkv):
    """Per-request digests gathered from per-descriptor ones, including an index past the table
    (PKV_ELAYOUT, that request's digest zeroed) and an empty batch."""
    import torch
    rng = np.random.default_rng(2)
    table = rng.integers(0, 256, size=(37, 16), dtype=np.uint8)
    idx = rng.integers(0, 37, size=1000).astype(np.int32)
    d_tab = torch.from_numpy(table).cuda()
    out = torch.full((1000, 16), 7, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_expand_digests(d_tab, torch.from_numpy(idx).cuda(), out, status)
    assert int(status.item()) == 0
    assert (out.cpu().numpy() == table[idx]).all()
    bad = idx.copy()
    bad[500] = 37
    pkv.pkv_expand_digests(d_tab, torch.from_numpy(bad).cuda(), out, status)
    got = out.cpu().numpy()
    assert int(status.item()) == pkv.PKV_ELAYOUT
    assert (got[500] == 0).all() and (np.delete(got, 500, 0) == np.delete(table[idx], 500, 0)).all()
    status.zero_()
    pkv.pkv_expand_digests(d_tab, torch.zeros(0, dtype=torch.int32, device="cuda"), out[:0], status)
    assert int(status.item()) == 0


def test_digest_batch_unaligned_pool(pkv):
    """Messages at odd byte offsets, one ending on the pool's last byte, and empty messages."""
    import torch
    rng = np.random.default_rng(1)
    encs, offs, pool = [], [], b""
    for i in range(70):
        n = int(rng.integers(0, 6))
        desc = [(b"f%d" % j, rng.bytes(int(rng.integers(0, 90)))) for j in range(n)]
        e = oracle.encode(desc)
        pool += rng.bytes(int(rng.integers(1, 4)))          # junk: the next message starts unaligned
        offs.append(len(pool))
        pool += e
        encs.append(e)
    offs.append(len(pool))                                   # an empty message at the very end
    encs.append(b"")
    lens = [len(e) for e in encs]
    d_pool = torch.from_numpy(np.frombuffer(pool, np.uint8).copy()).cuda()
    d_off = torch.tensor(offs, dtype=torch.int64, device="cuda")
    d_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    out = torch.zeros((len(encs), 16), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_digest_batch(d_pool, d_off, d_len, out, status)
    got = out.cpu().numpy()
    assert int(status.item()) == 0
    for i, e in enumerate(encs):
        assert got[i].tobytes() == oracle.sha256(e)[:16]


@pytest.mark.gpu
@pytest.mark.parametrize("shift", [0, 1, 3])
def test_digest_batch_every_length(pkv, shift):
    """Messages of every length 0..200 bytes (every padding case of one to four SHA-256 blocks:
    55/56 and 119/120 bytes put the length in the same or the next block), 4-byte aligned
    (shift 0) or not, in a pool whose last message ends on its last byte; 201 messages span
    several workgroups and leave a partial one."""
    import torch
    rng = np.random.default_rng(100 + shift)
    lens = list(range(201))
    rng.shuffle(lens)
    offs, pool = [], bytearray()
    for n in lens:
        pool += b"\0" * ((-len(pool)) % 4 + shift)            # the message starts `shift` past a word
        offs.append(len(pool))
        pool += rng.bytes(n)
    d_pool = torch.from_numpy(np.frombuffer(bytes(pool), np.uint8).copy()).cuda()
    d_off = torch.tensor(offs, dtype=torch.int64, device="cuda")
    d_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    out = torch.zeros((len(lens), 16), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_digest_batch(d_pool, d_off, d_len, out, status)
    got = out.cpu().numpy()
    assert int(status.item()) == 0
    for i, (o, n) in enumerate(zip(offs, lens)):
        assert got[i].tobytes() == oracle.sha256(bytes(pool[o:o + n]))[:16], (n, shift)


@pytest.mark.parametrize("block", [1, 2, 3, 7, 15, 16, 17, 31, 32, 48, 64, 100, 256, 257])
def test_derive_matches_oracle_any_block(pkv, block):
    rng = np.random.default_rng(block)
    b = _ragged_batch(rng, n_req=131, max_len=min(40 * block, 9000), block=block)
    announce(f"derive block={block} n_req={b.n_req} tokens={b.tokens.shape[0]}")
    db = gpu_batch(b)
    db.digest()
    db.derive()
    got = db.host_keys()
    assert db.host_status() == 0
    want, ko = oracle_keys(b)
    assert (db.key_off.cpu().numpy() == ko).all()
    assert got.shape == want.shape
    assert (got == want).all()


def test_derive_unaligned_token_offsets(pkv):
    rng = np.random.default_rng(5)
    lens = np.array([17, 33, 1, 16, 48, 65, 0, 130, 31], np.int64)   # request starts at odd token offsets
    off = np.concatenate([[0], np.cumsum(lens)])
    toks = rng.integers(0, 100000, size=int(off[-1]), dtype=np.int32)
    for block in (16, 32):
        b = Batch(toks, off, block, [[(b"model_id", b"m")]], np.zeros(lens.shape[0], np.int32))
        db = gpu_batch(b)
        db.digest()
        db.derive()
        want, _ = oracle_keys(b)
        assert (db.host_keys() == want).all()


def test_derive_reports_inconsistent_offsets(pkv):
    import torch
    rng = np.random.default_rng(6)
    b = _ragged_batch(rng, 70, 300, 16)
    db = gpu_batch(b)
    db.digest()
    bad = db.key_off.clone()
    bad[5:] += 1                                           # request 4 claims one key too many
    pkv.pkv_derive_keys(db.tokens, db.tok_off, db.digests, 16, bad, db.keys, db.status)
    torch.cuda.synchronize()
    assert db.host_status() == pkv.PKV_ELAYOUT
    db.status.zero_()
    bad_tok = db.tok_off.clone()
    bad_tok[-1] = db.tokens.numel() + 64                   # past the token buffer
    pkv.pkv_derive_keys(db.tokens, bad_tok, db.digests, 16, db.key_off, db.keys, db.status)
    torch.cuda.synchronize()
    assert db.host_status() == pkv.PKV_ELAYOUT


# ---- lookup and store on arbitrary keys ---------------------------------------------------------

def _key_batch(rng, pool, n_req, max_keys):
    lens = rng.integers(0, max_keys + 1, size=n_req)
    ko = np.zeros(n_req + 1, np.int64)
    ko[1:] = np.cumsum(lens)
    return pool[rng.integers(0, pool.shape[0], size=int(ko[-1]))], ko


def _dev(a, dtype):
    """numpy -> device tensor; uint64 arrays travel as int64 with the same bits."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    if a.size == 0:
        return torch.zeros(1, dtype=dtype, device="cuda")
    return torch.from_numpy(a).to("cuda").view(dtype)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("capacity", [64, 1024])
def test_lookup_and_store_random_keys(pkv, seed, capacity):
    import torch
    from paper_2609_38706_amd.pipeline import export_sorted
    rng = np.random.default_rng(seed)
    pool = rng.integers(0, 256, size=(60, 16), dtype=np.uint8)
    pool[0] = 0xFF                                          # the key equal to the empty marker
    pool[1, :8] = pool[2, :8]                               # same home bucket, different key
    idx = oracle.Index(capacity)
    table = pkv.Table(capacity)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
    for rnd in range(3):
        n_req = int(rng.integers(1, 90))
        keys, ko = _key_batch(rng, pool, n_req, 12)
        locs = rng.permutation(1 << 20)[: keys.shape[0]].astype(np.uint64) + np.uint64(rnd << 40)
        hits_o = idx.lookup(keys, ko)
        dk, dko = _dev(keys, torch.uint8).reshape(-1, 16), _dev(ko, torch.int64)
        hits = torch.zeros(max(1, n_req), dtype=torch.int32, device="cuda")
        pkv.pkv_lookup_prefix(table, dk, dko, hits[:n_req], status)
        assert (hits[:n_req].cpu().numpy() == hits_o).all(), (rnd, hits[:n_req].cpu().numpy(), hits_o)
        # store from the lookup result, or (last round) from arbitrary hit counts, which may exceed
        # the lookup's: keys below the given count are never inserted
        h = rng.integers(0, 14, size=n_req).astype(np.int32) if rnd == 2 else hits_o
        rc = idx.store(keys, ko, h, locs)
        pkv.pkv_store(table, dk, dko, _dev(h, torch.int32), _dev(locs, torch.int64), n_new, status)
        torch.cuda.synchronize()
        assert rc == 0 and int(status.item()) == 0
        gk, gl = export_sorted(table)
        ok, ol = idx.dump()
        assert gk.shape == ok.shape and (gk == ok).all() and (gl == ol).all()
        assert check_structure(table) == len(idx)


@pytest.mark.parametrize("shape", ["long-first", "long-last", "long-middle", "alternating", "many-empty"])
def test_store_with_skewed_request_lengths(pkv, shape):
    """Each store wavefront finds the request of its first key from a guess that assumes equal
    lengths and widens from there (up or down); very unequal lengths and runs of empty requests
    must give the same index as the oracle."""
    import torch
    from paper_2609_38706_amd.pipeline import export_sorted
    rng = np.random.default_rng(7 + len(shape))
    n_req = 700
    lens = np.zeros(n_req, np.int64)
    if shape == "long-first":
        lens[0] = 3000
        lens[1:] = rng.integers(0, 3, size=n_req - 1)
    elif shape == "long-last":
        lens[:-1] = rng.integers(0, 3, size=n_req - 1)
        lens[-1] = 3000
    elif shape == "long-middle":
        lens[:] = rng.integers(0, 2, size=n_req)
        lens[350] = 2500
        lens[351:360] = 0
    elif shape == "alternating":
        lens[::2] = 0
        lens[1::2] = rng.integers(1, 12, size=n_req // 2)
    else:
        lens[rng.permutation(n_req)[:20]] = rng.integers(60, 200, size=20)
    ko = np.zeros(n_req + 1, np.int64)
    ko[1:] = np.cumsum(lens)
    n_keys = int(ko[-1])
    keys = rng.integers(0, 256, size=(n_keys, 16), dtype=np.uint8)
    keys[: n_keys // 3] = keys[n_keys // 3: 2 * (n_keys // 3)]       # duplicates across requests
    locs = rng.permutation(1 << 22)[:n_keys].astype(np.uint64)
    h = np.minimum(rng.integers(0, 4, size=n_req), lens).astype(np.int32)
    capacity = 1 << 14
    idx = oracle.Index(capacity)
    table = pkv.Table(capacity)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
    rc = idx.store(keys, ko, h, locs)
    pkv.pkv_store(table, _dev(keys, torch.uint8).reshape(-1, 16), _dev(ko, torch.int64), _dev(h, torch.int32),
                  _dev(locs, torch.int64), n_new, status)
    torch.cuda.synchronize()
    assert rc == 0 and int(status.item()) == 0
    gk, gl = export_sorted(table)
    ok, ol = idx.dump()
    assert gk.shape == ok.shape and (gk == ok).all() and (gl == ol).all()
    assert int(n_new.item()) == len(idx)


@pytest.mark.parametrize("seed", range(3))
def test_earlier_entries_keep_their_location(pkv, seed):
    """Each store call lowers only the locations of the entries it inserts itself: rounds whose
    locations are smaller than every earlier round's, over keys that repeat within a batch and across
    batches (marker-like keys included), give the oracle's index after every round (section 3.4:
    an entry already present is never replaced; the smallest location of a batch wins)."""
    import torch
    from paper_2609_38706_amd.pipeline import export_sorted
    rng = np.random.default_rng(700 + seed)
    pool = np.concatenate([_marker_prefixed_pool(rng), rng.integers(0, 256, size=(30, 16), dtype=np.uint8)])
    capacity = 256
    idx = oracle.Index(capacity)
    table = pkv.Table(capacity)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for rnd in range(4):
        n_req = int(rng.integers(20, 60))
        keys, ko = _key_batch(rng, pool, n_req, 6)
        locs = rng.permutation(1 << 16)[: keys.shape[0]].astype(np.uint64) + np.uint64((3 - rnd) << 40)
        zero = np.zeros(n_req, np.int32)
        assert idx.store(keys, ko, zero, locs) == 0
        n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
        pkv.pkv_store(table, _dev(keys, torch.uint8).reshape(-1, 16), _dev(ko, torch.int64), _dev(zero, torch.int32),
                      _dev(locs, torch.int64), n_new, status)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        gk, gl = export_sorted(table)
        ok, ol = idx.dump()
        assert gk.shape == ok.shape and (gk == ok).all() and (gl == ol).all(), rnd
        assert check_structure(table) == len(idx)


def _marker_prefixed_pool(rng):
    """Keys whose first 8 bytes (the slot claim word, little-endian) equal the never-used marker
    (all 0xFF), the removed marker (0xFE then 0xFF) or the substitute claim word (0xFD then 0xFF),
    with random and all-ones second halves; the all-0xFF key and the all-0xFF key ending in 0xFE
    (whose second halves also equal a free slot's key bytes); ordinary keys.  The first three
    prefixes all map to the last buckets, so they also contend and wrap around."""
    pool = []
    for first in (0xFF, 0xFE, 0xFD):
        for hi in range(6):
            k = np.full(16, 0xFF, np.uint8)
            k[0] = first
            if hi < 4:
                k[8:] = rng.integers(0, 256, size=8, dtype=np.uint8)
            elif hi == 5:
                k[8] = 0xFE                                 # one byte off all ones
            pool.append(k)
    pool.append(np.full(16, 0xFF, np.uint8))                # all 0xFF
    tomb = np.full(16, 0xFF, np.uint8)
    tomb[15] = 0xFE
    pool.append(tomb)                                       # all 0xFF but the last byte
    pool.extend(rng.integers(0, 256, size=(10, 16), dtype=np.uint8))
    return np.stack(pool)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("capacity", [32, 256])
def test_marker_prefixed_keys(pkv, seed, capacity):
    """Claim-word edge cases: keys that claim with the substitute word keep their own identity
    (their tags' flags), equal keys still merge, lookups find exactly the stored ones, and a rollback
    restores the index."""
    import torch
    from paper_2609_38706_amd.pipeline import export_sorted
    rng = np.random.default_rng(100 + seed)
    pool = _marker_prefixed_pool(rng)
    idx = oracle.Index(capacity)
    table = pkv.Table(capacity)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for rnd in range(3):
        n_req = int(rng.integers(1, 60))
        keys, ko = _key_batch(rng, pool, n_req, 8)
        locs = rng.permutation(1 << 16)[: keys.shape[0]].astype(np.uint64) + np.uint64(rnd << 40)
        hits_o = idx.lookup(keys, ko)
        dk, dko = _dev(keys, torch.uint8).reshape(-1, 16), _dev(ko, torch.int64)
        hits = torch.zeros(max(1, n_req), dtype=torch.int32, device="cuda")
        pkv.pkv_lookup_prefix(table, dk, dko, hits[:n_req], status)
        assert (hits[:n_req].cpu().numpy() == hits_o).all(), (rnd, hits[:n_req].cpu().numpy(), hits_o)
        before = export_sorted(table)
        n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
        slots = torch.empty(max(1, keys.shape[0]), dtype=torch.int64, device="cuda")
        rc = idx.store(keys, ko, hits_o, locs)
        pkv.pkv_store(table, dk, dko, hits[:n_req], _dev(locs, torch.int64), n_new, status, slots)
        torch.cuda.synchronize()
        assert rc == 0 and int(status.item()) == 0
        gk, gl = export_sorted(table)
        ok, ol = idx.dump()
        assert gk.shape == ok.shape and (gk == ok).all() and (gl == ol).all()
        assert check_structure(table) == len(idx)
        if rnd == 1:                                        # undo this round on both sides
            pkv.pkv_table_rollback(table, slots, n_new)
            after = export_sorted(table)
            assert (after[0] == before[0]).all() and (after[1] == before[1]).all()
            check_structure(table)
            idx = oracle.Index(capacity)
            if before[0].shape[0]:
                assert idx.store(before[0], np.array([0, before[0].shape[0]], np.int64), np.zeros(1, np.int32),
                                 before[1]) == 0


def test_duplicate_heavy_store_is_deterministic(pkv):
    """Every request carries the same key chain: maximal contention on one set of slots.  The index
    must equal the oracle's whatever the request order and however the lanes race."""
    import torch
    from paper_2609_38706_amd.pipeline import export_sorted
    rng = np.random.default_rng(21)
    chain = rng.integers(0, 256, size=(40, 16), dtype=np.uint8)
    n_req = 700
    keys = np.tile(chain, (n_req, 1))
    ko = np.arange(n_req + 1, dtype=np.int64) * 40
    ref = None
    for trial in range(3):
        perm = rng.permutation(n_req * 40)
        locs = perm.astype(np.uint64) + np.uint64(7)
        idx = oracle.Index(256)
        assert idx.store(keys, ko, np.zeros(n_req, np.int32), locs) == 0
        table = pkv.Table(256)
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
        pkv.pkv_store(table, _dev(keys, torch.uint8).reshape(-1, 16), _dev(ko, torch.int64),
                      torch.zeros(n_req, dtype=torch.int32, device="cuda"), _dev(locs, torch.int64), n_new, status)
        gk, gl = export_sorted(table)
        assert int(status.item()) == 0 and int(n_new.item()) == 40
        ok, ol = idx.dump()
        assert (gk == ok).all() and (gl == ol).all()
        check_structure(table)
        if ref is None:
            ref = gk
        assert (gk == ref).all()


def test_full_index_reports_efull(pkv):
    import torch
    rng = np.random.default_rng(8)
    keys = rng.integers(0, 256, size=(65, 16), dtype=np.uint8)
    ko = np.array([0, 64], np.int64)
    for n, expect in ((64, 0), (65, pkv.PKV_EFULL)):
        idx = oracle.Index(64)
        kk = keys[:n]
        k_o = np.array([0, n], np.int64)
        rc = idx.store(kk, k_o, np.zeros(1, np.int32), np.arange(n, dtype=np.uint64))
        table = pkv.Table(64)
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
        pkv.pkv_store(table, _dev(kk, torch.uint8).reshape(-1, 16), _dev(k_o, torch.int64),
                      torch.zeros(1, dtype=torch.int32, device="cuda"),
                      _dev(np.arange(n, dtype=np.uint64), torch.int64), n_new, status)
        torch.cuda.synchronize()
        assert rc == expect and int(status.item()) == expect
        if expect == 0:
            # a full index still answers lookups (the probe path ends after one full turn)
            hits = torch.zeros(2, dtype=torch.int32, device="cuda")
            other = rng.integers(0, 256, size=(1, 16), dtype=np.uint8)
            both = np.concatenate([kk, other])
            pkv.pkv_lookup_prefix(table, _dev(both, torch.uint8).reshape(-1, 16),
                                  _dev(np.array([0, 64, 65], np.int64), torch.int64), hits, status)
            assert hits.cpu().tolist() == [64, 0]
    del ko


def test_reserved_location_reported(pkv):
    import torch
    keys = np.arange(32, dtype=np.uint8).reshape(2, 16)
    table = pkv.Table(64)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
    pkv.pkv_store(table, _dev(keys, torch.uint8).reshape(-1, 16), _dev(np.array([0, 2], np.int64), torch.int64),
                  torch.zeros(1, dtype=torch.int32, device="cuda"),
                  _dev(np.array([5, 1 << 62], np.uint64), torch.int64), n_new, status)
    torch.cuda.synchronize()
    assert int(status.item()) == pkv.PKV_ERESERVED


def test_lookup_reports_inconsistent_offsets(pkv):
    import torch
    table = pkv.Table(64)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    keys = torch.zeros((4, 16), dtype=torch.uint8, device="cuda")
    hits = torch.full((2,), 7, dtype=torch.int32, device="cuda")
    pkv.pkv_lookup_prefix(table, keys, _dev(np.array([0, 2, 9], np.int64), torch.int64), hits, status)
    torch.cuda.synchronize()
    assert int(status.item()) == pkv.PKV_ELAYOUT
    assert hits.cpu().tolist() == [0, 0]


def test_rollback_restores_the_index(pkv):
    from paper_2609_38706_amd.pipeline import export_sorted
    w = make_workload("tiny")
    table = pkv.Table(w.capacity)
    gpu_fill(table, w.fill)
    before = export_sorted(table)
    db = gpu_batch(w.batch)
    db.step(table)
    mid = export_sorted(table)
    assert mid[0].shape[0] == 128 and int(db.n_new.item()) == 64
    db.rollback(table)
    after = export_sorted(table)
    assert (before[0] == after[0]).all() and (before[1] == after[1]).all()
    check_structure(table)


def test_store_without_slot_log_matches(pkv):
    from paper_2609_38706_amd.pipeline import export_sorted
    w = make_workload("tiny")
    t1, t2 = pkv.Table(w.capacity), pkv.Table(w.capacity)
    for t, log in ((t1, True), (t2, False)):
        db = gpu_batch(w.batch)
        db.digest(); db.derive(); db.lookup(t); db.store(t, log=log)
    a, b = export_sorted(t1), export_sorted(t2)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()


# ---- the five workloads ---------------------------------------------------------------------------

def _compare_dump(table, index):
    from paper_2609_38706_amd.pipeline import export_sorted
    gk, gl = export_sorted(table)
    ok, ol = index.dump()
    assert gk.shape == ok.shape, (gk.shape, ok.shape)
    assert (gk == ok).all() and (gl == ol).all()


def test_workload_tiny(pkv):
    w = make_workload("tiny")
    announce("workload tiny")
    idx = oracle.Index(w.capacity)
    oracle_fill(idx, w.fill)
    okeys, ko = oracle_keys(w.batch)
    ohits = idx.lookup(okeys, ko)
    table = pkv.Table(w.capacity)
    gpu_fill(table, w.fill)
    db = gpu_batch(w.batch)
    db.step(table)
    assert (db.host_keys() == okeys).all()
    assert (db.host_hits() == ohits).all() and ohits.tolist() == w.meta["expect_first"]
    idx.store(okeys, ko, ohits, locations(ko, w.batch.tag))
    _compare_dump(table, idx)
    db.lookup(table)
    assert db.host_hits().tolist() == w.meta["expect_second"]
    assert db.host_status() == 0
    check_structure(table)


@pytest.mark.slow
def test_workload_c2(pkv):
    w = make_workload("c2")
    announce("workload c2: oracle")
    idx = oracle.Index(w.capacity, threads=THREADS)
    oracle_fill(idx, w.fill)
    assert len(idx) == w.meta["fill_entries"]
    okeys, ko = oracle_keys(w.batch)
    ohits = idx.lookup(okeys, ko)
    announce("workload c2: gpu")
    table = pkv.Table(w.capacity)
    fill = gpu_fill(table, w.fill)
    assert fill.host_status() == 0
    db = gpu_batch(w.batch)
    db.step(table)
    assert (db.host_keys() == okeys).all()
    hits = db.host_hits()
    assert (hits == ohits).all()
    m = w.batch.meta
    assert (hits == np.where(m["bf16"], m["prefix_len"] // 16, 0)).all()
    assert idx.store(okeys, ko, ohits, locations(ko, w.batch.tag)) == 0
    announce("workload c2: dump")
    _compare_dump(table, idx)
    assert db.host_status() == 0
    assert check_structure(table) == len(idx)


@pytest.mark.slow
def test_workload_c3(pkv):
    w = make_workload("c3")
    announce("workload c3: oracle")
    idx = oracle.Index(w.capacity)
    wkeys, wko = oracle_keys(w.warmup)
    assert idx.store(wkeys, wko, idx.lookup(wkeys, wko), locations(wko, w.warmup.tag)) == 0
    okeys, ko = oracle_keys(w.batch)
    ohits = idx.lookup(okeys, ko)
    assert idx.store(okeys, ko, ohits, locations(ko, w.batch.tag)) == 0
    announce("workload c3: gpu")
    table = pkv.Table(w.capacity)
    warm = gpu_batch(w.warmup)
    warm.step(table)
    db = gpu_batch(w.batch)
    db.step(table)
    assert (warm.host_keys() == wkeys).all()
    assert (db.host_keys() == okeys).all()
    assert (db.host_hits() == ohits).all()
    # closed form: a request hits its prefix's full chunks iff the warm-up stored that
    # (prefix, descriptor) pair
    pairs = set(zip(w.warmup.meta["prefix_id"].tolist(), w.warmup.desc_idx.tolist()))
    expect = [(pl // 256) if (p, d) in pairs else 0 for p, d, pl in
              zip(w.batch.meta["prefix_id"].tolist(), w.batch.desc_idx.tolist(), w.batch.meta["prefix_len"].tolist())]
    assert db.host_hits().tolist() == expect
    _compare_dump(table, idx)
    assert warm.host_status() == 0 and db.host_status() == 0
    check_structure(table)


@pytest.mark.slow
def test_workload_c5(pkv):
    w = make_workload("c5")
    announce("workload c5: gpu")
    table = pkv.Table(w.capacity)
    db = gpu_batch(w.batch)
    db.step(table)
    hits1 = db.host_hits()
    db.lookup(table)
    hits2 = db.host_hits()
    gkeys = db.host_keys()
    assert db.host_status() == 0
    assert hits1.tolist() == w.meta["expect_first"]
    assert hits2.tolist() == w.meta["expect_second"]
    announce("workload c5: oracle")
    okeys, ko = oracle_keys(w.batch)
    assert (gkeys == okeys).all()
    idx = oracle.Index(w.capacity)
    assert idx.store(okeys, ko, np.zeros(w.batch.n_req, np.int32), locations(ko, w.batch.tag)) == 0
    _compare_dump(table, idx)
    check_structure(table)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_workload_c4(pkv):
    """Full-size lookup-heavy run: a 2^25-entry fill of a 2^26-slot index, then 16384 x 256 probe keys
    derived, looked up and stored.  Every key, every hit length and the whole index after the store
    (sorted (key, location) pairs and their count) equal the oracle's, and so do the keys and hit
    lengths of the fused derive-and-lookup call on the same index; the hit lengths also follow
    the recipe's closed form (the stored prefix under a matching descriptor, 0 under a descriptor
    that differs in one dimension)."""
    w = make_workload("c4")
    announce("workload c4: gpu fill (2^25 keys) and probe step")
    table = pkv.Table(w.capacity)
    fill = gpu_fill(table, w.fill)
    assert fill.host_status() == 0
    assert int(fill.n_new.item()) == w.meta["fill_entries"]
    del fill
    db = gpu_batch(w.batch)
    db.digest()
    db.derive_lookup(table)                                  # keys and hits in one call, as well
    fkeys, fhits = db.host_keys(), db.host_hits()
    db.step(table)
    gkeys, hits = db.host_keys(), db.host_hits()
    assert db.host_status() == 0
    m = w.batch.meta
    assert (hits == np.where(m["own"], m["stored_blocks"], 0)).all()
    announce("workload c4: oracle fill, derive, lookup, store")
    idx = oracle.Index(w.capacity, threads=THREADS)
    oracle_fill(idx, w.fill)
    assert len(idx) == w.meta["fill_entries"]
    okeys, ko = oracle_keys(w.batch)
    assert (gkeys == okeys).all() and (fkeys == okeys).all()
    del gkeys, fkeys
    ohits = idx.lookup(okeys, ko)
    assert (hits == ohits).all() and (fhits == ohits).all()
    assert idx.store(okeys, ko, ohits, locations(ko, w.batch.tag)) == 0
    assert int(db.n_new.item()) == len(idx) - w.meta["fill_entries"]
    announce("workload c4: index dump")
    _compare_dump(table, idx)
    assert check_structure(table) == len(idx)


@pytest.mark.gpu
def test_key_offsets_long_requests_and_block_sizes(pkv):
    """Lengths beyond 2^32 tokens and block sizes that are and are not powers of two give the oracle's
    floor(len / B) sums (only the offsets are read, so no tokens are allocated)."""
    import torch
    rng = np.random.default_rng(44)
    n_req = 3000
    lens = rng.integers(0, 1 << 12, size=n_req)
    big = rng.random(n_req) < 0.1
    lens[big] = rng.integers(1 << 31, 1 << 40, size=int(big.sum()))
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    for block in (1, 2, 7, 16, 1000, 1 << 20, 3000000019, 0xFFFFFFFF):
        tok_off = torch.from_numpy(off).cuda()
        key_off = torch.full((n_req + 1,), -5, dtype=torch.int64, device="cuda")
        pkv.pkv_key_offsets(tok_off, block, key_off)
        assert (key_off.cpu().numpy() == oracle.key_offsets(off, block)).all(), block


@pytest.mark.parametrize("n_req", [1, 8192, 16383, 16384, 16385, 3 * 16384 + 5, 100000])
def test_key_offsets_across_scan_chunks(pkv, n_req):
    """The key-offset scan works in chunks of 16384 requests; sizes around and across chunk ends must
    give the oracle's prefix sums of floor(len / B)."""
    import torch
    rng = np.random.default_rng(n_req)
    lens = rng.integers(0, 80, size=n_req)
    lens[rng.random(n_req) < 0.2] = 0
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    for block in (16, 7):
        tok_off = torch.from_numpy(off).cuda()
        key_off = torch.full((n_req + 1,), -5, dtype=torch.int64, device="cuda")
        pkv.pkv_key_offsets(tok_off, block, key_off)
        assert (key_off.cpu().numpy() == oracle.key_offsets(off, block)).all(), block
