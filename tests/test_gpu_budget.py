"""The fixed-budget tier on the GPU (section 6.5: eviction under a fixed budget), through the C ABI:
touching lookups and stores and generational eviction must match the oracle step by step (hit
lengths, the number removed, and every entry's key, location and epoch), probe paths must run
through removed slots, stores must reuse them, and a rollback must restore them."""

import numpy as np
import pytest

import oracle
from tests.gpu_util import EMPTY, TOMB, announce, check_structure, gpu_available, gpu_batch, oracle_keys, raw_table
from tests.test_gpu_pipeline import _batches
from workloads import locations

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def raw_entries(table):
    """(keys, locs, epochs) of every entry, sorted by key."""
    keys, locs = raw_table(table)
    ep = table.epochs.cpu().numpy().view(np.uint32)
    live = (locs != EMPTY) & (locs != TOMB)
    k, l, e = [keys[live]], [locs[live]], [ep[live]]
    k, l, e = np.concatenate(k), np.concatenate(l), np.concatenate(e)
    if k.shape[0] == 0:
        return k.reshape(0, 16), l, e
    w = np.ascontiguousarray(k).view(">u8").reshape(-1, 2)
    o = np.lexsort((w[:, 1], w[:, 0]))
    return k[o], l[o], e[o]


def _touch_step(pkv, table, db, epoch):
    db.n_new.zero_()
    pkv.pkv_lookup_prefix_touch(table, db.keys, db.key_off, epoch, db.hits[: max(1, db.n_req)], db.status)
    pkv.pkv_store_touch(table, db.keys, db.key_off, db.hits[: max(1, db.n_req)], db.locs, db.n_new, db.status,
                        epoch, db.new_slots)


def test_budget_sequence_matches_oracle(pkv):
    import torch
    announce("budget tier: 8 epochs, 1024 slots, budget 300")
    cap, budget = 1024, 300
    table = pkv.Table(cap, epochs=True)
    idx = oracle.Index(cap)
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")
    evicted_total = 0
    for epoch, b in enumerate(_batches(8, seed=51, n_req=20), start=1):
        db = gpu_batch(b)
        db.digest()
        db.derive()
        _touch_step(pkv, table, db, epoch)
        k, ko = oracle_keys(b)
        want_hits = idx.lookup_touch(k, ko, epoch)
        assert idx.store_touch(k, ko, want_hits, locations(ko, b.tag), epoch) == 0
        assert db.host_status() == 0
        assert (db.host_hits() == want_hits).all(), epoch
        pkv.pkv_table_evict(table, budget, n_ev)
        want_ev = idx.evict(budget)
        assert int(n_ev.item()) == want_ev, epoch
        evicted_total += want_ev
        gk, gl, ge = raw_entries(table)
        ok, ol = idx.dump()
        assert (gk == ok).all() and (gl == ol).all(), epoch
        assert (ge == idx.dump_epochs()).all(), epoch
        assert check_structure(table) == len(idx) <= budget
    assert evicted_total > 0
    keys, locs = raw_table(table)
    assert (locs[:cap] == TOMB).sum() > 0          # removed slots exist and paths run through them


def test_rollback_restores_removed_slots(pkv):
    import torch
    cap = 256
    table = pkv.Table(cap, epochs=True)
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")
    bs = _batches(3, seed=52, n_req=12)
    for epoch, b in enumerate(bs[:2], start=1):
        db = gpu_batch(b)
        db.digest()
        db.derive()
        _touch_step(pkv, table, db, epoch)
    pkv.pkv_table_evict(table, 40, n_ev)
    assert int(n_ev.item()) > 0
    before = [x.copy() for x in raw_table(table)]
    db = gpu_batch(bs[2])
    db.digest()
    db.derive()
    _touch_step(pkv, table, db, 3)
    assert db.host_status() == 0
    log = db.new_slots[: int(db.n_new.item())].cpu().numpy().view(np.uint64)
    assert (log >> np.uint64(63)).any()             # some new entries reused removed slots
    db.rollback(table)
    after = raw_table(table)
    assert (before[0] == after[0]).all() and (before[1] == after[1]).all()
    check_structure(table)


def test_marker_keys_and_wide_epochs(pkv):
    """Keys whose bytes equal the slot markers (all 0xFF; all 0xFF ending in 0xFE; first halves equal
    to the claim markers) are ordinary entries: stored, touched and evicted like any other."""
    import torch
    cap = 64
    table = pkv.Table(cap, epochs=True)
    idx = oracle.Index(cap)
    rng = np.random.default_rng(53)
    keys = rng.integers(0, 256, size=(10, 16), dtype=np.uint8)
    keys[3] = 0xFF
    keys[7] = 0xFF
    keys[7, 15] = 0xFE
    # first 8 bytes equal to the never-used and removed claim markers and to the substitute word
    keys[1, :8] = 0xFF
    keys[5, :8] = 0xFF
    keys[5, 0] = 0xFE
    keys[8, :8] = 0xFF
    keys[8, 0] = 0xFD
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")
    # one key per call, epochs that differ in both 16-bit digits
    epochs = [5, 70000, 70001, 3 * 65536 + 9, 65535, 65536, 2, 1 << 31, (1 << 32) - 1, 131072]
    for i, e in enumerate(epochs):
        kd = torch.from_numpy(keys[i:i + 1].copy()).cuda()
        ko = torch.tensor([0, 1], dtype=torch.int64, device="cuda")
        hits = torch.zeros(1, dtype=torch.int32, device="cuda")
        locs = torch.tensor([i], dtype=torch.int64, device="cuda")
        pkv.pkv_store_touch(table, kd, ko, hits, locs, n_new, status, e)
        idx.store_touch(keys[i:i + 1], np.array([0, 1], np.int64), np.zeros(1, np.int32), np.array([i], np.uint64), e)
    assert int(status.item()) == 0 and int(n_new.item()) == 10
    kd = torch.from_numpy(keys.copy()).cuda()
    ko = torch.tensor([0, 10], dtype=torch.int64, device="cuda")
    hits = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_lookup_prefix(table, kd, ko, hits, status)
    assert int(hits.item()) == 10
    for budget in (9, 6, 4, 1, 0):
        pkv.pkv_table_evict(table, budget, n_ev)
        assert int(n_ev.item()) == idx.evict(budget), budget
        gk, gl, ge = raw_entries(table)
        ok, ol = idx.dump()
        assert (gk == ok).all() and (gl == ol).all() and (ge == idx.dump_epochs()).all(), budget
        assert check_structure(table) == len(idx)
    assert len(idx) == 0


def test_store_without_never_used_slots_reuses_removed_ones(pkv):
    """A table whose slots are all live or removed (none never used): a new key's scan runs a whole
    cycle of its path without meeting a free slot and then claims the first removed slot on it; a
    lookup of an absent key ends after one cycle; a batch beyond the capacity reports EFULL."""
    import torch
    announce("budget tier: store into a table with no never-used slot")
    cap = 64
    table = pkv.Table(cap, epochs=True)
    idx = oracle.Index(cap)
    rng = np.random.default_rng(54)
    keys = rng.integers(0, 256, size=(cap + 20, 16), dtype=np.uint8)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_new = torch.zeros(1, dtype=torch.int64, device="cuda")
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")

    def store(lo, hi, epoch):
        kk = keys[lo:hi]
        ko = np.array([0, hi - lo], np.int64)
        locs = np.arange(lo, hi, dtype=np.uint64)
        pkv.pkv_store_touch(table, torch.from_numpy(kk.copy()).cuda(), torch.from_numpy(ko).cuda(),
                            torch.zeros(1, dtype=torch.int32, device="cuda"),
                            torch.from_numpy(locs.view(np.int64)).cuda(), n_new, status, epoch)
        return idx.store_touch(kk, ko, np.zeros(1, np.int32), locs, epoch)

    def same():
        gk, gl, ge = raw_entries(table)
        ok, ol = idx.dump()
        assert (gk == ok).all() and (gl == ol).all() and (ge == idx.dump_epochs()).all()
        assert check_structure(table) == len(idx)

    assert store(0, 16, 1) == 0 and store(16, cap, 2) == 0       # every slot taken
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    same()
    pkv.pkv_table_evict(table, cap - 16, n_ev)                    # the 16 entries of epoch 1 removed
    assert int(n_ev.item()) == idx.evict(cap - 16) == 16
    keys_now, locs_now = raw_table(table)
    assert (locs_now[:cap] == EMPTY).sum() == 0 and (locs_now[:cap] == TOMB).sum() == 16
    same()
    assert store(cap, cap + 10, 3) == 0                           # 10 new keys into removed slots
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    same()
    # a lookup of stored keys followed by an absent one (its path has no never-used slot)
    both = np.concatenate([keys[16:20], keys[cap + 19:cap + 20]])
    hits = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_lookup_prefix(table, torch.from_numpy(both.copy()).cuda(),
                          torch.tensor([0, 5], dtype=torch.int64, device="cuda"), hits, status)
    torch.cuda.synchronize()
    assert int(hits.item()) == 4 and int(status.item()) == 0
    # 7 more new keys with 6 removed slots left: beyond the capacity
    assert store(cap + 10, cap + 17, 4) == pkv.PKV_EFULL
    torch.cuda.synchronize()
    assert int(status.item()) == pkv.PKV_EFULL
