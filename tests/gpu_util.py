"""Shared helpers of the GPU parity tests: run a workload through the oracle and through the HIP
path, and inspect raw index arrays."""

from __future__ import annotations

import os

import numpy as np

import oracle
from workloads import locations

THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def announce(msg: str):
    print(f"[gpu-test] {msg}", flush=True)


# ---- oracle side --------------------------------------------------------------------------------

def oracle_keys(batch):
    ko = oracle.key_offsets(batch.tok_off, batch.block)
    keys = oracle.derive(batch.tokens, batch.tok_off, oracle.batch_digests(batch), batch.block, THREADS)
    return keys, ko


def oracle_fill(index, batch):
    keys, ko = oracle_keys(batch)
    rc = index.store(keys, ko, np.zeros(batch.n_req, np.int32), locations(ko, batch.tag))
    assert rc == 0, rc
    return keys, ko


# ---- HIP side ----------------------------------------------------------------------------------

def gpu_batch(batch):
    from paper_2609_38706_amd.pipeline import DeviceBatch
    db = DeviceBatch.from_batch(batch)
    db.set_locations(locations(db.key_off.cpu().numpy(), batch.tag))
    return db


def gpu_fill(table, batch):
    db = gpu_batch(batch)
    db.digest()
    db.derive()
    db.hits.zero_()
    db.store(table)
    return db


EMPTY = np.uint64(0xFFFFFFFFFFFFFFFF)
PENDING = np.uint64(0xFFFFFFFFFFFFFFFE)
TOMB = np.uint64(0xFFFFFFFFFFFFFFFD)
TOMB_KEY = np.array([0xFF] * 15 + [0xFE], np.uint8)


LO_EMPTY = np.uint64(0xFFFFFFFFFFFFFFFF)
LO_REMOVED = np.uint64(0xFFFFFFFFFFFFFFFE)
LO_SUB = np.uint64(0xFFFFFFFFFFFFFFFD)


def raw_slots(table):
    """The index's slot records as uint64 [capacity, 4]: claim word, tag, key bytes 8..15, location."""
    cap = table.capacity
    w = table.slots.cpu().numpy().view(np.uint64)
    assert w.shape[0] == cap * 4, "index buffer is not 32 bytes per slot"
    return w.reshape(cap, 4)


def raw_table(table):
    """The index decoded slot by slot (include/pkv.h layout) into (keys uint8 [capacity, 16], locs
    uint64 [capacity]): a never-used slot reads as the all-0xFF key with location EMPTY, a removed
    slot as TOMB_KEY with location TOMB, a claimed but unpublished slot with location PENDING (these
    key values only stand in for free slots here; a live slot may hold any key).  Also checks the
    layout's own invariants (free slots hold no key bytes, tag or location; a tag's flag appears only
    with the substitute claim word)."""
    r = raw_slots(table)
    claim, tag, hi, loc = (np.ascontiguousarray(r[:, i]) for i in range(4))
    flag = tag & np.uint64(3)
    free = (claim == LO_EMPTY) | (claim == LO_REMOVED)
    assert (tag[free] == 0).all() and (hi[free] == EMPTY).all() and (loc[free] == EMPTY).all(), \
        "free slot with contents"
    assert ((flag == 0) | (claim == LO_SUB)).all(), "substitute flag without the substitute claim word"
    assert (flag <= 2).all(), "unknown substitute flag"
    lo = np.where(claim == LO_SUB, np.where(flag == 1, LO_EMPTY, np.where(flag == 2, LO_REMOVED, claim)), claim)
    keys = np.concatenate([lo.view(np.uint8).reshape(-1, 8), hi.view(np.uint8).reshape(-1, 8)], axis=1)
    locs = np.where(loc == EMPTY, PENDING, loc)
    keys[claim == LO_EMPTY] = 0xFF
    locs[claim == LO_EMPTY] = EMPTY
    keys[claim == LO_REMOVED] = TOMB_KEY
    locs[claim == LO_REMOVED] = TOMB
    return keys, locs


def check_structure(table):
    """Index invariants: every live slot lies on its key's probe path (include/pkv.h) with no
    never-used slot before it on the path (removed slots do not break paths); no claimed-but-unpublished or batch-marked slot
    survives a store and every live slot carries the generation of the store that inserted it;
    empty slots hold no key bytes and removed slots the removed placeholder; no key is stored twice.  Returns the number of entries (live slots)."""
    keys, locs = raw_table(table)
    cap = table.capacity
    assert locs.shape[0] == cap
    occ = locs != EMPTY                      # on some probe path: live or removed
    tomb = locs == TOMB
    live = occ & ~tomb
    assert not (locs == PENDING).any(), "pending slot left behind"
    assert not (locs[live] >= np.uint64(1 << 62)).any(), "location outside the caller's range"
    tags = np.ascontiguousarray(raw_slots(table)[:, 1])
    assert ((tags[live] >> np.uint64(2)) != 0).all(), "live slot without the generation of its store"
    assert (keys[~occ] == 0xFF).all(), "empty slot with key bytes"
    assert (keys[tomb] == TOMB_KEY[None, :]).all(), "removed slot without the removed placeholder"
    if live.any():
        claim = np.ascontiguousarray(raw_slots(table)[:, 0])
        lo = keys[:, :8].copy().view("<u8").reshape(-1)
        n_b = cap // 4
        s = np.flatnonzero(live).astype(np.int64)
        home = (lo[s] & np.uint64(n_b - 1)).astype(np.int64)
        rot = (keys[s, 8] & 3).astype(np.int64)            # the path's first slot in each bucket
        b_s, j_s = s // 4, s % 4
        # buckets from the home bucket up to the slot's own: none may hold a never-used slot
        has_empty = (~occ).reshape(n_b, 4).any(axis=1)
        bidx = np.arange(n_b, dtype=np.int64)
        last = np.maximum.accumulate(np.where(has_empty, bidx, -1))     # last such bucket at or before b
        if has_empty.any():
            wrap_last = int(bidx[has_empty][-1]) - n_b
            last = np.where(last < 0, wrap_last, last)
            before = np.where(b_s > 0, last[b_s - 1], wrap_last)          # strictly before b_s, cyclically
            dist_home = (b_s - home) % n_b
            dist_empty = b_s - before
            assert (dist_home < dist_empty).all(), "live slot behind a bucket with a never-used slot"
        # inside its bucket: the slots that come before it on the path are not never-used
        pos = (j_s - rot) & 3
        for i in range(3):
            earlier = b_s * 4 + ((rot + i) & 3)
            bad = (i < pos) & ~occ[earlier]
            assert not bad.any(), "live slot behind a never-used slot of its bucket"
        assert not ((claim == LO_EMPTY) | (claim == LO_REMOVED))[live].any(), "live slot with a free marker"
        w = np.ascontiguousarray(keys[live]).view(">u8").reshape(-1, 2)
        order = np.argsort(w[:, 0])
        first = w[order, 0]
        tie = np.flatnonzero(first[1:] == first[:-1])      # equal keys share their first 8 bytes
        if tie.size:
            sub = w[order[np.unique(np.concatenate([tie, tie + 1]))]]
            sub = sub[np.lexsort((sub[:, 1], sub[:, 0]))]
            assert not ((sub[1:] == sub[:-1]).all(axis=1)).any(), "duplicate key stored"
    return int(live.sum())
