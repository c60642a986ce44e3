"""Device-resident request batches and the hot-path step built on the C ABI.

``DeviceBatch`` marshals one batch onto the GPU once:
  * tokens and request offsets;
  * a pool of the canonical encodings of the batch's distinct descriptors, with their offsets and
    lengths, and each request's descriptor index.
It also preallocates every output.  One step then launches only library kernels:
  key offsets -> descriptor digests (one per distinct descriptor, then expanded per request) ->
  chained keys -> longest-prefix lookup -> store of misses.
"""

from __future__ import annotations

import numpy as np

from . import (Table, pkv_derive_keys, pkv_derive_lookup, pkv_descriptor_encode, pkv_digest_batch, pkv_expand_digests,
               pkv_key_offsets, pkv_lookup_prefix, pkv_store, pkv_table_export, pkv_table_rollback)


class DeviceBatch:
    def __init__(self, tokens: np.ndarray, tok_off: np.ndarray, block: int, descs, desc_idx: np.ndarray,
                 device: str = "cuda"):
        import torch
        self.block = int(block)
        self.n_req = int(tok_off.shape[0] - 1)
        self.device = device
        if isinstance(tokens, torch.Tensor):             # already on the device: used as is
            if tokens.dtype != torch.int32 or not tokens.is_contiguous() or not tokens.is_cuda:
                raise ValueError("device tokens must be a contiguous int32 GPU tensor")
            self.tokens = tokens
        else:
            self.tokens = torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).to(device)
        if self.tokens.numel() == 0:
            self.tokens = torch.zeros(1, dtype=torch.int32, device=device)[:0]
        self.tok_off = torch.from_numpy(np.ascontiguousarray(tok_off, dtype=np.int64)).to(device)
        encs = [pkv_descriptor_encode(d) for d in descs]
        lens = np.array([len(e) for e in encs], dtype=np.int64)
        # each encoding starts on a 4-byte boundary, so the digest kernel reads whole words
        padded = [e + b"\0" * (-len(e) % 4) for e in encs]
        offs = np.zeros(len(encs), dtype=np.int64)
        if len(encs) > 1:
            offs[1:] = np.cumsum([len(e) for e in padded])[:-1]
        pool = np.frombuffer(b"".join(padded) or b"\0", dtype=np.uint8)
        didx = np.asarray(desc_idx, dtype=np.int64)
        if didx.shape[0] != self.n_req or (self.n_req and (didx.min() < 0 or didx.max() >= len(encs))):
            raise ValueError("desc_idx must hold one descriptor index per request")
        self.n_desc = len(encs)
        self.pool = torch.from_numpy(pool.copy()).to(device)
        self.msg_off = torch.from_numpy(offs).to(device)
        self.msg_len = torch.from_numpy(lens.astype(np.int32)).to(device)
        self.desc_idx = torch.from_numpy(didx.astype(np.int32)).to(device)
        self.desc_digests = torch.empty((max(1, self.n_desc), 16), dtype=torch.uint8, device=device)
        self.digests = torch.empty((max(1, self.n_req), 16), dtype=torch.uint8, device=device)
        self.key_off = torch.empty(self.n_req + 1, dtype=torch.int64, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        pkv_key_offsets(self.tok_off, self.block, self.key_off)
        self.n_keys = int(self.key_off[-1].item())
        self.keys = torch.empty((max(1, self.n_keys), 16), dtype=torch.uint8, device=device)
        self.hits = torch.zeros(max(1, self.n_req), dtype=torch.int32, device=device)
        self.n_new = torch.zeros(1, dtype=torch.int64, device=device)
        self.new_slots = torch.empty(max(1, self.n_keys), dtype=torch.int64, device=device)
        self.locs = None

    @classmethod
    def from_batch(cls, batch, device="cuda"):
        return cls(batch.tokens, batch.tok_off, batch.block, batch.descs, batch.desc_idx, device)

    def set_locations(self, locs: np.ndarray):
        import torch
        self.locs = torch.from_numpy(np.ascontiguousarray(locs).view(np.int64)).to(self.device)
        if self.locs.numel() == 0:
            self.locs = torch.zeros(1, dtype=torch.int64, device=self.device)

    # ---- the steps of the hot path ------------------------------------------------------------
    def key_offsets(self, stream=None):
        pkv_key_offsets(self.tok_off, self.block, self.key_off, stream)

    def digest(self, stream=None):
        """One digest per distinct descriptor, then one per request."""
        pkv_digest_batch(self.pool, self.msg_off, self.msg_len, self.desc_digests[: self.n_desc], self.status, stream)
        pkv_expand_digests(self.desc_digests[: self.n_desc], self.desc_idx, self.digests[: self.n_req], self.status,
                           stream)

    def derive(self, stream=None):
        pkv_derive_keys(self.tokens, self.tok_off, self.digests[: max(1, self.n_req)], self.block, self.key_off,
                        self.keys, self.status, stream)

    def lookup(self, table: Table, stream=None):
        pkv_lookup_prefix(table, self.keys, self.key_off, self.hits[: max(1, self.n_req)], self.status, stream)

    def derive_lookup(self, table: Table, stream=None):
        """Keys and hit lengths in one call (the fused kernel where it applies)."""
        pkv_derive_lookup(self.tokens, self.tok_off, self.digests[: max(1, self.n_req)], self.block, self.key_off,
                          self.keys, table, self.hits[: max(1, self.n_req)], self.status, stream)

    def store(self, table: Table, stream=None, log=True):
        pkv_store(table, self.keys, self.key_off, self.hits[: max(1, self.n_req)], self.locs, self.n_new,
                  self.status, self.new_slots if log else None, stream)

    def rollback(self, table: Table, stream=None):
        pkv_table_rollback(table, self.new_slots, self.n_new, stream)

    def step(self, table: Table, stream=None):
        """One pass of the whole hot path over this batch."""
        self.key_offsets(stream)
        self.digest(stream)
        self.derive(stream)
        self.lookup(table, stream)
        self.store(table, stream)

    def step_fused(self, table: Table, stream=None):
        """The same pass with keys and hit lengths from one call."""
        self.key_offsets(stream)
        self.digest(stream)
        self.derive_lookup(table, stream)
        self.store(table, stream)

    # ---- host views (synchronizing) ----------------------------------------------------------
    def host_keys(self) -> np.ndarray:
        return self.keys[: self.n_keys].cpu().numpy()

    def host_hits(self) -> np.ndarray:
        return self.hits[: self.n_req].cpu().numpy()

    def host_status(self) -> int:
        return int(self.status.item())


def export_sorted(table: Table):
    """(keys uint8 [n, 16], locs uint64 [n]) of every occupied slot, sorted by key bytes."""
    import torch
    cap = table.capacity
    keys = torch.empty((cap, 16), dtype=torch.uint8, device=table.slots.device)
    locs = torch.empty(cap, dtype=torch.int64, device=table.slots.device)
    count = torch.zeros(1, dtype=torch.int64, device=table.slots.device)
    pkv_table_export(table, keys, locs, count)
    n = int(count.item())
    k = keys[:n].cpu().numpy()
    v = locs[:n].cpu().numpy().view(np.uint64)
    return sort_pairs(k, v)


def key_order(keys: np.ndarray) -> np.ndarray:
    """Permutation that sorts 16-byte keys by their bytes (unsigned, most significant first): an
    argsort by the first 8 bytes, then runs that share them ordered by the last 8 bytes too."""
    words = np.ascontiguousarray(keys).view(">u8").reshape(-1, 2)
    order = np.argsort(words[:, 0])
    first = words[order, 0]
    tie = np.flatnonzero(first[1:] == first[:-1])
    if tie.size:
        pos = np.unique(np.concatenate([tie, tie + 1]))      # every position inside such a run
        sub = order[pos]
        order[pos] = sub[np.lexsort((words[sub, 1], words[sub, 0]))]
    return order


def sort_pairs(keys: np.ndarray, locs: np.ndarray):
    if keys.shape[0] == 0:
        return keys.reshape(0, 16), locs
    order = key_order(keys)
    return keys[order], locs[order]


class TwoStreamRunner:
    """Runs consecutive batches through the hot path on two HIP streams.

    Key derivation touches no index state, so the derive of batch k+1 can run while batch k is looked
    up and stored.  Every index operation (lookup, store, rollback) stays on one stream in batch
    order, so the hit lengths and the index contents equal those of running the batches one after
    another.  The preparation of a batch (descriptor digests, key offsets) also runs on the index
    stream, two passes ahead: the digests of batch k+2 right after the derive of batch k (whose
    digest buffers they may reuse) and its key offsets after batch k's index work (whose key
    offsets they may overwrite), so that the derive of batch k+2 is ready to start once the derive
    of batch k+1 ends and is launched onto a GPU whose index stream has gone quiet.

    Both streams have the default priority.  A ``DeviceBatch`` may be reused (its buffers are
    recycled once its previous pass has finished) but not twice in a row.
    """

    def __init__(self, table: Table):
        import torch
        self.table = table
        self.s_derive = torch.cuda.Stream()
        self.s_index = torch.cuda.Stream()

    def run(self, batches, rollback: bool = False, derive_events=None, index_work=None):
        """Enqueue one pass per entry of ``batches``; returns without synchronizing.
        ``derive_events[k]`` (a pair of timing events), when given, brackets the derive of pass k on
        the derive stream.  ``index_work(k, batch, stream)``, when given, enqueues pass k's index
        operations on ``stream`` in place of the default (lookup, store, optional rollback); it is
        called in pass order."""
        import torch
        batches = list(batches)
        for a, b in zip(batches, batches[1:]):
            if a is b:
                raise ValueError("the same DeviceBatch cannot run twice in a row")
        cur = torch.cuda.current_stream()
        self.s_derive.wait_stream(cur)
        self.s_index.wait_stream(cur)
        if not batches:
            return
        ready = {}

        def mark(j):
            ev = torch.cuda.Event()
            ev.record(self.s_index)
            ready[j] = ev

        for j in range(min(2, len(batches))):
            batches[j].digest(self.s_index)
            batches[j].key_offsets(self.s_index)
            mark(j)
        for k, db in enumerate(batches):
            self.s_derive.wait_event(ready.pop(k))
            ev = derive_events[k] if derive_events is not None else None
            if ev is not None:
                ev[0].record(self.s_derive)
            db.derive(self.s_derive)
            done = ev[1] if ev is not None else torch.cuda.Event()
            done.record(self.s_derive)
            self.s_index.wait_event(done)
            ahead = batches[k + 2] if k + 2 < len(batches) else None
            if ahead is not None:
                ahead.digest(self.s_index)
            if index_work is not None:
                index_work(k, db, self.s_index)
            else:
                with torch.cuda.stream(self.s_index):
                    db.n_new.zero_()
                db.lookup(self.table, self.s_index)
                db.store(self.table, self.s_index)
                if rollback:
                    db.rollback(self.table, self.s_index)
            if ahead is not None:
                ahead.key_offsets(self.s_index)
                mark(k + 2)
        cur.wait_stream(self.s_derive)
        cur.wait_stream(self.s_index)
