"""Differential omission test (section 5.4, Eq. 4) at key level on the GPU.

For every key binding R and every registered dimension d, the keys of the base configurations c
and of c[d -> v'] are compared over the same tokens x; a coinciding key under a dimension that is
declared to change the state (or the sharing permission) is an omission.  The comparison runs in
the store-side form of section 6.4: the base keys of every binding are stored in one index and
the variant keys are looked up, so a hit is a key the two configurations share.  Because v'
differs from every base value, a variant key can only coincide with the base key of its own
binding and request position, and chained keys coincide either on every block (the projected
descriptors are equal) or on none, so the hit lengths count the coinciding blocks exactly.

One combined batch holds, for every binding, the base requests and then, per dimension, the
variant requests (all over the same tokens), so a single derive launch covers every
configuration.  This module only arranges inputs and launches: the descriptor projection is
host-side marshalling of byte fields; digests, keys, the index and the sums are kernels.
"""

from __future__ import annotations

import numpy as np

from . import Table, pkv_lookup_prefix, pkv_store, pkv_sum_hits
from .pipeline import DeviceBatch


def _project(desc, names):
    return [(n, v) for n, v in desc if names is None or n in names]


def _vary(desc, name, value):
    return [(n, v) for n, v in desc if n != name] + [(name, value)]


class OmissionRun:
    """Device buffers of one omission test; ``run()`` enqueues the whole test on a stream."""

    def __init__(self, case, device="cuda"):
        import torch
        b = case.batch
        self.case = case
        nb, nd, n = len(case.bindings), len(case.dims), b.n_req
        self.nb, self.nd, self.n = nb, nd, n
        groups = nb * (1 + nd)
        # distinct projected descriptors; per base descriptor, the index of each projection
        descs, seen = [], {}

        def index_of(d):
            k = tuple(sorted(d))
            if k not in seen:
                seen[k] = len(descs)
                descs.append(d)
            return seen[k]

        n_base = len(b.descs)
        base_ix = np.empty((nb, n_base), np.int32)
        var_ix = np.empty((nb, nd, n_base), np.int32)
        for i, (_label, names) in enumerate(case.bindings):
            for k, d in enumerate(b.descs):
                base_ix[i, k] = index_of(_project(d, names))
                for j, dim in enumerate(case.dims):
                    var_ix[i, j, k] = index_of(_project(_vary(d, dim, case.variants[dim]), names))
        didx = np.concatenate([base_ix[:, b.desc_idx].reshape(-1), var_ix[:, :, b.desc_idx].reshape(-1)])
        # every group keys the same tokens: the request offsets repeat with a stride of the token count
        total = int(b.tok_off[-1])
        tok_off = (b.tok_off[:-1][None, :] + total * np.arange(groups, dtype=np.int64)[:, None]).reshape(-1)
        tok_off = np.concatenate([tok_off, [total * groups]]).astype(np.int64)
        tokens = torch.from_numpy(np.ascontiguousarray(b.tokens, dtype=np.int32)).to(device).repeat(groups)
        self.db = DeviceBatch(tokens, tok_off, b.block, descs, didx.astype(np.int32), device)
        ko = self.db.key_off.cpu().numpy()
        self.n_keys = int(ko[-1])
        self.base_keys = int(ko[nb * n])
        # locations: any value below the reserved range; the index is only probed for presence
        self.db.set_locations(np.arange(self.n_keys, dtype=np.uint64))
        cap = 4
        while cap < 2 * max(1, self.base_keys):
            cap *= 2
        self.table = Table(cap, device=device, init=False)
        self.group_off = torch.from_numpy(np.arange(nb * nd + 1, dtype=np.int64) * n).to(device)
        self.sums = torch.zeros(nb * nd, dtype=torch.int64, device=device)
        self.n_new = torch.zeros(1, dtype=torch.int64, device=device)

    def run(self, stream=None, derive_events=None):
        """Digests, keys, index of the base keys, lookup of the variant keys, per-group sums.
        ``derive_events`` (a pair of timing events), when given, brackets the derive launch."""
        import torch
        from . import pkv_table_init
        db, nb, n = self.db, self.nb, self.n
        s = stream if stream is not None else torch.cuda.current_stream()
        db.key_offsets(stream)
        db.digest(stream)
        if derive_events is not None:
            derive_events[0].record(s)
        db.derive(stream)
        if derive_events is not None:
            derive_events[1].record(s)
        pkv_table_init(self.table, stream)
        with torch.cuda.stream(s):
            db.hits[: nb * n].zero_()
            self.n_new.zero_()
        pkv_store(self.table, db.keys, db.key_off[: nb * n + 1], db.hits[: nb * n], db.locs, self.n_new, db.status,
                  db.new_slots, stream)
        pkv_lookup_prefix(self.table, db.keys, db.key_off[nb * n:], db.hits[nb * n:], db.status, stream)
        pkv_sum_hits(db.hits[nb * n:], self.group_off, self.sums, db.status, stream)

    def result(self):
        """(collisions int64 [bindings, dims], omission bool [bindings, dims], blocks per configuration);
        synchronizes."""
        if self.db.host_status() != 0:
            raise RuntimeError(f"omission test failed on the device: status {self.db.host_status()}")
        coll = self.sums.cpu().numpy().reshape(self.nb, self.nd)
        changes = np.array([bool(self.case.changes[d]) for d in self.case.dims])
        return {"collisions": coll, "omission": (coll > 0) & changes[None, :], "blocks": self.base_keys // self.nb}

    def variant_hits(self, binding: int, dim: int):
        """Per-request hit lengths of one (binding, dimension) group (host copy)."""
        start = self.nb * self.n + (binding * self.nd + dim) * self.n
        return self.db.hits[start:start + self.n].cpu().numpy()


def omission_check(case, device="cuda"):
    run = OmissionRun(case, device)
    run.run()
    return run.result()
