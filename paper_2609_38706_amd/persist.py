"""Index persistence: save an index's (key, location) pairs to a file and rebuild an index from
them, for restart parity (section 6.3: a restarted worker must keep hitting what the store
holds).  Keys depend only on the bytes of tokens and descriptor fields, so an index rebuilt from
its pairs serves a restarted process exactly as before.

The pairs leave the GPU through ``pkv_table_export`` and enter a new index through ``pkv_store``
(one request holding every pair, hit length 0, so every pair is inserted); only the file I/O
runs on the host.  File format: numpy ``.npz`` with ``capacity`` (int64), ``keys`` (uint8 [n, 16])
and ``locs`` (uint64 [n]), pairs in ascending key order.
"""

from __future__ import annotations

import numpy as np

from . import Table, pkv_store
from .pipeline import export_sorted


def save_table(table: Table, path: str):
    keys, locs = export_sorted(table)
    np.savez(path, capacity=np.int64(table.capacity), keys=keys, locs=locs.astype(np.uint64))


def import_pairs(table: Table, keys, locs, stream=None):
    """Inserts (key, location) pairs (device tensors uint8 [n, 16], int64 [n]) into `table`;
    returns the status word (device) and the new-entry counter (device)."""
    import torch
    dev = table.slots.device
    n = int(keys.shape[0])
    key_off = torch.tensor([0, n], dtype=torch.int64, device=dev)
    hits = torch.zeros(1, dtype=torch.int32, device=dev)
    n_new = torch.zeros(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    if n == 0:
        return status, n_new
    pkv_store(table, keys, key_off, hits, locs, n_new, status, None, stream)
    return status, n_new


def load_table(path: str, device="cuda", capacity: int | None = None) -> Table:
    """A new index holding the saved pairs (capacity: the saved one unless given)."""
    import torch
    with np.load(path, allow_pickle=False) as f:
        cap = int(f["capacity"]) if capacity is None else int(capacity)
        keys = np.ascontiguousarray(f["keys"], dtype=np.uint8).reshape(-1, 16)
        locs = np.ascontiguousarray(f["locs"], dtype=np.uint64)
    table = Table(cap, device=device)
    if keys.shape[0]:
        kd = torch.from_numpy(keys).to(device)
        ld = torch.from_numpy(locs.view(np.int64)).to(device)
        status, n_new = import_pairs(table, kd, ld)
        st = int(status.item())
        if st != 0:
            raise RuntimeError(f"index import failed: status {st}")
        if int(n_new.item()) != keys.shape[0]:
            raise RuntimeError("index import: saved pairs are not distinct")
    return table
