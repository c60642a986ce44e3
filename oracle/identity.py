"""Content identities of adapters and checkpoints -- TEST INFRASTRUCTURE ONLY.

Section 5.3 binds an adapter by an identity of its contents (every tensor's name, dtype, shape and
bytes, with the meaningful configuration fields), and section 6.5 reports the cost of computing
it.  The paper fixes no hash for it, so this build defines one (written out here in its plain
form, with the oracle's SHA-256):

  leaf_i(x)  = SHA-256(0x00 | x[1024 i : 1024 (i + 1)])          leaves of 1024 bytes; an empty
                                                                 tensor has one empty leaf
  node(c..)  = SHA-256(0x01 | c_1 | ... | c_k)                    k <= 16 consecutive children
  level j+1  = nodes over consecutive groups of 16 level-j digests; the first level with a
               single digest holds the tensor's root
  record(t)  = "PKVT" | u32(|name|) name | u32(|dtype|) dtype | u32(ndim) u64(dim)* |
               u64(byte length) | root                            (little-endian integers)
  identity   = SHA-256("PKVA" | u32(#tensors) | records in name order |
                       u32(#fields) | (u32(|k|) k u32(|v|) v)* in key order)   (32 bytes)
"""

from __future__ import annotations

import struct

from . import sha256

LEAF = 1024
FANIN = 16


def leaves(data: bytes):
    if len(data) == 0:
        return [sha256(b"\x00")]
    return [sha256(b"\x00" + data[i:i + LEAF]) for i in range(0, len(data), LEAF)]


def tensor_root(data: bytes) -> bytes:
    level = leaves(bytes(data))
    while len(level) > 1:
        level = [sha256(b"\x01" + b"".join(level[i:i + FANIN])) for i in range(0, len(level), FANIN)]
    return level[0]


def record(name: bytes, dtype: bytes, shape, data: bytes, root: bytes | None = None) -> bytes:
    root = tensor_root(data) if root is None else root
    out = b"PKVT" + struct.pack("<I", len(name)) + name + struct.pack("<I", len(dtype)) + dtype
    out += struct.pack("<I", len(shape)) + b"".join(struct.pack("<Q", int(d)) for d in shape)
    return out + struct.pack("<Q", len(data)) + root


def identity(tensors, config=()) -> bytes:
    """tensors: iterable of (name, dtype, shape, data bytes); config: (key, value) byte pairs."""
    recs = sorted((bytes(n), record(bytes(n), bytes(dt), shape, bytes(d))) for n, dt, shape, d in tensors)
    msg = b"PKVA" + struct.pack("<I", len(recs)) + b"".join(r for _, r in recs)
    cfg = sorted((bytes(k), bytes(v)) for k, v in config)
    msg += struct.pack("<I", len(cfg))
    for k, v in cfg:
        msg += struct.pack("<I", len(k)) + k + struct.pack("<I", len(v)) + v
    return sha256(msg)
