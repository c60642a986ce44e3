"""Pins of the oracle's content identity (section 5.3: an adapter is bound by the identity of its
contents; the hash is this build's definition, see oracle/identity.py).  The tree is recomputed
with the library SHA-256 (hashlib) on small tensors, including every leaf and fan-in edge, and the
identity must respond to every field it covers and to nothing else."""

import hashlib
import struct

import numpy as np
import pytest

from oracle.identity import identity, leaves, record, tensor_root


def _h(b):
    return hashlib.sha256(b).digest()


def _lib_root(data):
    lv = [_h(b"\x00" + data[i:i + 1024]) for i in range(0, len(data), 1024)] or [_h(b"\x00")]
    while len(lv) > 1:
        lv = [_h(b"\x01" + b"".join(lv[i:i + 16])) for i in range(0, len(lv), 16)]
    return lv[0]


@pytest.mark.parametrize("n", [0, 1, 1023, 1024, 1025, 16 * 1024, 16 * 1024 + 1, 17 * 1024, 256 * 1024 + 7])
def test_root_matches_library_sha256(n):
    data = np.random.default_rng(n).integers(0, 256, size=n, dtype=np.uint8).tobytes()
    assert tensor_root(data) == _lib_root(data)


def test_tree_shape_edges():
    one = bytes(1024)
    assert tensor_root(one) == _h(b"\x00" + one)                      # one leaf: the leaf is the root
    two = bytes(1025)
    assert tensor_root(two) == _h(b"\x01" + _h(b"\x00" + bytes(1024)) + _h(b"\x00" + bytes(1)))
    sixteen = bytes(16 * 1024)
    assert len(leaves(sixteen)) == 16
    assert tensor_root(sixteen) == _h(b"\x01" + b"".join([_h(b"\x00" + bytes(1024))] * 16))


def _adapter(rng, n=5):
    return [(b"layer.%d.lora_%s" % (i, b"AB"[i % 2:i % 2 + 1]), b"bfloat16", (16, 64 + i),
             rng.integers(0, 256, size=2 * 16 * (64 + i), dtype=np.uint8).tobytes()) for i in range(n)]


def test_identity_definition_and_sensitivity():
    rng = np.random.default_rng(7)
    ts = _adapter(rng)
    cfg = [(b"r", b"16"), (b"alpha", b"32")]
    base = identity(ts, cfg)
    recs = sorted((n, record(n, dt, sh, d)) for n, dt, sh, d in ts)
    msg = b"PKVA" + struct.pack("<I", 5) + b"".join(r for _, r in recs) + struct.pack("<I", 2)
    for k, v in sorted(cfg):
        msg += struct.pack("<I", len(k)) + k + struct.pack("<I", len(v)) + v
    assert base == _h(msg)
    assert identity(list(reversed(ts)), list(reversed(cfg))) == base          # order-free
    n, dt, sh, d = ts[2]
    flipped = bytearray(d)
    flipped[len(d) // 2] ^= 1
    variants = [
        ts[:2] + [(n, dt, sh, bytes(flipped))] + ts[3:],                      # one bit of content
        ts[:2] + [(n + b"x", dt, sh, d)] + ts[3:],                            # a name
        ts[:2] + [(n, b"float16", sh, d)] + ts[3:],                           # a dtype
        ts[:2] + [(n, dt, (sh[1], sh[0]), d)] + ts[3:],                        # a shape
        ts[:4],                                                               # a tensor dropped
    ]
    for v in variants:
        assert identity(v, cfg) != base
    assert identity(ts, cfg[:1]) != base
    assert identity(ts, [(b"r", b"16"), (b"alpha", b"33")]) != base


def test_record_layout_written_out():
    # the record of one small tensor, byte by byte (little-endian integers; the root from hashlib)
    data = bytes(range(12))
    root = _h(b"\x00" + data)
    want = (b"PKVT" + b"\x01\x00\x00\x00" + b"w" + b"\x04\x00\x00\x00" + b"bf16" + b"\x02\x00\x00\x00"
            + b"\x02\x00\x00\x00\x00\x00\x00\x00" + b"\x03\x00\x00\x00\x00\x00\x00\x00"
            + b"\x0c\x00\x00\x00\x00\x00\x00\x00" + root)
    assert record(b"w", b"bf16", (2, 3), data) == want
    assert len(want) == 4 + 4 + 1 + 4 + 4 + 4 + 16 + 8 + 32
