"""Pins of the oracle's chained block keys.

key_i = H(key_{i-1} | d | LE32 tokens of block i), key_0 = 0^16, H = SHA-256 truncated to 128
bits, only complete blocks keyed (section 4.4).  The pins are the library routine on the first
key (the chain seed is a constant, so key_1 is one SHA-256 of an explicit byte string) and
invariants that break if a term, an index or an operand order is wrong."""

import hashlib
import struct

import numpy as np
import pytest

import oracle


def _req(tokens_list, block, digests=None, threads=1):
    chunks = [np.asarray(t, np.int32) for t in tokens_list]
    off = np.zeros(len(chunks) + 1, np.int64)
    off[1:] = np.cumsum([c.shape[0] for c in chunks])
    toks = np.concatenate(chunks) if chunks else np.zeros(0, np.int32)
    if digests is None:
        digests = np.zeros((len(chunks), 16), np.uint8)
    keys = oracle.derive(toks, off, np.asarray(digests, np.uint8), block, threads)
    ko = oracle.key_offsets(off, block)
    return [keys[ko[r]:ko[r + 1]] for r in range(len(chunks))]


@pytest.mark.parametrize("block", [1, 3, 16, 17, 256])
def test_first_key_is_library_sha256(block):
    rng = np.random.default_rng(block)
    toks = rng.integers(-2**31, 2**31, size=block * 2 + 1, dtype=np.int64).astype(np.int32)
    d = rng.integers(0, 256, size=16, dtype=np.uint8)
    (keys,) = _req([toks], block, d[None])
    msg = bytes(16) + d.tobytes() + struct.pack("<%di" % block, *toks[:block].tolist())
    assert keys[0].tobytes() == hashlib.sha256(msg).digest()[:16]


@pytest.mark.parametrize("length,block,n", [(0, 16, 0), (15, 16, 0), (16, 16, 1), (31, 16, 1), (32, 16, 2),
                                            (2048, 16, 128), (8191, 256, 31), (8192, 256, 32), (5, 1, 5)])
def test_only_complete_blocks_are_keyed(length, block, n):
    (keys,) = _req([np.arange(length)], block)
    assert keys.shape == (n, 16)


def test_shared_prefix_shares_exactly_its_complete_blocks():
    rng = np.random.default_rng(1)
    block = 16
    base = rng.integers(0, 1000, size=160, dtype=np.int32)
    for fork in [0, 1, 15, 16, 17, 64, 100, 159]:
        other = base.copy()
        other[fork] += 1                       # first differing token
        a, b = _req([base, other], block)
        shared = fork // block                 # complete blocks before the fork
        assert all((a[i] == b[i]).all() for i in range(shared))
        assert all((a[i] != b[i]).any() for i in range(shared, a.shape[0]))


def test_changing_one_token_changes_its_block_and_every_later_key():
    rng = np.random.default_rng(2)
    toks = rng.integers(0, 1000, size=16 * 20, dtype=np.int32)
    (ref,) = _req([toks], 16)
    for pos in [0, 5, 16 * 7 + 3, 16 * 19 + 15]:
        t2 = toks.copy()
        t2[pos] ^= 1
        (k2,) = _req([t2], 16)
        j = pos // 16
        assert (k2[:j] == ref[:j]).all()
        assert all((k2[i] != ref[i]).any() for i in range(j, 20))


def test_digest_is_bound_into_every_key():
    rng = np.random.default_rng(3)
    toks = rng.integers(0, 1000, size=16 * 10, dtype=np.int32)
    d = rng.integers(0, 256, size=(2, 16), dtype=np.uint8)
    d[1] = d[0]
    d[1, 15] ^= 0x80                             # one bit of the digest differs
    a, b = _req([toks, toks], 16, d)
    assert all((a[i] != b[i]).any() for i in range(10))


def test_same_block_at_another_position_keys_differently():
    blk = np.arange(16, dtype=np.int32)
    (k,) = _req([np.concatenate([blk, blk, blk])], 16)
    assert len({bytes(x) for x in k}) == 3      # the chain makes each occurrence distinct


def test_token_bytes_are_little_endian_int32():
    # 0x01020304 vs 0x04030201 must differ, and the LE serialisation is what the library sees
    (k,) = _req([np.array([0x01020304], np.int32)], 1)
    assert k[0].tobytes() == hashlib.sha256(bytes(32) + bytes([4, 3, 2, 1])).digest()[:16]


def test_threads_do_not_change_results():
    rng = np.random.default_rng(4)
    reqs = [rng.integers(0, 5000, size=int(rng.integers(0, 700)), dtype=np.int32) for _ in range(37)]
    d = rng.integers(0, 256, size=(37, 16), dtype=np.uint8)
    a = _req(reqs, 16, d, threads=1)
    b = _req(reqs, 16, d, threads=5)
    assert all((x == y).all() for x, y in zip(a, b))


def _library_chain(tokens, digest: bytes, block: int):
    """The chain written out with the library SHA-256: key_i = SHA-256(key_{i-1} | d | LE32 tokens)[:16]."""
    prev, out = bytes(16), []
    for i in range(len(tokens) // block):
        blk = struct.pack("<%di" % block, *[int(t) for t in tokens[i * block:(i + 1) * block]])
        prev = hashlib.sha256(prev + digest + blk).digest()[:16]
        out.append(prev)
    return out


@pytest.mark.parametrize("block", [1, 2, 5, 16, 17, 64, 256])
def test_whole_chains_match_library_sha256(block):
    """Brute force on tiny inputs: every key of several ragged requests, recomputed from the byte-level
    definition with the library routine (OpenSSL SHA-256), not with the oracle's own hash."""
    rng = np.random.default_rng(100 + block)
    reqs = [rng.integers(-2**31, 2**31, size=int(rng.integers(0, 5 * block + 3)), dtype=np.int64).astype(np.int32)
            for _ in range(6)]
    digs = rng.integers(0, 256, size=(6, 16), dtype=np.uint8)
    got = _req(reqs, block, digs)
    for r in range(6):
        want = _library_chain(reqs[r], digs[r].tobytes(), block)
        assert [bytes(k) for k in got[r]] == want
