"""CPU oracle for provenance-bound KV-cache keys -- TEST INFRASTRUCTURE ONLY.

A plain C implementation (``pkv_oracle.c``) of what the hot path computes, loaded through
ctypes.  Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may
import this package; the product library and its binding never do.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# PKV_ORACLE_LIB points the tests at another build of this oracle (the mutation tests use it).
LIB_PATH = os.environ.get("PKV_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")
SOURCES = [os.path.join(HERE, "pkv_oracle.c")]

OK, EINVAL, EDUPDIM, ERESERVED, EFULL = 0, -1, -2, -3, -4


def build(verbose: bool = False) -> str:
    """Compile the oracle with the host C compiler (plain -O2, no target-specific extensions)."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared", "-o", tmp] + SOURCES + ["-lpthread"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


class _Field(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("name_len", ctypes.c_uint32),
                ("value", ctypes.c_char_p), ("value_len", ctypes.c_uint32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.orc_sha256.argtypes = [P, ctypes.c_uint64, P]
        L.orc_sha256_constants.argtypes = [P, P]
        L.orc_encode.argtypes = [P, ctypes.c_uint32, P, ctypes.c_uint64, P]
        L.orc_digest.argtypes = [P, ctypes.c_uint32, P]
        L.orc_key_offsets.argtypes = [P, ctypes.c_uint32, ctypes.c_uint32, P]
        L.orc_key_offsets.restype = ctypes.c_int64
        L.orc_derive.argtypes = [P, P, ctypes.c_uint32, P, ctypes.c_uint32, P, ctypes.c_int]
        L.orc_index_new.argtypes = [ctypes.c_uint64]
        L.orc_index_new.restype = P
        L.orc_index_set_threads.argtypes = [P, ctypes.c_int]
        L.orc_index_free.argtypes = [P]
        L.orc_index_clone.argtypes = [P]
        L.orc_index_clone.restype = P
        L.orc_index_size.argtypes = [P]
        L.orc_index_size.restype = ctypes.c_uint64
        L.orc_index_dump.argtypes = [P, P, P]
        L.orc_lookup.argtypes = [P, P, P, ctypes.c_uint32, P]
        L.orc_store.argtypes = [P, P, P, ctypes.c_uint32, P, P]
        L.orc_index_dump_epochs.argtypes = [P, P]
        L.orc_lookup_touch.argtypes = [P, P, P, ctypes.c_uint32, P, ctypes.c_uint32]
        L.orc_store_touch.argtypes = [P, P, P, ctypes.c_uint32, P, P, ctypes.c_uint32]
        L.orc_evict.argtypes = [P, ctypes.c_uint64]
        L.orc_evict.restype = ctypes.c_uint64
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _fields(desc):
    arr = (_Field * max(1, len(desc)))()
    keep = []
    for i, (n, v) in enumerate(desc):
        n, v = bytes(n), bytes(v)
        keep += [n, v]
        arr[i] = _Field(n, len(n), v, len(v))
    return arr, keep


def sha256(msg: bytes) -> bytes:
    out = (ctypes.c_uint8 * 32)()
    buf = np.frombuffer(bytes(msg) + b"\0", dtype=np.uint8)
    lib().orc_sha256(_ptr(buf), len(msg), out)
    return bytes(out)


def sha256_constants():
    k = np.zeros(64, np.uint32)
    iv = np.zeros(8, np.uint32)
    lib().orc_sha256_constants(_ptr(k), _ptr(iv))
    return k, iv


def encode(desc) -> bytes:
    arr, _keep = _fields(desc)
    n = ctypes.c_uint64(0)
    rc = lib().orc_encode(arr, len(desc), None, 0, ctypes.byref(n))
    if rc:
        raise OracleError(rc)
    out = np.zeros(max(1, n.value), np.uint8)
    rc = lib().orc_encode(arr, len(desc), _ptr(out), n.value, ctypes.byref(n))
    if rc:
        raise OracleError(rc)
    return out[: n.value].tobytes()


def digest(desc) -> bytes:
    arr, _keep = _fields(desc)
    out = (ctypes.c_uint8 * 16)()
    rc = lib().orc_digest(arr, len(desc), out)
    if rc:
        raise OracleError(rc)
    return bytes(out)


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle error {code}")
        self.code = code


def key_offsets(tok_off: np.ndarray, block: int) -> np.ndarray:
    tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
    out = np.zeros(tok_off.shape[0], np.int64)
    lib().orc_key_offsets(_ptr(tok_off), tok_off.shape[0] - 1, block, _ptr(out))
    return out


def derive(tokens, tok_off, digests, block, threads=1):
    """Keys of every complete block of every request: uint8 [n_keys, 16]."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    tok_off = np.ascontiguousarray(tok_off, dtype=np.int64)
    digests = np.ascontiguousarray(digests, dtype=np.uint8).reshape(-1, 16)
    n_req = tok_off.shape[0] - 1
    assert digests.shape[0] == n_req
    ko = key_offsets(tok_off, block)
    keys = np.zeros((max(1, int(ko[-1])), 16), np.uint8)
    rc = lib().orc_derive(_ptr(tokens), _ptr(tok_off), n_req, _ptr(digests), block, _ptr(keys), threads)
    if rc:
        raise OracleError(rc)
    return keys[: int(ko[-1])]


def batch_digests(batch) -> np.ndarray:
    """Per-request digests of a ``workloads.Batch`` (one computation per distinct descriptor)."""
    per_desc = [digest(d) for d in batch.descs]
    table = np.frombuffer(b"".join(per_desc), np.uint8).reshape(-1, 16) if per_desc else np.zeros((0, 16), np.uint8)
    return table[np.asarray(batch.desc_idx, dtype=np.int64)]


class Index:
    """The oracle's index: a sorted set of (key, location) pairs with a capacity."""

    def __init__(self, capacity: int, _handle=None, threads: int = 1):
        """``threads``: how many threads the store's sort and the lookup may use (results do not
        depend on it)."""
        self.capacity = capacity
        self._h = _handle if _handle is not None else lib().orc_index_new(capacity)
        if _handle is None:
            lib().orc_index_set_threads(self._h, int(threads))

    def clone(self) -> "Index":
        h = lib().orc_index_clone(self._h)
        if not h:
            raise MemoryError("oracle index clone")
        return Index(self.capacity, h)

    def __del__(self):
        if getattr(self, "_h", None):
            lib().orc_index_free(self._h)
            self._h = None

    def __len__(self):
        return int(lib().orc_index_size(self._h))

    def dump(self):
        n = len(self)
        keys = np.zeros((max(1, n), 16), np.uint8)
        locs = np.zeros(max(1, n), np.uint64)
        lib().orc_index_dump(self._h, _ptr(keys), _ptr(locs))
        return keys[:n], locs[:n]

    def dump_epochs(self) -> np.ndarray:
        n = len(self)
        ep = np.zeros(max(1, n), np.uint32)
        lib().orc_index_dump_epochs(self._h, _ptr(ep))
        return ep[:n]

    def lookup_touch(self, keys, key_off, epoch: int) -> np.ndarray:
        keys = np.ascontiguousarray(keys, dtype=np.uint8)
        key_off = np.ascontiguousarray(key_off, dtype=np.int64)
        hits = np.zeros(max(1, key_off.shape[0] - 1), np.int32)
        lib().orc_lookup_touch(self._h, _ptr(keys), _ptr(key_off), key_off.shape[0] - 1, _ptr(hits), epoch)
        return hits[: key_off.shape[0] - 1]

    def store_touch(self, keys, key_off, hits, locs, epoch: int) -> int:
        keys = np.ascontiguousarray(keys, dtype=np.uint8)
        key_off = np.ascontiguousarray(key_off, dtype=np.int64)
        hits = np.ascontiguousarray(hits, dtype=np.int32)
        locs = np.ascontiguousarray(locs, dtype=np.uint64)
        return int(lib().orc_store_touch(self._h, _ptr(keys), _ptr(key_off), key_off.shape[0] - 1, _ptr(hits),
                                         _ptr(locs), epoch))

    def evict(self, budget: int) -> int:
        return int(lib().orc_evict(self._h, budget))

    def lookup(self, keys, key_off) -> np.ndarray:
        keys = np.ascontiguousarray(keys, dtype=np.uint8)
        key_off = np.ascontiguousarray(key_off, dtype=np.int64)
        hits = np.zeros(max(1, key_off.shape[0] - 1), np.int32)
        lib().orc_lookup(self._h, _ptr(keys), _ptr(key_off), key_off.shape[0] - 1, _ptr(hits))
        return hits[: key_off.shape[0] - 1]

    def store(self, keys, key_off, hits, locs) -> int:
        keys = np.ascontiguousarray(keys, dtype=np.uint8)
        key_off = np.ascontiguousarray(key_off, dtype=np.int64)
        hits = np.ascontiguousarray(hits, dtype=np.int32)
        locs = np.ascontiguousarray(locs, dtype=np.uint64)
        return int(lib().orc_store(self._h, _ptr(keys), _ptr(key_off), key_off.shape[0] - 1, _ptr(hits), _ptr(locs)))
