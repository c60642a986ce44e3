"""Python binding of the pkv C ABI (include/pkv.h): provenance-bound shared-tier KV-cache keys on
MI355X.  Argument marshalling only -- every step runs in the HIP library ``lib/libpkv.so``.

Device buffers are torch tensors on the current HIP device; uint64 buffers are int64 tensors with
the same bits.  Every device call is asynchronous on ``stream`` (default: torch's current stream).
"""

from __future__ import annotations

import ctypes
import os

from ._build import LIB_PATH, build  # noqa: F401

PKV_OK, PKV_EINVAL, PKV_EDUPDIM, PKV_ERESERVED, PKV_EFULL, PKV_EHIP, PKV_ELAYOUT, PKV_ESTALL = 0, -1, -2, -3, -4, -5, -6, -7
PKV_LOC_LIMIT = 1 << 62
ERROR_NAMES = {0: "PKV_OK", -1: "PKV_EINVAL", -2: "PKV_EDUPDIM", -3: "PKV_ERESERVED", -4: "PKV_EFULL",
               -5: "PKV_EHIP", -6: "PKV_ELAYOUT", -7: "PKV_ESTALL"}

EXPORTED = ["pkv_descriptor_encode", "pkv_descriptor_digest", "pkv_digest_batch", "pkv_expand_digests",
            "pkv_key_offsets",
            "pkv_derive_keys", "pkv_derive_lookup", "pkv_table_bytes", "pkv_table_init", "pkv_lookup_prefix", "pkv_store", "pkv_table_rollback",
            "pkv_table_export", "pkv_sum_hits", "pkv_lookup_prefix_touch", "pkv_store_touch",
            "pkv_table_evict", "pkv_tree_work_bytes", "pkv_tensor_roots", "pkv_tensor_roots_static",
            "pkv_content_identity",
            "pkv_last_error", "pkv_version"]

EVICT_WORK_BYTES = 3 * 2048 * 4 + 64   # PKV_EVICT_WORK_BYTES
STATIC_TREE_WORK_BYTES = 8 << 20      # PKV_STATIC_TREE_WORK_BYTES


class PkvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


class pkv_field(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("name_len", ctypes.c_uint32),
                ("value", ctypes.c_char_p), ("value_len", ctypes.c_uint32)]


class pkv_table(ctypes.Structure):
    _fields_ = [("slots", ctypes.c_void_p), ("capacity", ctypes.c_uint64)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded HIP library.  Raises if it has not been built: there is no fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"the pkv HIP library is not built ({LIB_PATH}); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, U32, U64, I32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int
        sig = {
            "pkv_descriptor_encode": [P, ctypes.c_size_t, P, ctypes.c_size_t, P],
            "pkv_descriptor_digest": [P, ctypes.c_size_t, P],
            "pkv_digest_batch": [P, U64, P, P, U32, P, P, P],
            "pkv_key_offsets": [P, U32, U32, P, P],
            "pkv_expand_digests": [P, U32, P, U32, P, P, P],
            "pkv_derive_keys": [P, U64, P, U32, P, U32, P, U64, P, P, P],
            "pkv_derive_lookup": [P, U64, P, U32, P, U32, P, U64, P, P, P, P, P],
            "pkv_table_init": [P, P],
            "pkv_lookup_prefix": [P, P, P, U32, U64, P, P, P],
            "pkv_store": [P, P, P, U32, U64, P, P, P, P, P, P],
            "pkv_table_rollback": [P, P, P, U64, P],
            "pkv_table_export": [P, P, P, P, P],
            "pkv_sum_hits": [P, U32, P, U32, P, P, P],
            "pkv_lookup_prefix_touch": [P, P, P, U32, U64, P, U32, P, P, P],
            "pkv_store_touch": [P, P, P, U32, U64, P, P, P, P, P, U32, P, P],
            "pkv_table_evict": [P, P, U64, P, P, P],
            "pkv_tensor_roots": [P, U64, P, P, U32, P, U64, P, P, P],
            "pkv_tensor_roots_static": [P, U64, P, P, U32, P, P, P],
            "pkv_content_identity": [P, U32, P, ctypes.c_size_t, P],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = I32
        L.pkv_tree_work_bytes.argtypes = [U64, U32]
        L.pkv_tree_work_bytes.restype = U64
        L.pkv_table_bytes.argtypes = [U64]
        L.pkv_table_bytes.restype = U64
        L.pkv_last_error.restype = ctypes.c_char_p
        L.pkv_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int):
    if rc != PKV_OK:
        raise PkvError(rc, lib().pkv_last_error().decode(errors="replace"))


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, dtype=None, device=True):
    if t is None:
        return None
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if device and not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    return ctypes.c_void_p(t.data_ptr())


def _fields(desc):
    arr = (pkv_field * max(1, len(desc)))()
    keep = []
    for i, (n, v) in enumerate(desc):
        n, v = bytes(n), bytes(v)
        keep += [n, v]
        arr[i] = pkv_field(n, len(n), v, len(v))
    return arr, keep


# ---- host -------------------------------------------------------------------------------------

def pkv_descriptor_encode(desc) -> bytes:
    arr, _keep = _fields(desc)
    n = ctypes.c_size_t(0)
    _check(lib().pkv_descriptor_encode(arr, len(desc), None, 0, ctypes.byref(n)))
    out = (ctypes.c_uint8 * n.value)()
    _check(lib().pkv_descriptor_encode(arr, len(desc), out, n.value, ctypes.byref(n)))
    return bytes(out)


def pkv_descriptor_digest(desc) -> bytes:
    arr, _keep = _fields(desc)
    out = (ctypes.c_uint8 * 16)()
    _check(lib().pkv_descriptor_digest(arr, len(desc), out))
    return bytes(out)


# ---- device -----------------------------------------------------------------------------------

def pkv_digest_batch(pool, msg_off, msg_len, digests, status, stream=None):
    import torch
    _check(lib().pkv_digest_batch(_ptr(pool, torch.uint8), pool.numel(), _ptr(msg_off, torch.int64),
                                  _ptr(msg_len, torch.int32), msg_off.numel(), _ptr(digests, torch.uint8),
                                  _ptr(status, torch.int32), _stream(stream)))


def pkv_expand_digests(desc_digests, desc_idx, digests, status, stream=None):
    """digests[r] = desc_digests[desc_idx[r]] (desc_idx: int32 tensor holding uint32 indices)."""
    import torch
    _check(lib().pkv_expand_digests(_ptr(desc_digests, torch.uint8), desc_digests.numel() // 16,
                                    _ptr(desc_idx, torch.int32), desc_idx.numel(), _ptr(digests, torch.uint8),
                                    _ptr(status, torch.int32), _stream(stream)))


def pkv_key_offsets(tok_off, block, key_off, stream=None):
    import torch
    _check(lib().pkv_key_offsets(_ptr(tok_off, torch.int64), tok_off.numel() - 1, block,
                                 _ptr(key_off, torch.int64), _stream(stream)))


def pkv_derive_keys(tokens, tok_off, digests, block, key_off, keys, status, stream=None):
    import torch
    _check(lib().pkv_derive_keys(_ptr(tokens, torch.int32), tokens.numel(), _ptr(tok_off, torch.int64),
                                 tok_off.numel() - 1, _ptr(digests, torch.uint8), block,
                                 _ptr(key_off, torch.int64), keys.numel() // 16, _ptr(keys, torch.uint8),
                                 _ptr(status, torch.int32), _stream(stream)))


class Table:
    """Device memory of one index: ``slots`` uint8 [pkv_table_bytes(capacity)] (128-byte buckets of
    four slots, see include/pkv.h); with ``epochs=True`` also ``epochs`` int32 [capacity] (the
    fixed-budget tier) and the eviction work area."""

    def __init__(self, capacity: int, device="cuda", init=True, stream=None, epochs=False):
        import torch
        nbytes = int(lib().pkv_table_bytes(capacity))
        if nbytes == 0:
            raise ValueError("capacity must be a power of two in [4, 2^56]")
        self.capacity = capacity
        # torch's caching allocator hands out blocks aligned to at least 512 bytes
        self.slots = torch.empty(nbytes, dtype=torch.uint8, device=device)
        if self.slots.data_ptr() % 128:
            raise RuntimeError("index memory is not 128-byte aligned")
        self.epochs = torch.zeros(capacity, dtype=torch.int32, device=device) if epochs else None
        self.work = torch.empty(EVICT_WORK_BYTES // 8, dtype=torch.int64, device=device) if epochs else None
        if init:
            pkv_table_init(self, stream)

    def struct(self) -> pkv_table:
        return pkv_table(self.slots.data_ptr(), self.capacity)

    def copy_from(self, other: "Table"):
        self.slots.copy_(other.slots)
        if self.epochs is not None and other.epochs is not None:
            self.epochs.copy_(other.epochs)


def pkv_table_init(table: Table, stream=None):
    t = table.struct()
    _check(lib().pkv_table_init(ctypes.byref(t), _stream(stream)))


def pkv_lookup_prefix(table: Table, keys, key_off, hits, status, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_lookup_prefix(ctypes.byref(t), _ptr(keys, torch.uint8), _ptr(key_off, torch.int64),
                                   key_off.numel() - 1, keys.numel() // 16, _ptr(hits, torch.int32),
                                   _ptr(status, torch.int32), _stream(stream)))


def pkv_derive_lookup(tokens, tok_off, digests, block, key_off, keys, table: Table, hits, status, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_derive_lookup(_ptr(tokens, torch.int32), tokens.numel(), _ptr(tok_off, torch.int64),
                                   tok_off.numel() - 1, _ptr(digests, torch.uint8), block,
                                   _ptr(key_off, torch.int64), keys.numel() // 16, _ptr(keys, torch.uint8),
                                   ctypes.byref(t), _ptr(hits, torch.int32), _ptr(status, torch.int32),
                                   _stream(stream)))


def pkv_store(table: Table, keys, key_off, hits, locs, n_new, status, new_slots=None, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_store(ctypes.byref(t), _ptr(keys, torch.uint8), _ptr(key_off, torch.int64),
                           key_off.numel() - 1, keys.numel() // 16, _ptr(hits, torch.int32),
                           _ptr(locs, torch.int64), _ptr(new_slots, torch.int64), _ptr(n_new, torch.int64),
                           _ptr(status, torch.int32), _stream(stream)))


def pkv_table_rollback(table: Table, new_slots, n_new, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_table_rollback(ctypes.byref(t), _ptr(new_slots, torch.int64), _ptr(n_new, torch.int64),
                                    new_slots.numel(), _stream(stream)))


def pkv_table_export(table: Table, keys_out, locs_out, count, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_table_export(ctypes.byref(t), _ptr(keys_out, torch.uint8), _ptr(locs_out, torch.int64),
                                  _ptr(count, torch.int64), _stream(stream)))


def pkv_lookup_prefix_touch(table: Table, keys, key_off, epoch: int, hits, status, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_lookup_prefix_touch(ctypes.byref(t), _ptr(keys, torch.uint8), _ptr(key_off, torch.int64),
                                         key_off.numel() - 1, keys.numel() // 16, _ptr(table.epochs, torch.int32),
                                         epoch, _ptr(hits, torch.int32), _ptr(status, torch.int32), _stream(stream)))


def pkv_store_touch(table: Table, keys, key_off, hits, locs, n_new, status, epoch: int, new_slots=None,
                    stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_store_touch(ctypes.byref(t), _ptr(keys, torch.uint8), _ptr(key_off, torch.int64),
                                 key_off.numel() - 1, keys.numel() // 16, _ptr(hits, torch.int32),
                                 _ptr(locs, torch.int64), _ptr(new_slots, torch.int64), _ptr(n_new, torch.int64),
                                 _ptr(table.epochs, torch.int32), epoch, _ptr(status, torch.int32),
                                 _stream(stream)))


def pkv_table_evict(table: Table, budget: int, n_evicted, stream=None):
    import torch
    t = table.struct()
    _check(lib().pkv_table_evict(ctypes.byref(t), _ptr(table.epochs, torch.int32), budget,
                                 _ptr(table.work, torch.int64), _ptr(n_evicted, torch.int64), _stream(stream)))


class pkv_tensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("name_len", ctypes.c_uint32), ("dtype", ctypes.c_char_p),
                ("dtype_len", ctypes.c_uint32), ("shape", ctypes.POINTER(ctypes.c_uint64)), ("ndim", ctypes.c_uint32),
                ("nbytes", ctypes.c_uint64), ("root", ctypes.c_char_p)]


def pkv_tree_work_bytes(n_bytes: int, n_tensors: int) -> int:
    return int(lib().pkv_tree_work_bytes(n_bytes, n_tensors))


def pkv_tensor_roots(data, tensor_off, tensor_len, work, roots, status, stream=None):
    import torch
    _check(lib().pkv_tensor_roots(_ptr(data, torch.uint8), data.numel(), _ptr(tensor_off, torch.int64),
                                  _ptr(tensor_len, torch.int64), tensor_off.numel(), _ptr(work),
                                  work.numel() * work.element_size(), _ptr(roots, torch.uint8),
                                  _ptr(status, torch.int32), _stream(stream)))


def pkv_tensor_roots_static(data, tensor_off, tensor_len, roots, status, stream=None):
    """pkv_tensor_roots without a work area argument: the library's per-device buffer is used."""
    import torch
    _check(lib().pkv_tensor_roots_static(_ptr(data, torch.uint8), data.numel(), _ptr(tensor_off, torch.int64),
                                         _ptr(tensor_len, torch.int64), tensor_off.numel(), _ptr(roots, torch.uint8),
                                         _ptr(status, torch.int32), _stream(stream)))


def pkv_content_identity(tensors, config=()) -> bytes:
    """tensors: (name, dtype, shape, nbytes, root) tuples (bytes, bytes, ints, int, 32 bytes)."""
    arr = (pkv_tensor * max(1, len(tensors)))()
    keep = []
    for i, (name, dtype, shape, nbytes, root) in enumerate(tensors):
        name, dtype, root = bytes(name), bytes(dtype), bytes(root)
        shp = (ctypes.c_uint64 * max(1, len(shape)))(*[int(d) for d in shape])
        keep += [name, dtype, root, shp]
        arr[i] = pkv_tensor(name, len(name), dtype, len(dtype), shp, len(shape), int(nbytes), root)
    cfg, keep2 = _fields(config)
    out = (ctypes.c_uint8 * 32)()
    _check(lib().pkv_content_identity(arr, len(tensors), cfg, len(config), out))
    return bytes(out)


def pkv_sum_hits(hits, group_off, sums, status, stream=None):
    import torch
    _check(lib().pkv_sum_hits(_ptr(hits, torch.int32), hits.numel(), _ptr(group_off, torch.int64),
                              group_off.numel() - 1, _ptr(sums, torch.int64), _ptr(status, torch.int32),
                              _stream(stream)))


def version() -> str:
    return lib().pkv_version().decode()
