"""Seeded synthetic workloads: five request-batch recipes with prefix sharing and provenance mixes.

The paper measures on live serving engines with public prompt datasets (section 4.1); those
are not available here, so every batch below is synthetic.  Each recipe reproduces the
shape of one workload: request count, tokens per request, block size, how prefixes are
shared, and how many provenance descriptors are mixed.

Conventions (data only, no hashing):
  * tokens are int32 ids, requests concatenated; ``tok_off[r]..tok_off[r+1]`` is request r;
  * a descriptor is a list of ``(name, value)`` byte pairs in an arbitrary (shuffled) order:
    the canonical order is the encoder's job, so the generator deliberately scrambles it;
  * integers are 8-byte little-endian values, strings are ASCII, salts are 8 raw bytes;
  * the location stored for key j (0-based) of request r is ``tag<<56 | r<<32 | j``.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

CORE_NAMES = (b"model_id", b"adapter_id", b"weight_dtype", b"weight_version", b"kv_format", b"salt")

SEEDS = {"tiny": 0x5EED0001, "c2": 0x5EED0002, "c3": 0x5EED0003, "c4": 0x5EED0004, "c5": 0x5EED0005,
         "omission": 0x5EED0007, "omission-tiny": 0x5EED0008}

TAG_STEP, TAG_FILL, TAG_WARMUP = 0, 1, 2


@dataclass
class Batch:
    tokens: np.ndarray          # int32 [total tokens]
    tok_off: np.ndarray         # int64 [n_req + 1]
    block: int                  # tokens per keyed block
    descs: list                 # list of descriptors, each a list of (name, value) byte pairs
    desc_idx: np.ndarray        # int32 [n_req]: descriptor of each request
    tag: int = TAG_STEP         # location tag
    meta: dict = field(default_factory=dict)

    @property
    def n_req(self) -> int:
        return int(self.tok_off.shape[0] - 1)

    def request_descs(self):
        return [self.descs[i] for i in self.desc_idx]


@dataclass
class Workload:
    name: str
    seed: int
    capacity: int               # index slots (power of two)
    batch: Batch                # the batch one step processes
    fill: Optional[Batch] = None    # stored (every block, zero hits) before the run
    warmup: Optional[Batch] = None  # derived, looked up and stored before the timed batch
    meta: dict = field(default_factory=dict)


def locations(key_off: np.ndarray, tag: int) -> np.ndarray:
    """uint64 location per key: ``tag<<56 | r<<32 | j`` for key j (0-based) of request r."""
    key_off = np.asarray(key_off, dtype=np.int64)
    n = np.diff(key_off)
    r = np.repeat(np.arange(n.shape[0], dtype=np.uint64), n)
    j = (np.arange(int(key_off[-1]), dtype=np.int64) - np.repeat(key_off[:-1], n)).astype(np.uint64)
    return (np.uint64(tag) << np.uint64(56)) | (r << np.uint64(32)) | j


# ----------------------------------------------------------------------------- helpers

def _streams(seed: int, k: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(k)]


def _u64(v: int) -> bytes:
    return int(v).to_bytes(8, "little")


def _shuffled(fields, g):
    order = g.permutation(len(fields))
    return [fields[i] for i in order]


def _ragged(chunks):
    """Concatenate int32 arrays; return (tokens, int64 offsets)."""
    lens = np.array([c.shape[0] for c in chunks], dtype=np.int64)
    off = np.zeros(lens.shape[0] + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    tokens = np.concatenate(chunks).astype(np.int32, copy=False) if chunks else np.zeros(0, np.int32)
    return tokens, off


def _full_blocks(n_tokens, block):
    # Number of complete blocks of a token run: used only to size filler so the index reaches
    # an exact entry count.
    return np.asarray(n_tokens, dtype=np.int64) // block


def _filler_offsets(n_keys, chain_blocks, block):
    """Offsets of random-token chains holding exactly ``n_keys`` full blocks (last one shorter)."""
    full, rem = divmod(int(n_keys), chain_blocks)
    lens = np.full(full + (1 if rem else 0), chain_blocks * block, dtype=np.int64)
    if rem:
        lens[-1] = rem * block
    off = np.zeros(lens.shape[0] + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    return off


def _random_into(g, out, vocab, chunk=1 << 24):
    for a in range(0, out.shape[0], chunk):
        b = min(out.shape[0], a + chunk)
        out[a:b] = g.integers(0, vocab, size=b - a, dtype=np.int32)


def _concat_batches(parts, block, descs, tag, meta=None, filler=None):
    """parts: list of (tokens, tok_off, desc_idx).  ``filler`` = (generator, tok_off, desc_idx,
    vocab): random chains generated straight into the output buffer."""
    total = sum(int(o[-1]) for _, o, _ in parts) + (int(filler[1][-1]) if filler else 0)
    tokens = np.empty(total, dtype=np.int32)
    offs, idxs = [np.zeros(1, np.int64)], []
    base = 0
    for t, o, d in parts:
        tokens[base: base + int(o[-1])] = t
        offs.append(o[1:] + base)
        idxs.append(np.asarray(d, dtype=np.int32))
        base += int(o[-1])
    if filler:
        g, fo, fd, vocab = filler
        _random_into(g, tokens[base:], vocab)
        offs.append(fo[1:] + base)
        idxs.append(np.asarray(fd, dtype=np.int32))
    return Batch(tokens, np.concatenate(offs), block, descs, np.concatenate(idxs), tag, meta or {})


# ----------------------------------------------------------------------------- recipes

def make_tiny(seed=SEEDS["tiny"]) -> Workload:
    """8 requests x 256 tokens in [0, 32000), block 16, six-dimension descriptors drawn per
    request; 1024 slots pre-filled with every key of requests 0-3."""
    g_tok, g_desc, g_ord = _streams(seed, 3)
    n_req, length, block = 8, 256, 16
    tokens = g_tok.integers(0, 32000, size=n_req * length, dtype=np.int32)
    tok_off = np.arange(n_req + 1, dtype=np.int64) * length
    adapters = [b"adapter-" + g_desc.bytes(4).hex().encode() for _ in range(2)]
    dtypes = [b"bfloat16", b"float8_e4m3fn"]
    kv = [b"bfloat16", b"fp8_e4m3"]
    descs = []
    for _ in range(n_req):
        descs.append([(b"model_id", b"m0"),
                      (b"adapter_id", adapters[int(g_desc.integers(2))]),
                      (b"weight_dtype", dtypes[int(g_desc.integers(2))]),
                      (b"weight_version", _u64(1 + int(g_desc.integers(2)))),
                      (b"kv_format", kv[int(g_desc.integers(2))]),
                      (b"salt", g_desc.bytes(8))])
    batch = Batch(tokens, tok_off, block, [_shuffled(d, g_ord) for d in descs],
                  np.arange(n_req, dtype=np.int32), TAG_STEP)
    # The fill presents the same descriptors with a different field order: keys must not change.
    fill = Batch(tokens[: 4 * length].copy(), tok_off[:5].copy(), block,
                 [_shuffled(d, g_ord) for d in descs[:4]], np.arange(4, dtype=np.int32), TAG_FILL)
    full = length // block
    return Workload("tiny", seed, 1 << 10, batch, fill=fill,
                    meta={"expect_first": [full] * 4 + [0] * 4, "expect_second": [full] * n_req})


def make_c2(seed=SEEDS["c2"]) -> Workload:
    """1024 requests x 2048 tokens, vocab 128256, block 16.  Each request = one of 64 shared
    prefixes (512-1536 tokens) + a random suffix.  32 provenance classes = 8 adapters x
    {bfloat16, float8} weights x 2 salts.  4M-slot index at load 0.5: the 64 prefixes under the
    16 bfloat16 classes plus filler chains under another model id."""
    g_pre, g_req, g_desc, g_ord, g_fill = _streams(seed, 5)
    n_req, length, block, vocab = 1024, 2048, 16, 128256
    capacity, target = 1 << 22, 1 << 21
    pre_len = g_pre.integers(512, 1536, size=64, endpoint=True)
    prefixes = [g_pre.integers(0, vocab, size=int(n), dtype=np.int32) for n in pre_len]
    pid = g_req.integers(0, 64, size=n_req)
    tok = g_req.integers(0, vocab, size=(n_req, length), dtype=np.int32)
    for r in range(n_req):
        tok[r, : pre_len[pid[r]]] = prefixes[pid[r]]
    adapters = [b"lora-" + g_desc.bytes(6).hex().encode() for _ in range(8)]
    salts = [g_desc.bytes(8) for _ in range(2)]
    dtypes = [b"bfloat16", b"float8_e4m3fn"]
    classes = []          # class index = a*4 + d*2 + s
    for a in range(8):
        for d in range(2):
            for s in range(2):
                classes.append(_shuffled([(b"model_id", b"synthetic-8b"), (b"adapter_id", adapters[a]),
                                          (b"weight_dtype", dtypes[d]), (b"weight_version", _u64(3)),
                                          (b"kv_format", b"bfloat16"), (b"salt", salts[s])], g_ord))
    cls = g_req.integers(0, 32, size=n_req).astype(np.int32)
    batch = Batch(tok.reshape(-1), np.arange(n_req + 1, dtype=np.int64) * length, block, classes, cls,
                  TAG_STEP, {"prefix_len": pre_len[pid], "prefix_id": pid,
                             "bf16": ((cls // 2) % 2 == 0)})
    # Index fill: every prefix under every bfloat16 class, then filler to exactly 2^21 entries.
    bf16_classes = [c for c in range(32) if (c // 2) % 2 == 0]
    pre_chunks, pre_desc = [], []
    for p in range(64):
        for c in bf16_classes:
            pre_chunks.append(prefixes[p])
            pre_desc.append(c)
    pt, po = _ragged(pre_chunks)
    n_prefix_keys = int(_full_blocks(pre_len, block).sum()) * len(bf16_classes)
    filler_descs = [_shuffled([(b"model_id", b"filler-model"), (b"adapter_id", b"filler-%d" % i),
                               (b"weight_dtype", b"bfloat16"), (b"weight_version", _u64(1)),
                               (b"kv_format", b"bfloat16")], g_ord) for i in range(4)]
    fo = _filler_offsets(target - n_prefix_keys, length // block, block)
    fdesc = 32 + (np.arange(fo.shape[0] - 1) % 4)
    fill = _concat_batches([(pt, po, pre_desc)], block, classes + filler_descs, TAG_FILL,
                           {"entries": target}, filler=(g_fill, fo, fdesc, vocab))
    return Workload("c2", seed, capacity, batch, fill=fill, meta={"fill_entries": target})


def _c3_batch(g, n_req, length, vocab, prefixes, pre_len, zipf_p, rank_to_prefix, n_desc):
    rank = g.choice(len(zipf_p), size=n_req, p=zipf_p)
    pid = rank_to_prefix[rank]
    tok = g.integers(0, vocab, size=(n_req, length), dtype=np.int32)
    for r in range(n_req):
        tok[r, : pre_len[pid[r]]] = prefixes[pid[r]]
    didx = g.integers(0, n_desc, size=n_req).astype(np.int32)
    return tok.reshape(-1), pid, didx


def make_c3(seed=SEEDS["c3"]) -> Workload:
    """Chunked keying: 4096 requests x 8192 tokens, chunk 256.  Prefix popularity Zipf s=1.1
    over 512 prefixes of 1024-6144 tokens; 16 six-dimension descriptors.  2^19 slots, empty; an
    untimed warm-up batch from the same distribution is stored first."""
    g_pre, g_desc, g_ord, g_warm, g_main = _streams(seed, 5)
    n_req, length, block, vocab, n_pre = 4096, 8192, 256, 128256, 512
    pre_len = g_pre.integers(1024, 6144, size=n_pre, endpoint=True)
    prefixes = [g_pre.integers(0, vocab, size=int(n), dtype=np.int32) for n in pre_len]
    ranks = np.arange(1, n_pre + 1, dtype=np.float64)
    zipf_p = ranks ** -1.1
    zipf_p /= zipf_p.sum()
    rank_to_prefix = g_pre.permutation(n_pre)
    dtypes = [b"bfloat16", b"float16", b"float8_e4m3fn"]
    kv = [b"bfloat16", b"fp8_e4m3", b"fp8_e5m2"]
    descs = []
    for i in range(16):
        descs.append(_shuffled([(b"model_id", b"synthetic-70b"),
                                (b"adapter_id", b"adapter-" + g_desc.bytes(4).hex().encode()),
                                (b"weight_dtype", dtypes[int(g_desc.integers(3))]),
                                (b"weight_version", _u64(int(g_desc.integers(1, 5)))),
                                (b"kv_format", kv[int(g_desc.integers(3))]),
                                (b"salt", g_desc.bytes(8))], g_ord))
    off = np.arange(n_req + 1, dtype=np.int64) * length
    wt, wp, wd = _c3_batch(g_warm, n_req, length, vocab, prefixes, pre_len, zipf_p, rank_to_prefix, 16)
    mt, mp, md = _c3_batch(g_main, n_req, length, vocab, prefixes, pre_len, zipf_p, rank_to_prefix, 16)
    warm = Batch(wt, off.copy(), block, descs, wd, TAG_WARMUP, {"prefix_id": wp, "prefix_len": pre_len[wp]})
    main = Batch(mt, off.copy(), block, descs, md, TAG_STEP, {"prefix_id": mp, "prefix_len": pre_len[mp]})
    return Workload("c3", seed, 1 << 19, main, warmup=warm)


def _fresh(g, old: bytes) -> bytes:
    while True:
        v = g.bytes(8)
        if v != old:
            return v


def make_c4(seed=SEEDS["c4"], filler=True) -> Workload:
    """Lookup-heavy: 16384 requests x 4096 tokens, block 16, 20 registered dimensions (6 core +
    14 extras), 64 base descriptors.  70% of requests have their own chain stored for L ~ U[1,256]
    blocks; 30% have the same tokens stored under a descriptor differing in exactly one dimension.
    Filler chains bring the 64M-slot index to exactly 2^25 entries (load 0.5).

    ``filler=False`` leaves the filler out (the same requests and prefixes; used for small checks)."""
    g_desc, g_ord, g_req, g_var, g_fill = _streams(seed, 5)
    n_req, length, block, vocab = 16384, 4096, 16, 128256
    capacity, target = 1 << 26, 1 << 25
    extras = [b"x%02d" % i for i in range(14)]
    dtypes = [b"bfloat16", b"float16", b"float8_e4m3fn", b"int4-awq"]
    kv = [b"bfloat16", b"float16", b"fp8_e4m3", b"fp8_e5m2"]

    def base_desc():
        f = [(b"model_id", b"model-" + g_desc.bytes(3).hex().encode()),
             (b"adapter_id", b"adapter-" + g_desc.bytes(4).hex().encode()),
             (b"weight_dtype", dtypes[int(g_desc.integers(4))]),
             (b"weight_version", _u64(int(g_desc.integers(1, 1 << 20)))),
             (b"kv_format", kv[int(g_desc.integers(4))]),
             (b"salt", g_desc.bytes(8))]
        f += [(x, g_desc.bytes(8)) for x in extras]
        return f

    base = [base_desc() for _ in range(64)]
    didx = g_req.integers(0, 64, size=n_req).astype(np.int32)
    tok = g_req.integers(0, vocab, size=(n_req, length), dtype=np.int32)
    own = np.zeros(n_req, dtype=bool)
    own[g_req.permutation(n_req)[: int(round(0.7 * n_req))]] = True
    stored_blocks = g_req.integers(1, length // block, size=n_req, endpoint=True)
    var_dim = np.full(n_req, -1, dtype=np.int32)
    descs = [_shuffled(d, g_ord) for d in base]
    fill_desc = np.empty(n_req, dtype=np.int32)
    for r in range(n_req):
        if own[r]:
            fill_desc[r] = didx[r]
            continue
        d = list(base[didx[r]])
        k = int(g_var.integers(20))
        var_dim[r] = k
        d[k] = (d[k][0], _fresh(g_var, d[k][1]))
        fill_desc[r] = len(descs)
        descs.append(_shuffled(d, g_ord))
    batch = Batch(tok.reshape(-1), np.arange(n_req + 1, dtype=np.int64) * length, block, descs[:64], didx,
                  TAG_STEP, {"own": own, "stored_blocks": stored_blocks, "var_dim": var_dim})
    pre_chunks = [tok[r, : stored_blocks[r] * block] for r in range(n_req)]
    pt, po = _ragged(pre_chunks)
    parts = [(pt, po, fill_desc)]
    fill_spec = None
    if filler:
        filler_descs = []
        for i in range(8):
            d = base_desc()
            d[0] = (b"model_id", b"filler-model-%d" % i)
            filler_descs.append(_shuffled(d, g_ord))
        n_fill_desc = len(descs)
        descs = descs + filler_descs
        fo = _filler_offsets(target - int(stored_blocks.sum()), length // block, block)
        fill_spec = (g_fill, fo, n_fill_desc + (np.arange(fo.shape[0] - 1) % 8), vocab)
    fill = _concat_batches(parts, block, descs, TAG_FILL, {"entries": target if filler else None},
                           filler=fill_spec)
    return Workload("c4", seed, capacity, batch, fill=fill,
                    meta={"fill_entries": target if filler else int(stored_blocks.sum())})


def make_c5(seed=SEEDS["c5"]) -> Workload:
    """Long context: 256 requests x 131072 tokens, block 16.  64 groups of 4 share a base
    sequence up to a uniform fork point; 64 descriptors = 2 adapters x 2 dtypes x 2 versions x
    2 KV formats x 4 salts, one per group.  2^22 slots, empty: derive, lookup, store, lookup."""
    g_seq, g_desc, g_ord = _streams(seed, 3)
    n_req, length, block, vocab = 256, 131072, 16, 128256
    adapters = [b"adapter-" + g_desc.bytes(4).hex().encode() for _ in range(2)]
    dtypes = [b"bfloat16", b"float8_e4m3fn"]
    kv = [b"bfloat16", b"fp8_e4m3"]
    salts = [g_desc.bytes(8) for _ in range(4)]
    combos = []
    for a in range(2):
        for d in range(2):
            for v in range(2):
                for k in range(2):
                    for s in range(4):
                        combos.append(_shuffled([(b"model_id", b"synthetic-long"), (b"adapter_id", adapters[a]),
                                                 (b"weight_dtype", dtypes[d]), (b"weight_version", _u64(v + 1)),
                                                 (b"kv_format", kv[k]), (b"salt", salts[s])], g_ord))
    group_desc = g_desc.permutation(64).astype(np.int32)
    tok = np.empty((n_req, length), dtype=np.int32)
    fork = g_seq.integers(0, length, size=n_req, endpoint=True)
    for grp in range(64):
        base_seq = g_seq.integers(0, vocab, size=length, dtype=np.int32)
        for m in range(4):
            r = 4 * grp + m
            tok[r] = g_seq.integers(0, vocab, size=length, dtype=np.int32)
            tok[r, : fork[r]] = base_seq[: fork[r]]
    didx = np.repeat(group_desc, 4)
    full = length // block
    batch = Batch(tok.reshape(-1), np.arange(n_req + 1, dtype=np.int64) * length, block, combos, didx,
                  TAG_STEP, {"fork": fork, "group": np.arange(n_req) // 4})
    return Workload("c5", seed, 1 << 22, batch,
                    meta={"expect_first": [0] * n_req, "expect_second": [full] * n_req})


WORKLOADS = {"tiny": make_tiny, "c2": make_c2, "c3": make_c3, "c4": make_c4, "c5": make_c5}


# ---- differential omission test inputs (section 5.4, Eq. 4) -------------------------------------

@dataclass
class OmissionCase:
    """Inputs of one differential omission test: fixed token sequences x, base configurations c,
    one replacement value v' per registered dimension, the declared effect of varying each
    dimension, and the key bindings to test.

    ``bindings`` is a list of ``(label, names)``: ``names`` is the set of dimension names the key
    binds (``None`` = every field of the descriptor, an empty set = a token-only key)."""
    batch: Batch                # tokens, request offsets, block, base descriptors, desc_idx
    dims: list                  # registered dimension names, in report order
    variants: dict              # name -> replacement value v' (differs from every base value)
    changes: dict               # name -> True if varying it changes KV state or sharing permission
    bindings: list              # [(label, frozenset of names or None)]
    name: str = "omission"


def make_omission(seed=SEEDS["omission"], n_req=512, length=1024, block=16, n_base=64, n_extra=14,
                  name="omission") -> OmissionCase:
    """A registry of 6 core + ``n_extra`` further dimensions (8-byte values), ``n_base`` base
    descriptors over it, ``n_req`` random token sequences of ``length`` tokens.  Bindings: the
    complete registry, each leave-one-dimension-out projection, and the token-only key.  Every
    dimension is declared to change state or sharing permission (the salt changes permission
    only; the others change the computed state)."""
    g_desc, g_ord, g_tok, g_var = _streams(seed, 4)
    extras = [b"x%02d" % i for i in range(n_extra)]
    dims = list(CORE_NAMES) + extras
    dtypes = [b"bfloat16", b"float16", b"float8_e4m3fn"]
    kv = [b"bfloat16", b"fp8_e4m3"]

    def base_desc():
        f = [(b"model_id", b"model-" + g_desc.bytes(3).hex().encode()),
             (b"adapter_id", b"adapter-" + g_desc.bytes(4).hex().encode()),
             (b"weight_dtype", dtypes[int(g_desc.integers(len(dtypes)))]),
             (b"weight_version", _u64(int(g_desc.integers(1, 1 << 20)))),
             (b"kv_format", kv[int(g_desc.integers(len(kv)))]),
             (b"salt", g_desc.bytes(8))]
        f += [(x, g_desc.bytes(8)) for x in extras]
        return f

    base = [base_desc() for _ in range(n_base)]
    variants = {}
    for d in dims:
        taken = {v for desc in base for n, v in desc if n == d}
        while True:
            v = b"variant-" + g_var.bytes(8)
            if v not in taken:
                variants[d] = v
                break
    didx = g_tok.integers(0, n_base, size=n_req).astype(np.int32)
    tok = g_tok.integers(0, 128256, size=n_req * length, dtype=np.int32)
    batch = Batch(tok, np.arange(n_req + 1, dtype=np.int64) * length, block,
                  [_shuffled(d, g_ord) for d in base], didx, TAG_STEP)
    bindings = [("complete", None)]
    bindings += [("without " + d.decode(), frozenset(x for x in dims if x != d)) for d in dims]
    bindings += [("token-only", frozenset())]
    return OmissionCase(batch, dims, variants, {d: True for d in dims}, bindings, name)


def make_omission_tiny(seed=SEEDS["omission-tiny"]) -> OmissionCase:
    """Small case for parity tests: 12 requests of 100..200 tokens (ragged tails), 2 extras."""
    case = make_omission(seed, n_req=12, length=160, n_base=5, n_extra=2, name="omission-tiny")
    g = np.random.default_rng(seed)
    lens = g.integers(100, 201, size=12)
    toks = [case.batch.tokens[r * 160:(r + 1) * 160] for r in range(12)]
    toks = [np.concatenate([t, g.integers(0, 128256, size=max(0, n - 160), dtype=np.int32)])[:n]
            for t, n in zip(toks, lens)]
    t, o = _ragged(toks)
    case.batch = Batch(t, o, 16, case.batch.descs, case.batch.desc_idx, TAG_STEP)
    return case


OMISSION_CASES = {"omission": make_omission, "omission-tiny": make_omission_tiny}


# ---- fixed-budget tier inputs (section 6.5: retention against provenance diversity) -------------

SEEDS["budget"] = 0x5EED0009


def make_budget(classes=8, n_batches=8, seed=SEEDS["budget"], n_req=1024, length=2048, n_prefix=64):
    """A stream of request batches for a fixed-budget tier: every batch has ``n_req`` requests of
    ``length`` tokens, each one of ``n_prefix`` shared prefixes (512-1536 tokens, shared by all
    batches) plus a fresh random suffix, under one of ``classes`` provenance classes (adapter
    identities) drawn uniformly.  Returns (batches, capacity, budget): a 1M-slot index with a
    budget of 2^18 entries."""
    g_pre, g_req, g_desc, g_ord = _streams(seed, 4)
    block, vocab = 16, 128256
    pre_len = g_pre.integers(512, 1536, size=n_prefix, endpoint=True)
    prefixes = [g_pre.integers(0, vocab, size=int(n), dtype=np.int32) for n in pre_len]
    descs = [_shuffled([(b"model_id", b"synthetic-8b"), (b"adapter_id", b"lora-" + g_desc.bytes(6).hex().encode()),
                        (b"weight_dtype", b"bfloat16"), (b"weight_version", _u64(3)), (b"kv_format", b"bfloat16"),
                        (b"salt", b"tenant-shared")], g_ord) for _ in range(classes)]
    batches = []
    for t in range(n_batches):
        pid = g_req.integers(0, n_prefix, size=n_req)
        tok = g_req.integers(0, vocab, size=(n_req, length), dtype=np.int32)
        for r in range(n_req):
            tok[r, : pre_len[pid[r]]] = prefixes[pid[r]]
        cls = g_req.integers(0, classes, size=n_req).astype(np.int32)
        batches.append(Batch(tok.reshape(-1), np.arange(n_req + 1, dtype=np.int64) * length, block, descs, cls,
                             TAG_STEP + 8 + t, {"prefix_blocks": _full_blocks(pre_len[pid], block)}))
    return batches, 1 << 20, 1 << 18


def make_workload(name: str, **kw) -> Workload:
    return WORKLOADS[name](**kw)


# ---- content identities (section 5.3 adapter identity from contents; section 6.5 startup costs) ----

def identity_shapes(kind="adapter"):
    """Tensor names, dtypes and shapes of the two objects section 6.5 times: a LoRA adapter of about
    40 MB (rank 8 on the seven projections of 28 layers of a 7B-class model, bfloat16) and a
    checkpoint of about 0.5 B parameters (24 layers, hidden 896, MLP 4864, vocabulary 151936,
    bfloat16).  Only shapes: the bytes are drawn from a seeded generator by the caller."""
    out = []
    if kind == "adapter":
        h, f, r = 4096, 14336, 8
        mods = {"q_proj": (h, h), "k_proj": (h, 1024), "v_proj": (h, 1024), "o_proj": (h, h),
                "gate_proj": (h, f), "up_proj": (h, f), "down_proj": (f, h)}
        for layer in range(28):
            for m, (din, dout) in mods.items():
                base = f"base_model.model.layers.{layer}.{m}"
                out.append((f"{base}.lora_A.weight".encode(), b"bfloat16", (r, din)))
                out.append((f"{base}.lora_B.weight".encode(), b"bfloat16", (dout, r)))
    elif kind == "checkpoint":
        h, f, v, kvd = 896, 4864, 151936, 128
        out.append((b"model.embed_tokens.weight", b"bfloat16", (v, h)))
        for layer in range(24):
            base = f"model.layers.{layer}"
            for name, shape in [("self_attn.q_proj.weight", (h, h)), ("self_attn.q_proj.bias", (h,)),
                                ("self_attn.k_proj.weight", (kvd, h)), ("self_attn.k_proj.bias", (kvd,)),
                                ("self_attn.v_proj.weight", (kvd, h)), ("self_attn.v_proj.bias", (kvd,)),
                                ("self_attn.o_proj.weight", (h, h)), ("mlp.gate_proj.weight", (f, h)),
                                ("mlp.up_proj.weight", (f, h)), ("mlp.down_proj.weight", (h, f)),
                                ("input_layernorm.weight", (h,)), ("post_attention_layernorm.weight", (h,))]:
                out.append((f"{base}.{name}".encode(), b"bfloat16", shape))
        out.append((b"model.norm.weight", b"bfloat16", (h,)))
    else:
        raise ValueError(kind)
    return out
