"""The KV provenance contract's properties, checked on the oracle (Def. 1, Def. 2 / Eq. 1-2,
Eq. 3, Prop. 1, Eq. 4, and the binding patterns of section 6.1-6.2 and 6.5)."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from workloads import CORE_NAMES, make_workload, locations

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _keys(tokens_list, descs, block=16):
    off = np.zeros(len(tokens_list) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in tokens_list])
    toks = np.concatenate([np.asarray(t, np.int32) for t in tokens_list])
    digs = np.stack([np.frombuffer(oracle.digest(d), np.uint8) for d in descs])
    keys = oracle.derive(toks, off, digs, block)
    ko = oracle.key_offsets(off, block)
    return [keys[ko[r]:ko[r + 1]] for r in range(len(tokens_list))], ko, keys


BASE = [(b"model_id", b"synthetic-8b"), (b"adapter_id", b"lora-A"), (b"weight_dtype", b"bfloat16"),
        (b"weight_version", (7).to_bytes(8, "little")), (b"kv_format", b"bfloat16"), (b"salt", b"tenant-1"),
        (b"x00", b"rope-10000")]


def _with(desc, name, value):
    out = [(n, v) for n, v in desc if n != name]
    if value is not None:
        out.append((name, value))
    return out


@pytest.mark.parametrize("name", [n for n, _ in BASE])
@pytest.mark.parametrize("change", ["value", "absent"])
def test_one_dimension_change_changes_every_block_key(name, change):
    """Eq. 4, key half: vary only d_i; every block key must differ (no omission)."""
    rng = np.random.default_rng(11)
    toks = [rng.integers(0, 128256, size=16 * 40 + 5, dtype=np.int32)]
    new_value = None if change == "absent" else dict(BASE)[name] + b"'"
    (a,), _, _ = _keys(toks, [BASE])
    (b,), _, _ = _keys(toks, [_with(BASE, name, new_value)])
    assert a.shape == b.shape == (40, 16)
    assert all((a[i] != b[i]).any() for i in range(40))


def test_adding_an_absent_dimension_later_keeps_keys_prop1():
    """Prop. 1: registering a new dimension changes keys only where a request carries it."""
    rng = np.random.default_rng(12)
    toks = [rng.integers(0, 128256, size=16 * 8, dtype=np.int32)]
    (a,), _, _ = _keys(toks, [BASE])
    (b,), _, _ = _keys(toks, [BASE])                      # request does not carry "rope_base"
    (c,), _, _ = _keys(toks, [BASE + [(b"rope_base", b"500000")]])
    assert (a == b).all()
    assert all((a[i] != c[i]).any() for i in range(8))


def test_token_only_baseline_collides_exactly_where_provenance_is_erased():
    """Def. 1: with every dimension projected away (R = {}), equal tokens give equal keys whatever the
    configuration; the bound key separates them.  R = {model_id, kv_format} mimics a connector that
    keeps only those fields (section 3.2): keys collide iff the two projections agree."""
    rng = np.random.default_rng(13)
    toks = rng.integers(0, 128256, size=16 * 12, dtype=np.int32)
    other = toks.copy()
    other[16 * 5] += 1
    descs = [BASE, _with(BASE, b"adapter_id", b"lora-B"), _with(BASE, b"weight_dtype", b"float8_e4m3fn"),
             _with(BASE, b"salt", b"tenant-2"), _with(BASE, b"kv_format", b"fp8_e4m3"),
             _with(BASE, b"model_id", b"synthetic-70b")]
    token_only = [[] for _ in descs]
    ks, _, _ = _keys([toks] * len(descs), token_only)
    assert all((k == ks[0]).all() for k in ks)
    (ko,), _, _ = _keys([other], [[]])
    assert (ko[:5] == ks[0][:5]).all() and all((ko[i] != ks[0][i]).any() for i in range(5, 12))
    bound, _, _ = _keys([toks] * len(descs), descs)
    assert len({bound[i][0].tobytes() for i in range(len(descs))}) == len(descs)
    keep = (b"model_id", b"kv_format")
    proj = [[(n, v) for n, v in d if n in keep] for d in descs]
    pk, _, _ = _keys([toks] * len(descs), proj)
    for i in range(len(descs)):
        for j in range(len(descs)):
            same_proj = sorted(proj[i]) == sorted(proj[j])
            assert ((pk[i] == pk[j]).all()) == same_proj


def test_binding_pattern_same_provenance_hits_cross_provenance_misses():
    """Section 6.1: same provenance -> full-prefix hit; any single-dimension cross -> zero; all five
    dimensions differing -> zero."""
    rng = np.random.default_rng(14)
    toks = rng.integers(0, 128256, size=16 * 24, dtype=np.int32)
    (seed_keys,), ko, _ = _keys([toks], [BASE])
    idx = oracle.Index(1 << 12)
    assert idx.store(seed_keys, np.array([0, 24], np.int64), np.zeros(1, np.int32),
                     np.arange(24, dtype=np.uint64)) == 0
    readers = [BASE] + [_with(BASE, n, v + b"#") for n, v in BASE if n in CORE_NAMES[1:]]
    readers.append([(n, (v + b"#") if n in CORE_NAMES[1:] else v) for n, v in BASE])
    ks, ko, keys = _keys([toks] * len(readers), readers)
    hits = idx.lookup(keys, ko)
    assert hits.tolist() == [24] + [0] * (len(readers) - 1)


def test_table3_adapter_identity_is_content_not_handle():
    """Section 6.1 / Table 3 at descriptor level: the same adapter content reached through another path
    has the same identity (hit); content replaced in place is a new identity (safe miss); a different
    salt is isolated."""
    rng = np.random.default_rng(15)
    toks = rng.integers(0, 128256, size=16 * 10, dtype=np.int32)
    content_id = b"sha256:aa11"
    seeded = _with(BASE, b"adapter_id", content_id)
    (k0,), _, _ = _keys([toks], [seeded])
    idx = oracle.Index(1 << 10)
    idx.store(k0, np.array([0, 10], np.int64), np.zeros(1, np.int32), np.arange(10, dtype=np.uint64))
    cases = {"another path": _with(BASE, b"adapter_id", content_id),
             "replaced in place": _with(BASE, b"adapter_id", b"sha256:bb22"),
             "tenant salt": _with(_with(BASE, b"adapter_id", content_id), b"salt", b"tenant-9")}
    ks, ko, keys = _keys([toks] * 3, list(cases.values()))
    assert idx.lookup(keys, ko).tolist() == [10, 0, 0]


def test_storage_grows_linearly_with_provenance_classes():
    """Section 6.5: k provenance classes over the same tokens need k times the entries; the token-only
    key deduplicates them into one copy."""
    rng = np.random.default_rng(16)
    toks = rng.integers(0, 128256, size=16 * 20, dtype=np.int32)
    for k in range(1, 5):
        descs = [_with(BASE, b"weight_version", (i + 1).to_bytes(8, "little")) for i in range(k)]
        for bound in (True, False):
            ds = descs if bound else [[] for _ in descs]
            _, ko, keys = _keys([toks] * k, ds)
            idx = oracle.Index(1 << 10)
            assert idx.store(keys, ko, np.zeros(k, np.int32), locations(ko, 0)) == 0
            assert len(idx) == (20 * k if bound else 20)


def test_tiny_workload_closed_form():
    w = make_workload("tiny")
    b = w.batch
    ko = oracle.key_offsets(b.tok_off, b.block)
    keys = oracle.derive(b.tokens, b.tok_off, oracle.batch_digests(b), b.block)
    fko = oracle.key_offsets(w.fill.tok_off, w.fill.block)
    fkeys = oracle.derive(w.fill.tokens, w.fill.tok_off, oracle.batch_digests(w.fill), w.fill.block)
    idx = oracle.Index(w.capacity)
    assert idx.store(fkeys, fko, np.zeros(w.fill.n_req, np.int32), locations(fko, w.fill.tag)) == 0
    hits = idx.lookup(keys, ko)
    assert hits.tolist() == w.meta["expect_first"]
    assert idx.store(keys, ko, hits, locations(ko, b.tag)) == 0
    assert idx.lookup(keys, ko).tolist() == w.meta["expect_second"]
    assert len(idx) == 8 * 16


_CHILD = r"""
import json, os, sys, random
import numpy as np
sys.path.insert(0, os.environ["PKV_ROOT"])
import oracle
from workloads import make_workload
w = make_workload("tiny")
b = w.batch
rnd = random.Random(int(os.environ["SHUFFLE"]))
descs = [list(d) for d in b.descs]
for d in descs:
    rnd.shuffle(d)
digs = np.stack([np.frombuffer(oracle.digest(descs[i]), np.uint8) for i in b.desc_idx])
keys = oracle.derive(b.tokens, b.tok_off, digs, b.block)
print(json.dumps(keys.tobytes().hex()))
"""


def test_keys_are_stable_across_processes_and_field_order():
    """Section 5.1 well-formedness: identities are cross-worker stable.  Separate interpreter
    processes with different hash seeds and field orders derive identical keys."""
    outs = set()
    for seed, shuffle in [("0", 1), ("12345", 2), ("random", 3)]:
        env = dict(os.environ, PYTHONHASHSEED=seed, SHUFFLE=str(shuffle), PKV_ROOT=ROOT)
        r = subprocess.run([sys.executable, "-c", _CHILD], env=env, capture_output=True, text=True, check=True)
        outs.add(json.loads(r.stdout.strip().splitlines()[-1]))
    assert len(outs) == 1
