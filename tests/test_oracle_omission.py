"""Pins of the oracle's differential omission test (section 5.4, Eq. 4; section 6.4).

The pattern is fixed by construction: a binding that includes the varied dimension never lets the
two keys coincide; a binding that withholds it makes every block coincide; a token-only key
coincides everywhere.  A second pin recomputes the key equalities with the library SHA-256
(hashlib) on a tiny case, and a third checks the declared-change conjunct of Eq. 4."""

import hashlib
import struct

import numpy as np

import oracle
from oracle.omission import equal_blocks, omission_matrix, project, vary
from workloads import Batch, OmissionCase, make_omission_tiny


def test_binding_pattern_is_the_closed_form():
    case = make_omission_tiny()
    res = omission_matrix(case, threads=4)
    coll, blocks = res["collisions"], res["blocks"]
    assert blocks > 0
    for i, (label, names) in enumerate(case.bindings):
        for j, d in enumerate(case.dims):
            bound = names is None or d in names
            assert coll[i, j] == (0 if bound else blocks), (label, d)
    labels = [b[0] for b in case.bindings]
    assert (coll[labels.index("complete")] == 0).all()
    assert (coll[labels.index("token-only")] == blocks).all()
    assert (res["omission"] == (coll > 0)).all()


def _lib_keys(tokens, desc, block):
    d = hashlib.sha256(oracle.encode(desc)).digest()[:16]
    prev, out = bytes(16), []
    for i in range(len(tokens) // block):
        blk = struct.pack("<%di" % block, *[int(t) for t in tokens[i * block:(i + 1) * block]])
        prev = hashlib.sha256(prev + d + blk).digest()[:16]
        out.append(prev)
    return out


def test_equal_blocks_matches_library_sha256():
    rng = np.random.default_rng(3)
    reqs = [rng.integers(0, 1000, size=n, dtype=np.int32) for n in (0, 17, 40, 33)]
    off = np.zeros(5, np.int64)
    off[1:] = np.cumsum([r.shape[0] for r in reqs])
    toks = np.concatenate(reqs)
    a = [[(b"model_id", b"m"), (b"salt", b"s%d" % i)] for i in range(4)]
    b = [[(b"model_id", b"m"), (b"salt", b"s%d" % (i if i % 2 else 9))] for i in range(4)]
    got = equal_blocks(toks, off, 8, a, b)
    want = [sum(x == y for x, y in zip(_lib_keys(reqs[r], a[r], 8), _lib_keys(reqs[r], b[r], 8))) for r in range(4)]
    assert got.tolist() == want
    assert want == [0, 2, 0, 4]


def test_declared_change_gates_the_report():
    case = make_omission_tiny()
    case.changes = {d: d != b"salt" for d in case.dims}
    res = omission_matrix(case)
    j = case.dims.index(b"salt")
    labels = [b[0] for b in case.bindings]
    assert res["collisions"][labels.index("token-only"), j] == res["blocks"]
    assert not res["omission"][:, j].any()
    assert res["omission"][labels.index("token-only")].sum() == len(case.dims) - 1


def test_absent_dimension_is_varied_by_adding_it():
    rng = np.random.default_rng(4)
    toks = rng.integers(0, 1000, size=64, dtype=np.int32)
    base = [(b"model_id", b"m")]
    b = Batch(toks, np.array([0, 64], np.int64), 16, [base], np.zeros(1, np.int32))
    case = OmissionCase(b, [b"model_id", b"adapter_id"], {b"model_id": b"m2", b"adapter_id": b"lora"},
                        {b"model_id": True, b"adapter_id": True},
                        [("complete", None), ("model only", frozenset([b"model_id"]))])
    res = omission_matrix(case)
    assert res["collisions"].tolist() == [[0, 0], [0, 4]]
    assert vary(base, b"adapter_id", b"lora") == [(b"model_id", b"m"), (b"adapter_id", b"lora")]
    assert project(vary(base, b"adapter_id", b"lora"), frozenset([b"model_id"])) == base
