"""Pins of the oracle's canonical descriptor encoding and digest (section 5.1 well-formedness,
section 5.2 Eq. 3 and Prop. 1)."""

import hashlib
import itertools
import os
import struct

import pytest

import oracle


def _worked_example(golden_dir):
    fields, enc = [], b""
    for line in open(os.path.join(golden_dir, "enc_worked_example.txt")):
        if line.startswith("field "):
            name, _, value = line[len("field "):].rstrip("\n").partition(" =")
            fields.append((name.encode(), bytes.fromhex(value.strip())))
        elif line.startswith("enc "):
            enc += bytes.fromhex(line.split()[1])
    return fields, enc


def test_worked_example(golden_dir):
    fields, enc = _worked_example(golden_dir)
    assert len(fields) == 5
    assert oracle.encode(fields) == enc
    # H is SHA-256 truncated to 128 bits: a special case of the library routine
    assert oracle.digest(fields) == hashlib.sha256(enc).digest()[:16]


def decode(enc: bytes):
    """Inverse of the encoding: returns the list of (name, value) pairs, or raises."""
    assert enc[:4] == b"PKV1"
    (m,) = struct.unpack_from("<I", enc, 4)
    pos, out = 8, []
    for _ in range(m):
        (ln,) = struct.unpack_from("<I", enc, pos)
        name = enc[pos + 4: pos + 4 + ln]
        pos += 4 + ln
        (lv,) = struct.unpack_from("<I", enc, pos)
        value = enc[pos + 4: pos + 4 + lv]
        pos += 4 + lv
        out.append((name, value))
    assert pos == len(enc)
    return out


# Values chosen to look like length prefixes, empty strings, zero bytes and prefixes of each other.
TRICKY = [None, b"", b"a", b"ab", b"\x00", b"\x01\x00\x00\x00a", b"\x02\x00\x00\x00ab"]


def _all_descriptors(names, domain):
    for values in itertools.product(domain, repeat=len(names)):
        yield [(n, v) for n, v in zip(names, values) if v is not None]


@pytest.mark.parametrize("names", [
    (b"model_id", b"salt", b"a"),             # core + extra
    (b"a", b"ab", b"b"),                      # extras whose names are prefixes of each other
    (b"adapter_id", b"weight_version", b"kv_format"),
])
def test_injective_by_brute_force(names):
    seen_enc, seen_dig = {}, {}
    for desc in _all_descriptors(names, TRICKY):
        enc = oracle.encode(desc)
        assert sorted(decode(enc)) == sorted(desc)          # decodes back to exactly the fields
        key = frozenset(desc)
        assert seen_enc.setdefault(enc, key) == key
        dig = oracle.digest(desc)
        assert seen_dig.setdefault(dig, key) == key
    assert len(seen_enc) == len(TRICKY) ** len(names)


def test_canonical_order_of_core_and_extras():
    desc = [(b"zz", b"1"), (b"salt", b"s"), (b"kv_format", b"k"), (b"weight_version", b"v"),
            (b"weight_dtype", b"d"), (b"adapter_id", b"a"), (b"model_id", b"m"), (b"a", b"2"), (b"ab", b"3")]
    names = [n for n, _ in decode(oracle.encode(desc))]
    assert names == [b"model_id", b"adapter_id", b"weight_dtype", b"weight_version", b"kv_format", b"salt",
                     b"a", b"ab", b"zz"]


def test_field_order_does_not_matter():
    desc = [(b"model_id", b"m"), (b"adapter_id", b"lora-1"), (b"weight_dtype", b"bfloat16"),
            (b"salt", b"\x00" * 8), (b"x1", b"e")]
    ref = oracle.digest(desc)
    for perm in itertools.permutations(desc):
        assert oracle.digest(list(perm)) == ref


def test_duplicate_names_rejected():
    with pytest.raises(oracle.OracleError) as e:
        oracle.encode([(b"salt", b"a"), (b"model_id", b"m"), (b"salt", b"b")])
    assert e.value.code == oracle.EDUPDIM


def test_dimension_extension_prop1():
    """Prop. 1: appending a registered dimension keeps distinct descriptors distinct; a request that
    does not carry the new dimension keeps its digest (absent fields are not encoded)."""
    base = [(b"model_id", b"m"), (b"salt", b"s")]
    d0 = oracle.digest(base)
    assert oracle.digest(base + [(b"rope_base", b"10000")]) != d0
    assert oracle.digest(base + [(b"rope_base", b"500000")]) != oracle.digest(base + [(b"rope_base", b"10000")])
    # carrying the new dimension with an empty value is still different from not carrying it
    assert oracle.digest(base + [(b"rope_base", b"")]) != d0


def test_empty_descriptor():
    assert oracle.encode([]) == b"PKV1\x00\x00\x00\x00"
    assert oracle.digest([]) == hashlib.sha256(b"PKV1\x00\x00\x00\x00").digest()[:16]
