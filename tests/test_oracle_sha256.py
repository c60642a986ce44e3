"""Pins of the oracle's SHA-256 (FIPS 180-4) against the standard's printed values and the
Python library routine."""

import hashlib
import os

import numpy as np
import pytest

import oracle


def _vectors(golden_dir):
    out = []
    for line in open(os.path.join(golden_dir, "fips180_sha256_vectors.txt")):
        if line.startswith("#") or not line.strip():
            continue
        spec, hexd = line.rstrip("\n").rsplit(" ", 1)
        kind, _, rest = spec.partition(":")
        if kind == "text":
            msg = rest.encode()
        else:
            count, _, text = rest.partition(":")
            msg = text.encode() * int(count)
        out.append((msg, bytes.fromhex(hexd)))
    return out


def test_fips_example_vectors(golden_dir):
    vecs = _vectors(golden_dir)
    assert len(vecs) == 5
    for msg, want in vecs:
        assert hashlib.sha256(msg).digest() == want      # the fixture itself is right
        assert oracle.sha256(msg) == want


def test_constants_match_the_printed_tables(golden_dir):
    k_printed, iv_printed = [], []
    for line in open(os.path.join(golden_dir, "fips180_sha256_constants.txt")):
        if line.startswith("K "):
            k_printed += [int(x, 16) for x in line.split()[1:]]
        elif line.startswith("IV "):
            iv_printed += [int(x, 16) for x in line.split()[1:]]
    k, iv = oracle.sha256_constants()
    assert [int(x) for x in k] == k_printed
    assert [int(x) for x in iv] == iv_printed


@pytest.mark.parametrize("length", [0, 1, 3, 4, 31, 32, 55, 56, 57, 63, 64, 65, 96, 119, 120, 127, 128, 129,
                                    1056, 1065])
def test_padding_edges_against_library(length):
    rng = np.random.default_rng(length)
    msg = rng.integers(0, 256, size=length, dtype=np.uint8).tobytes()
    assert oracle.sha256(msg) == hashlib.sha256(msg).digest()


def test_random_lengths_against_library():
    rng = np.random.default_rng(7)
    for _ in range(300):
        n = int(rng.integers(0, 2001))
        msg = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        assert oracle.sha256(msg) == hashlib.sha256(msg).digest()
