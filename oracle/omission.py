"""Differential omission test at key level -- TEST INFRASTRUCTURE ONLY.

Section 5.4, Eq. 4: for a dimension d of the registry, hold the tokens x and every other dimension
fixed, replace d's value by a distinct v', and report an omission iff the state changes while the
key does not:

    KV(x, c) != KV(x, c[d -> v'])   and   Key(x, c) == Key(x, c[d -> v'])

No model runs here, so the first condition is declared per dimension by the caller (whether
varying it changes the computed state or, for the permission invariant of Eq. 2, the sharing
permission).  The second condition is computed from its definition: the keys of every complete
block of x are derived under both configurations and compared position by position.  A key
binding R keys with the configuration projected onto the dimensions in R (all fields when R is
None; nothing, i.e. a token-only key, when R is empty).  The result counts, per (binding,
dimension), the blocks whose two keys are equal.

Only the tests and the benchmark's CPU-baseline leg use this module.
"""

from __future__ import annotations

import numpy as np

from . import derive, digest, key_offsets


def project(desc, names):
    """The configuration restricted to the bound dimensions (all of them when names is None)."""
    return [(n, v) for n, v in desc if names is None or n in names]


def vary(desc, name, value):
    """c[d -> v']: the configuration with dimension `name` set to `value` (added if absent)."""
    return [(n, v) for n, v in desc if n != name] + [(name, value)]


def _digests(descs, cache):
    out = np.zeros((len(descs), 16), np.uint8)
    for i, d in enumerate(descs):
        k = tuple(sorted(d))
        if k not in cache:
            cache[k] = np.frombuffer(digest(d), np.uint8)
        out[i] = cache[k]
    return out


def equal_blocks(tokens, tok_off, block, descs_a, descs_b, threads=1, cache=None):
    """Per request r: the number of complete blocks whose key under descs_a[r] equals the key under
    descs_b[r] (both over the same tokens)."""
    cache = {} if cache is None else cache
    ka = derive(tokens, tok_off, _digests(descs_a, cache), block, threads)
    kb = derive(tokens, tok_off, _digests(descs_b, cache), block, threads)
    ko = key_offsets(tok_off, block)
    same = np.concatenate([[0], np.cumsum((ka == kb).all(axis=1), dtype=np.int64)])
    return same[ko[1:]] - same[ko[:-1]]


def omission_matrix(case, threads=1):
    """Eq. 4 over every (binding, dimension) pair of an omission case.

    Returns ``collisions`` int64 [bindings, dims] (blocks whose keys coincide), ``omission`` bool
    [bindings, dims] (declared change and at least one coinciding key) and ``blocks`` (complete
    blocks per configuration)."""
    b = case.batch
    base = b.request_descs()
    cache = {}
    coll = np.zeros((len(case.bindings), len(case.dims)), np.int64)
    for i, (_label, names) in enumerate(case.bindings):
        base_p = [project(d, names) for d in base]
        for j, dim in enumerate(case.dims):
            var_p = [project(vary(d, dim, case.variants[dim]), names) for d in base]
            coll[i, j] = equal_blocks(b.tokens, b.tok_off, b.block, base_p, var_p, threads, cache).sum()
    changes = np.array([bool(case.changes[d]) for d in case.dims])
    return {"collisions": coll, "omission": (coll > 0) & changes[None, :],
            "blocks": int(key_offsets(b.tok_off, b.block)[-1])}
