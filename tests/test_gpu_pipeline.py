"""The two-stream runner: overlapping the derive of batch k+1 with the lookup and store of batch k
must give exactly the hit lengths and index contents of running the batches one after another,
and both must equal the oracle's sequence of lookups and stores."""

import numpy as np
import pytest

import oracle
from tests.gpu_util import announce, check_structure, gpu_available, gpu_batch, oracle_keys
from workloads import Batch, locations

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def _batches(n_batches, seed=31, n_req=24, block=16):
    """Batches whose requests share prefixes with earlier batches, so later lookups hit what earlier
    stores inserted; some requests repeat inside a batch (duplicate keys in one store)."""
    rng = np.random.default_rng(seed)
    prefixes = [rng.integers(0, 128256, size=int(rng.integers(16, 300)), dtype=np.int32) for _ in range(8)]
    descs = [[(b"model_id", b"m"), (b"salt", bytes([i]) * 8)] for i in range(3)]
    out = []
    for b in range(n_batches):
        reqs = []
        for r in range(n_req):
            if r > 0 and rng.random() < 0.15:
                reqs.append(reqs[-1].copy())
                continue
            p = prefixes[int(rng.integers(8))]
            suffix = rng.integers(0, 128256, size=int(rng.integers(0, 120)), dtype=np.int32)
            reqs.append(np.concatenate([p[: int(rng.integers(0, p.shape[0] + 1))], suffix]))
        off = np.zeros(n_req + 1, np.int64)
        off[1:] = np.cumsum([x.shape[0] for x in reqs])
        out.append(Batch(np.concatenate(reqs), off, block, descs, rng.integers(0, 3, size=n_req).astype(np.int32),
                         tag=1 + b))
    return out


def _oracle_sequence(batches, capacity):
    idx = oracle.Index(capacity)
    hits_all = []
    for b in batches:
        keys, ko = oracle_keys(b)
        hits = idx.lookup(keys, ko)
        assert idx.store(keys, ko, hits, locations(ko, b.tag)) == 0
        hits_all.append(hits)
    return hits_all, idx.dump()


def test_overlapped_batches_equal_serial_and_oracle(pkv):
    import torch
    from paper_2609_38706_amd.pipeline import TwoStreamRunner, export_sorted
    announce("two-stream runner: 6 batches with shared prefixes")
    batches = _batches(6)
    cap = 1 << 12
    want_hits, (want_k, want_l) = _oracle_sequence(batches, cap)
    # serial on one stream
    t_serial = pkv.Table(cap)
    for b, wh in zip(batches, want_hits):
        db = gpu_batch(b)
        db.n_new.zero_()
        db.step(t_serial)
        assert db.host_status() == 0
        assert (db.host_hits() == wh).all()
    # overlapped on two streams
    t_pipe = pkv.Table(cap)
    dbs = [gpu_batch(b) for b in batches]
    TwoStreamRunner(t_pipe).run(dbs)
    torch.cuda.synchronize()
    for db, wh in zip(dbs, want_hits):
        assert db.host_status() == 0
        assert (db.host_hits() == wh).all()
    for t in (t_serial, t_pipe):
        k, l = export_sorted(t)
        assert (k == want_k).all() and (l == want_l).all()
        assert check_structure(t) == want_k.shape[0]


def test_recycled_buffers_with_rollback_repeat_the_first_pass(pkv):
    """Two buffer sets of one batch alternate with rollback (the benchmark's pattern): every pass must
    meet the same index and give the same hits, and the index must end as it began."""
    import torch
    from paper_2609_38706_amd.pipeline import TwoStreamRunner, export_sorted
    announce("two-stream runner: recycled buffers with rollback")
    pre, run = _batches(2, seed=32)
    cap = 1 << 12
    table = pkv.Table(cap)
    db = gpu_batch(pre)
    db.step(table)
    before = export_sorted(table)
    idx = oracle.Index(cap)
    k0, ko0 = oracle_keys(pre)
    idx.store(k0, ko0, np.zeros(pre.n_req, np.int32), locations(ko0, pre.tag))
    k1, ko1 = oracle_keys(run)
    want = idx.lookup(k1, ko1)
    a, b, c = gpu_batch(run), gpu_batch(run), gpu_batch(run)
    runner = TwoStreamRunner(table)
    # two buffer sets alternating (a pass's preparation reuses the buffers of the pass two before),
    # then three in a cycle, then a single pass
    for order in ([a, b] * 5, [a, b, c] * 4, [c]):
        for x in (a, b, c):
            x.hits.fill_(-7)
        runner.run(order, rollback=True)
        torch.cuda.synchronize()
        for x in set(order):
            assert x.host_status() == 0
            assert (x.host_hits() == want).all()
        after = export_sorted(table)
        assert (before[0] == after[0]).all() and (before[1] == after[1]).all()
    with pytest.raises(ValueError):
        runner.run([a, a])
