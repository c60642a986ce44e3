"""Index persistence and restart parity (section 6.3, an adapter's prefix keeps hitting across a
restart): an index saved by one process and rebuilt by a fresh process holds the same pairs and
answers lookups exactly as the oracle's index does."""

import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import announce, gpu_available, gpu_batch, oracle_keys
from tests.test_gpu_pipeline import _batches
from workloads import locations

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys, numpy as np
sys.path.insert(0, sys.argv[1])
from paper_2609_38706_amd.persist import load_table
from paper_2609_38706_amd.pipeline import export_sorted
from tests.gpu_util import gpu_batch
from tests.test_gpu_pipeline import _batches
table = load_table(sys.argv[2])
probe = _batches(4, seed=41)[3]
db = gpu_batch(probe)
db.digest(); db.derive(); db.lookup(table)
k, l = export_sorted(table)
assert db.host_status() == 0
np.savez(sys.argv[3], hits=db.host_hits(), keys=k, locs=l)
print("child done", flush=True)
"""


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def test_saved_index_serves_a_restarted_process(pkv, tmp_path):
    from paper_2609_38706_amd.persist import load_table, save_table
    from paper_2609_38706_amd.pipeline import export_sorted
    announce("persistence: save, reload in this process and in a fresh process")
    batches = _batches(4, seed=41)
    cap = 1 << 12
    table = pkv.Table(cap)
    idx = oracle.Index(cap)
    for b in batches[:3]:
        db = gpu_batch(b)
        db.n_new.zero_()
        db.step(table)
        assert db.host_status() == 0
        k, ko = oracle_keys(b)
        idx.store(k, ko, idx.lookup(k, ko), locations(ko, b.tag))
    path = str(tmp_path / "index.npz")
    save_table(table, path)
    want_k, want_l = idx.dump()
    # same process
    t2 = load_table(path)
    k2, l2 = export_sorted(t2)
    assert (k2 == want_k).all() and (l2 == want_l).all()
    # fresh process
    out = str(tmp_path / "child.npz")
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT, path, out], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    with np.load(out, allow_pickle=False) as f:
        hits, k3, l3 = f["hits"], f["keys"], f["locs"]
    assert (k3 == want_k).all() and (l3 == want_l).all()
    pk, pko = oracle_keys(batches[3])
    assert (hits == idx.lookup(pk, pko)).all()
    assert hits.sum() > 0


def test_load_into_a_larger_index(pkv, tmp_path):
    from paper_2609_38706_amd.persist import load_table, save_table
    from paper_2609_38706_amd.pipeline import export_sorted
    b = _batches(1, seed=42)[0]
    table = pkv.Table(1 << 10)
    db = gpu_batch(b)
    db.n_new.zero_()
    db.step(table)
    path = str(tmp_path / "small.npz")
    save_table(table, path)
    big = load_table(path, capacity=1 << 14)
    a, b2 = export_sorted(table), export_sorted(big)
    assert big.capacity == 1 << 14
    assert (a[0] == b2[0]).all() and (a[1] == b2[1]).all()
