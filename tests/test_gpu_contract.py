"""The contract's properties and the degenerate inputs, exercised on the HIP path (through the C ABI):
empty and ragged batches, requests shorter than one block, the switches between the derive
kernels, every-key-changes on a one-dimension change (Eq. 4), token-only erasure (Def. 1), the
binding pattern (section 6.1) and storage growth (section 6.5)."""

import numpy as np
import pytest

import oracle
from tests.gpu_util import check_structure, gpu_available, gpu_batch, oracle_keys
from workloads import Batch, locations

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

BASE = [(b"model_id", b"synthetic-8b"), (b"adapter_id", b"lora-A"), (b"weight_dtype", b"bfloat16"),
        (b"weight_version", (7).to_bytes(8, "little")), (b"kv_format", b"bfloat16"), (b"salt", b"tenant-1"),
        (b"x00", b"rope-10000")]


def _with(desc, name, value):
    out = [(n, v) for n, v in desc if n != name]
    if value is not None:
        out.append((name, value))
    return out


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def _derive(tokens_list, descs, block=16):
    off = np.zeros(len(tokens_list) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in tokens_list])
    toks = np.concatenate([np.asarray(t, np.int32) for t in tokens_list]) if tokens_list else np.zeros(0, np.int32)
    b = Batch(toks, off, block, descs, np.arange(len(tokens_list), dtype=np.int32))
    db = gpu_batch(b)
    db.digest()
    db.derive()
    keys = db.host_keys()
    ko = db.key_off.cpu().numpy()
    assert db.host_status() == 0
    return [keys[ko[r]:ko[r + 1]] for r in range(len(tokens_list))], db, b


def test_empty_batch(pkv):
    import torch
    b = Batch(np.zeros(0, np.int32), np.zeros(1, np.int64), 16, [], np.zeros(0, np.int32))
    db = gpu_batch(b)
    table = pkv.Table(64)
    db.step(table)
    torch.cuda.synchronize()
    assert db.n_keys == 0 and db.host_status() == 0 and int(db.n_new.item()) == 0


def test_requests_shorter_than_a_block_have_no_keys(pkv):
    rng = np.random.default_rng(1)
    reqs = [rng.integers(0, 1000, size=n, dtype=np.int32) for n in [0, 1, 15, 0, 7]]
    ks, db, b = _derive(reqs, [BASE] * 5)
    assert db.n_keys == 0 and all(k.shape[0] == 0 for k in ks)
    table = pkv.Table(64)
    db.lookup(table)
    db.store(table)
    assert db.host_hits().tolist() == [0] * 5 and int(db.n_new.item()) == 0


def test_ragged_with_empty_requests_in_between(pkv):
    rng = np.random.default_rng(2)
    lens = [0, 33, 0, 0, 16, 1, 200, 0, 64, 17]
    reqs = [rng.integers(0, 128256, size=n, dtype=np.int32) for n in lens]
    descs = [_with(BASE, b"salt", b"s%d" % i) for i in range(len(lens))]
    ks, db, b = _derive(reqs, descs)
    want, ko = oracle_keys(b)
    assert (db.host_keys() == want).all()
    assert [k.shape[0] for k in ks] == [n // 16 for n in lens]


@pytest.mark.parametrize("n_req,block", [(8192, 16), (8193, 16), (16384, 16), (16385, 16), (8192, 32), (8193, 32),
                                         (8193, 48), (9000, 256), (16385, 48)])
def test_derive_kernels_agree_at_the_switches(pkv, n_req, block):
    """The kernel switches at 256 compute units.  B = 16: up to 8192 requests run one lane-pair
    consumer/helper pair per workgroup (32 chains each), 8193..16384 two pairs per workgroup, from
    16385 on one lane per chain.  B = 16m: up to 8192 requests the lane-pair kernel, 8193..16384 the
    consumer/helper kernel with one lane per chain, from 16385 on the one-wavefront kernel.  Every
    kernel must give the oracle's keys."""
    rng = np.random.default_rng(n_req + block)
    lens = rng.integers(0, 4 * block, size=n_req)
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = rng.integers(0, 128256, size=int(off[-1]), dtype=np.int32)
    descs = [_with(BASE, b"salt", b"%d" % i) for i in range(7)]
    b = Batch(toks, off, block, descs, rng.integers(0, 7, size=n_req).astype(np.int32))
    db = gpu_batch(b)
    db.digest()
    db.derive()
    want, _ = oracle_keys(b)
    assert db.host_status() == 0
    assert (db.host_keys() == want).all()


@pytest.mark.parametrize("block", [16, 32])
@pytest.mark.parametrize("n_req", [1, 7, 8, 9, 15, 16, 17, 24, 31, 33, 40, 63, 65])
def test_lane_pair_rows_with_partial_waves(pkv, n_req, block):
    """The lane-pair kernels give chain i of a row lanes i and i + 8; request counts that end inside
    a row, inside a wavefront or just past one, with chains of different lengths (0 to 40 keys, so
    partners stop at different keys), must all give the oracle's keys."""
    rng = np.random.default_rng(1000 + n_req + block)
    lens = rng.integers(0, 40 * block, size=n_req)
    off = np.zeros(n_req + 1, np.int64)
    off[1:] = np.cumsum(lens)
    toks = rng.integers(0, 128256, size=int(off[-1]), dtype=np.int32)
    descs = [_with(BASE, b"salt", b"%d" % i) for i in range(5)]
    b = Batch(toks, off, block, descs, rng.integers(0, 5, size=n_req).astype(np.int32))
    db = gpu_batch(b)
    db.digest()
    db.derive()
    want, _ = oracle_keys(b)
    assert db.host_status() == 0
    assert (db.host_keys() == want).all()


@pytest.mark.parametrize("name", [n for n, _ in BASE])
def test_one_dimension_change_changes_every_key_on_gpu(pkv, name):
    rng = np.random.default_rng(11)
    toks = rng.integers(0, 128256, size=16 * 40 + 5, dtype=np.int32)
    descs = [BASE, _with(BASE, name, dict(BASE)[name] + b"'"), _with(BASE, name, None)]
    (a, b, c), _, _ = _derive([toks] * 3, descs)
    for other in (b, c):
        assert all((a[i] != other[i]).any() for i in range(40))


def test_token_only_keys_collide_bound_keys_do_not(pkv):
    rng = np.random.default_rng(12)
    toks = rng.integers(0, 128256, size=16 * 12, dtype=np.int32)
    descs = [BASE, _with(BASE, b"adapter_id", b"lora-B"), _with(BASE, b"weight_dtype", b"float8_e4m3fn"),
             _with(BASE, b"salt", b"tenant-2")]
    token_only, _, _ = _derive([toks] * 4, [[]] * 4)
    bound, _, _ = _derive([toks] * 4, descs)
    assert all((k == token_only[0]).all() for k in token_only)
    assert len({k[0].tobytes() for k in bound}) == 4


def test_binding_pattern_on_gpu(pkv):
    """Same provenance -> full-prefix hit; any single-dimension cross -> 0 (section 6.1)."""
    rng = np.random.default_rng(13)
    toks = rng.integers(0, 128256, size=16 * 24, dtype=np.int32)
    readers = [BASE] + [_with(BASE, n, v + b"#") for n, v in BASE]
    table = pkv.Table(1 << 12)
    _, seed_db, _ = _derive([toks], [BASE])
    seed_db.set_locations(locations(seed_db.key_off.cpu().numpy(), 1))
    seed_db.hits.zero_()
    seed_db.store(table)
    _, db, _ = _derive([toks] * len(readers), readers)
    db.lookup(table)
    assert db.host_hits().tolist() == [24] + [0] * (len(readers) - 1)


def test_storage_grows_linearly_with_provenance_classes_on_gpu(pkv):
    rng = np.random.default_rng(14)
    toks = rng.integers(0, 128256, size=16 * 20, dtype=np.int32)
    for k in range(1, 5):
        descs = [_with(BASE, b"weight_version", (i + 1).to_bytes(8, "little")) for i in range(k)]
        for bound in (True, False):
            _, db, _ = _derive([toks] * k, descs if bound else [[]] * k)
            db.set_locations(locations(db.key_off.cpu().numpy(), 0))
            table = pkv.Table(1 << 10)
            db.hits.zero_()
            db.store(table)
            assert int(db.n_new.item()) == (20 * k if bound else 20)
            assert check_structure(table) == (20 * k if bound else 20)
