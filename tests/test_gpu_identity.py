"""Content identities on the GPU (section 5.3; the tree hash defined in oracle/identity.py): tensor
roots from the kernels must equal the oracle's for every leaf and fan-in edge, with tensors placed
anywhere in one pool (gaps, shared bytes), and the identity of a set of torch tensors must equal
the oracle's."""

import numpy as np
import pytest

from oracle.identity import identity as oracle_identity
from oracle.identity import tensor_root
from tests.gpu_util import announce, gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

SIZES = [0, 1, 3, 4, 1023, 1024, 1025, 16 * 1024, 16 * 1024 + 1, 17 * 1024 + 3, 256 * 1024, 256 * 1024 + 5,
         300000, 5 * 1024 * 1024 + 7]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def test_roots_at_every_edge(pkv):
    import torch
    announce("tensor roots: 14 sizes in one pool with gaps and a shared range")
    rng = np.random.default_rng(61)
    datas = [rng.integers(0, 256, size=n, dtype=np.uint8).tobytes() for n in SIZES]
    starts, pos = [], 0
    for d in datas:
        pos += int(rng.integers(0, 3)) * 4            # gaps between tensors
        starts.append(pos)
        pos += (len(d) + 3) // 4 * 4
    # room at the end for the shared tensor below: the lengths may add up to the pool size at most
    pool = np.zeros(pos + 64 + (len(datas[9]) + 3) // 4 * 4, np.uint8)
    for st, d in zip(starts, datas):
        pool[st:st + len(d)] = np.frombuffer(d, np.uint8)
    # one more tensor sharing the bytes of tensor 9
    starts.append(starts[9])
    datas.append(datas[9])
    lens = [len(d) for d in datas]
    dev = torch.from_numpy(pool).cuda()
    off = torch.tensor(starts, dtype=torch.int64, device="cuda")
    ln = torch.tensor(lens, dtype=torch.int64, device="cuda")
    work = torch.empty((pkv.pkv_tree_work_bytes(dev.numel(), len(datas)) + 7) // 8, dtype=torch.int64, device="cuda")
    roots = torch.empty((len(datas), 32), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_tensor_roots(dev, off, ln, work, roots, status)
    got = [bytes(r) for r in roots.cpu().numpy()]
    assert int(status.item()) == 0
    assert got == [tensor_root(d) for d in datas]


# Sizes whose leaves take the 16-byte path when their start is 16-byte aligned: tails of a multiple
# of 16 bytes and not, and 1..17, 31..33, 255..257 leaves, so the first node level holds every
# child count from 1 to 16.
ALIGNED_SIZES = [16, 48, 1008, 1024 + 16, 1024 + 20] + [k * 1024 for k in range(1, 18)] + \
    [31 * 1024, 32 * 1024 + 32, 33 * 1024 + 1, 255 * 1024, 256 * 1024, 257 * 1024 + 496]


def test_roots_of_aligned_tensors(pkv):
    import torch
    announce(f"tensor roots: {len(ALIGNED_SIZES)} sizes, starts 16-byte aligned or 4 mod 16")
    rng = np.random.default_rng(63)
    datas = [rng.integers(0, 256, size=n, dtype=np.uint8).tobytes() for n in ALIGNED_SIZES]
    starts, pos = [], 0
    for i, d in enumerate(datas):
        pos = (pos + 15) // 16 * 16 + (4 if i % 5 == 4 else 0)      # every fifth start is 4 mod 16
        starts.append(pos)
        pos += (len(d) + 3) // 4 * 4
    pool = np.zeros(pos + 64, np.uint8)
    for st, d in zip(starts, datas):
        pool[st:st + len(d)] = np.frombuffer(d, np.uint8)
    dev = torch.from_numpy(pool).cuda()
    off = torch.tensor(starts, dtype=torch.int64, device="cuda")
    ln = torch.tensor([len(d) for d in datas], dtype=torch.int64, device="cuda")
    work = torch.empty((pkv.pkv_tree_work_bytes(dev.numel(), len(datas)) + 7) // 8, dtype=torch.int64, device="cuda")
    roots = torch.empty((len(datas), 32), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_tensor_roots(dev, off, ln, work, roots, status)
    got = [bytes(r) for r in roots.cpu().numpy()]
    assert int(status.item()) == 0
    assert got == [tensor_root(d) for d in datas]


def test_roots_of_many_tensors(pkv):
    # more tensors than the kernels stage in LDS for their owner search (1024 CSR entries)
    import torch
    announce("tensor roots: 1500 tensors of 0..5000 bytes")
    rng = np.random.default_rng(64)
    datas = [rng.integers(0, 256, size=int(n), dtype=np.uint8).tobytes() for n in rng.integers(0, 5000, size=1500)]
    starts, pos = [], 0
    for d in datas:
        starts.append(pos)
        pos += (len(d) + 15) // 16 * 16
    pool = np.zeros(pos + 16, np.uint8)
    for st, d in zip(starts, datas):
        pool[st:st + len(d)] = np.frombuffer(d, np.uint8)
    dev = torch.from_numpy(pool).cuda()
    off = torch.tensor(starts, dtype=torch.int64, device="cuda")
    ln = torch.tensor([len(d) for d in datas], dtype=torch.int64, device="cuda")
    work = torch.empty((pkv.pkv_tree_work_bytes(dev.numel(), len(datas)) + 7) // 8, dtype=torch.int64, device="cuda")
    roots = torch.empty((len(datas), 32), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_tensor_roots(dev, off, ln, work, roots, status)
    got = [bytes(r) for r in roots.cpu().numpy()]
    assert int(status.item()) == 0
    assert got == [tensor_root(d) for d in datas]


def test_misplaced_tensor_reports_elayout(pkv):
    import torch
    dev = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    work = torch.empty((pkv.pkv_tree_work_bytes(4096, 2) + 7) // 8, dtype=torch.int64, device="cuda")
    roots = torch.empty((2, 32), dtype=torch.uint8, device="cuda")
    for off, ln in [([0, 2], [10, 10]), ([0, 4000], [10, 100])]:        # unaligned start; past the end
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        pkv.pkv_tensor_roots(dev, torch.tensor(off, dtype=torch.int64, device="cuda"),
                             torch.tensor(ln, dtype=torch.int64, device="cuda"), work, roots, status)
        assert int(status.item()) == pkv.PKV_ELAYOUT


def test_identity_of_torch_tensors_matches_oracle(pkv):
    import torch
    from paper_2609_38706_amd.identity import content_identity
    g = torch.Generator(device="cpu").manual_seed(62)
    tensors = [
        (b"base_model.layers.0.q.lora_A", torch.randn(8, 896, generator=g).to(torch.bfloat16)),
        (b"base_model.layers.0.q.lora_B", torch.randn(896, 8, generator=g).to(torch.bfloat16)),
        (b"base_model.layers.0.mlp.scale", torch.randn(3, generator=g)),              # 12 bytes
        (b"base_model.layers.0.mlp.idx", torch.randint(-128, 127, (7,), generator=g, dtype=torch.int8)),
        (b"empty", torch.zeros(0)),
    ]
    config = [(b"r", b"8"), (b"lora_alpha", b"16"), (b"target_modules", b"q,v")]
    got = content_identity([(n, t.cuda()) for n, t in tensors], config)
    want = oracle_identity([(n, str(t.dtype).replace("torch.", "").encode(), tuple(t.shape),
                             t.contiguous().reshape(-1).view(torch.uint8).numpy().tobytes()) for n, t in tensors],
                           config)
    assert got == want


def _roots_call(pkv, pool_bytes, starts, lens, guard=4096):
    """One pkv_tensor_roots call; the work buffer carries `guard` canary bytes past the size the
    library asks for.  Returns (status, roots, canary intact)."""
    import torch
    dev = torch.from_numpy(pool_bytes).cuda()
    off = torch.tensor(starts, dtype=torch.int64, device="cuda")
    ln = torch.tensor(lens, dtype=torch.int64, device="cuda")
    need = pkv.pkv_tree_work_bytes(dev.numel(), len(starts))
    work = torch.full(((need + guard + 7) // 8,), 0x5A5A5A5A5A5A5A5A, dtype=torch.int64, device="cuda")
    roots = torch.empty((len(starts), 32), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    pkv.pkv_tensor_roots(dev, off, ln, work[: (need + 7) // 8], roots, status)
    tail = work[(need + 7) // 8:].cpu().numpy()
    return int(status.item()), [bytes(r) for r in roots.cpu().numpy()], bool((tail == 0x5A5A5A5A5A5A5A5A).all())


def test_overlapping_tensors_within_the_pool_match_oracle(pkv):
    """Tensors that share bytes, with lengths adding up to no more than the pool: the roots are the
    oracle's."""
    announce("tensor roots: overlapping tensors whose lengths sum to the pool size")
    rng = np.random.default_rng(65)
    pool = rng.integers(0, 256, size=1 << 20, dtype=np.uint8)
    starts = [0, 4096, 100000, 100000, 524288]
    lens = [300000, 200000, 150000, 150000, 200000]
    assert sum(lens) <= pool.shape[0]
    status, got, intact = _roots_call(pkv, pool, starts, lens)
    assert status == 0 and intact
    assert got == [tensor_root(pool[s:s + n].tobytes()) for s, n in zip(starts, lens)]


def test_tensors_longer_than_the_pool_report_elayout(pkv):
    """Eight tensors that each span a whole 1 MiB pool need eight times the leaves the work area
    reserves: the call reports PKV_ELAYOUT and writes nothing past the work area."""
    announce("tensor roots: 8 tensors spanning one 1 MiB pool (expect ELAYOUT, canary intact)")
    pool = np.arange(1 << 20, dtype=np.uint32).astype(np.uint8)
    status, _roots, intact = _roots_call(pkv, pool, [0] * 8, [1 << 20] * 8)
    assert status == pkv.PKV_ELAYOUT
    assert intact
