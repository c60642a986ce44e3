"""The allocation-free variant of the tensor-root call (pkv_tensor_roots_static, for callers that
cannot allocate device memory) against pkv_tensor_roots on the same inputs: two calls in a row, the
second on a smaller input, so the second call runs in a work area that still holds the first call's
digests.  (The refusal of inputs past the library's buffer is a host check, tested on the CPU.)"""

import numpy as np
import pytest

from tests.gpu_util import announce, gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def pkv():
    import paper_2609_38706_amd as m
    m.lib()
    return m


def _case(seed, n_tensors, max_len):
    """A pool of tensors at 4-byte aligned starts with gaps, lengths 0 .. max_len bytes."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, max_len, size=n_tensors)
    lens[rng.random(n_tensors) < 0.1] = 0
    starts, pos = [], 0
    for n in lens:
        pos += int(rng.integers(0, 3)) * 4
        starts.append(pos)
        pos += (int(n) + 3) // 4 * 4
    pool = rng.integers(0, 256, size=pos + 16, dtype=np.uint8)
    return pool, starts, [int(n) for n in lens]


def _both(pkv, pool, starts, lens):
    import torch
    dev = torch.from_numpy(pool).cuda()
    off = torch.tensor(starts, dtype=torch.int64, device="cuda")
    ln = torch.tensor(lens, dtype=torch.int64, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    work = torch.empty((pkv.pkv_tree_work_bytes(dev.numel(), len(starts)) + 7) // 8, dtype=torch.int64, device="cuda")
    want = torch.empty((len(starts), 32), dtype=torch.uint8, device="cuda")
    pkv.pkv_tensor_roots(dev, off, ln, work, want, status)
    got = torch.full((len(starts), 32), 0xA5, dtype=torch.uint8, device="cuda")
    pkv.pkv_tensor_roots_static(dev, off, ln, got, status)
    torch.cuda.synchronize()
    return int(status.item()), got.cpu().numpy(), want.cpu().numpy()


def test_static_roots_equal_the_work_area_call_twice(pkv):
    announce("tensor roots, allocation-free entry point: 300 tensors up to 200 KB, then 40 up to 5 KB")
    big = _case(71, 300, 200_000)
    assert pkv.pkv_tree_work_bytes(big[0].shape[0], 300) <= pkv.STATIC_TREE_WORK_BYTES
    status, got, want = _both(pkv, *big)
    assert status == 0
    assert (got == want).all()
    small = _case(72, 40, 5_000)
    status, got, want = _both(pkv, *small)
    assert status == 0
    assert (got == want).all()
