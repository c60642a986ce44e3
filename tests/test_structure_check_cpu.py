"""The GPU tests' index-structure check (tests/gpu_util.check_structure) on index images built on
the host: images that follow the probe-path rule of include/pkv.h pass, and images with an entry
moved off its path, a duplicate key or a pending slot fail."""

import numpy as np
import pytest

from tests.gpu_util import check_structure

EMPTY = 0xFFFFFFFFFFFFFFFF


class _Image:
    """A host-side index image with the `slots` / `capacity` interface check_structure reads."""

    class _Slots:
        def __init__(self, words):
            self.words = words

        def cpu(self):
            return self

        def numpy(self):
            return self.words.view(np.uint8)

    def __init__(self, capacity):
        self.capacity = capacity
        w = np.empty((capacity, 4), np.uint64)
        w[:, 0] = EMPTY
        w[:, 1] = 0
        w[:, 2] = EMPTY
        w[:, 3] = EMPTY
        self.w = w
        self.slots = self._Slots(w.reshape(-1))

    def path(self, key: bytes):
        lo = int.from_bytes(key[:8], "little")
        n_b = self.capacity // 4
        b, r = lo & (n_b - 1), key[8] & 3
        for i in range(self.capacity):
            yield ((b + i // 4) % n_b) * 4 + ((r + i) & 3)

    def insert(self, key: bytes, loc: int, removed_ok=True):
        for s in self.path(key):
            if self.w[s, 0] == EMPTY or (removed_ok and self.w[s, 0] == EMPTY - 1):
                self.put(s, key, loc)
                return s
        raise AssertionError("full")

    def put(self, s, key: bytes, loc: int):
        self.w[s, 0] = int.from_bytes(key[:8], "little")
        self.w[s, 1] = (12345 << 2)
        self.w[s, 2] = int.from_bytes(key[8:], "little")
        self.w[s, 3] = loc

    def clear(self, s):
        self.w[s] = [EMPTY, 0, EMPTY, EMPTY]


def _filled(seed, capacity=256, n=150, clustered=True):
    rng = np.random.default_rng(seed)
    img = _Image(capacity)
    keys = []
    for i in range(n):
        k = bytearray(rng.bytes(16))
        if clustered:                       # few home buckets, so paths run over several buckets
            k[0] = int(rng.integers(0, 8))
            k[1:8] = b"\0" * 7
        keys.append(bytes(k))
        img.insert(bytes(k), i)
    return img, keys


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_images_that_follow_the_path_rule_pass(seed):
    img, keys = _filled(seed)
    assert check_structure(img) == len(keys)
    img2, keys2 = _filled(seed, n=100, clustered=False)
    assert check_structure(img2) == len(keys2)


def test_an_entry_behind_a_never_used_slot_of_its_bucket_fails():
    img = _Image(64)
    key = bytes([5] + [0] * 7 + [2] + [9] * 7)       # home bucket 5, path starts at slot 2 of it
    s = img.insert(key, 7)
    assert s == 5 * 4 + 2
    assert check_structure(img) == 1
    img.clear(s)
    img.put(5 * 4 + 3, key, 7)                         # second slot on the path, the first is never used
    with pytest.raises(AssertionError, match="never-used slot of its bucket"):
        check_structure(img)
    img.clear(5 * 4 + 3)
    img.put(5 * 4 + 1, key, 7)                         # last slot on the path, the first three never used
    with pytest.raises(AssertionError, match="never-used slot of its bucket"):
        check_structure(img)


def test_an_entry_past_a_bucket_with_a_never_used_slot_fails():
    img = _Image(64)
    key = bytes([5] + [0] * 7 + [0] + [9] * 7)
    for j in range(3):                                 # bucket 5 keeps one never-used slot
        img.put(5 * 4 + j, bytes([5] + [0] * 7 + [1, j] + [0] * 6), 100 + j)
    img.put(6 * 4 + 0, key, 7)                         # in the next bucket: off its path
    with pytest.raises(AssertionError, match="bucket with a never-used slot"):
        check_structure(img)
    img.put(5 * 4 + 3, bytes([5] + [0] * 7 + [1, 3] + [0] * 6), 103)   # bucket 5 now full
    assert check_structure(img) == 5


def test_wrapping_paths_pass_and_fail_like_the_others():
    img = _Image(32)                                   # 8 buckets; home bucket 7 wraps to bucket 0
    for j in range(4):
        img.put(7 * 4 + j, bytes([7] + [0] * 7 + [j, 1] + [0] * 6), j)
    key = bytes([7] + [0] * 7 + [1] + [9] * 7)
    assert img.insert(key, 9) == 0 * 4 + 1
    assert check_structure(img) == 5
    img.clear(7 * 4 + 2)
    with pytest.raises(AssertionError, match="bucket with a never-used slot"):
        check_structure(img)


def test_duplicate_and_pending_entries_fail():
    img, keys = _filled(4, n=40)
    free = [i for i in img.path(keys[0]) if img.w[i, 0] == EMPTY][0]
    img.put(free, keys[0], 999)                        # the same key twice on its path
    with pytest.raises(AssertionError, match="duplicate key"):
        check_structure(img)
    img3, keys3 = _filled(5, n=40)
    s3 = next(iter(img3.path(keys3[0])))
    img3.w[s3, 3] = EMPTY                              # claimed, location never published
    with pytest.raises(AssertionError):
        check_structure(img3)
