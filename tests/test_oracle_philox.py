"""Pins the oracle's Philox4x64-10 against numpy's own Philox bit generator
(a library implementation of the same published generator), and its 128-bit
multiply against Python's arbitrary-precision integers."""
import random

import numpy as np
import pytest

from oracle.philox import philox4x64, mulhilo64

MAX64 = (1 << 64) - 1


def _numpy_block(counter, key):
    # numpy's Philox increments its 256-bit counter before producing a block,
    # so the block for counter c is obtained by seeding it with c - 1.
    v = sum(int(c) << (64 * i) for i, c in enumerate(counter))
    v = (v - 1) % (1 << 256)
    prev = np.array([(v >> (64 * i)) & MAX64 for i in range(4)], dtype=np.uint64)
    g = np.random.Philox(counter=prev, key=np.array(key, dtype=np.uint64))
    return g.random_raw(4)


@pytest.mark.parametrize("key", [(0, 0), (7, 9), (MAX64, 12345), (1002, 0), (0x0123456789ABCDEF, MAX64)])
@pytest.mark.parametrize("counter", [(0, 0, 0, 0), (1, 0, 0, 0), (5, 34, 2, 0), (MAX64, 3, 4, 5),
                                     (255, 63, 6, 17), (MAX64, MAX64, MAX64, MAX64)])
def test_philox_matches_numpy(key, counter):
    ref = _numpy_block(counter, key)
    mine = philox4x64(np.array(counter, dtype=np.uint64), (np.uint64(key[0]), np.uint64(key[1])))
    assert np.array_equal(ref, mine)


def test_philox_vectorised_matches_scalar():
    rng = random.Random(3)
    ctrs = np.array([[rng.getrandbits(64) for _ in range(4)] for _ in range(64)], dtype=np.uint64)
    key = (np.uint64(rng.getrandbits(64)), np.uint64(rng.getrandbits(64)))
    batch = philox4x64(ctrs, key)
    for i in range(0, 64, 7):
        ref = _numpy_block(ctrs[i].tolist(), (int(key[0]), int(key[1])))
        assert np.array_equal(batch[i], ref)


def test_mulhilo_against_python_ints():
    rng = random.Random(11)
    vals = [0, 1, MAX64, 1 << 63, (1 << 32) - 1, 1 << 32] + [rng.getrandbits(64) for _ in range(200)]
    for a in vals:
        for b in vals[:20]:
            hi, lo = mulhilo64(np.uint64(a), np.uint64(b))
            assert int(hi) == (a * b) >> 64
            assert int(lo) == (a * b) & MAX64
