"""The frozen Case-III mask draws of tests/golden/case3_masks.txt (written
by tests/golden/make_golden.py from oracle/ only; Sec. 3.1, generator
reading R5): the oracle still draws the same words and the same masks, and
within the file the bits follow from the words by the exact threshold
floor(p * 2^64) (a word below it drops the neuron)."""
import os
from fractions import Fraction

import numpy as np

from oracle import masks as om

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "case3_masks.txt")


def _cases():
    lines = [l.strip() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    i = 0
    while i < len(lines):
        _, seed, step, stream, T, K, p = lines[i].split()
        seed, step, stream, T, K, p = int(seed), int(step), int(stream), int(T), int(K), float(p)
        words = [int(w, 16) for w in lines[i + 1].split()[1:]]
        rows = lines[i + 2:i + 2 + T]
        yield seed, step, stream, T, K, p, words, rows
        i += 2 + T


def test_golden_masks_reproduced():
    n = 0
    for seed, step, stream, T, K, p, words, rows in _cases():
        u = om.uniform_words(seed, step, stream, T, K)
        assert [int(w) for w in u[0, :4]] == words
        m = om.keep_mask(seed, step, stream, T, K, p)
        assert ["".join(str(int(v)) for v in m[t]) for t in range(T)] == rows
        n += 1
    assert n == 3


def test_golden_bits_follow_words():
    for seed, step, stream, T, K, p, words, rows in _cases():
        thr = int(Fraction(p) * (1 << 64))
        for k, w in enumerate(words[:K]):
            assert rows[0][k] == ("0" if w < thr else "1")
        assert all(len(r) == K and set(r) <= {"0", "1"} for r in rows)
