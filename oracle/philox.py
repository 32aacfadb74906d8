"""Philox4x64-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11), written from that
paper's definition.  Test infrastructure only (see the package docstring).

The paper under study does not say how its dropout masks are drawn; this
oracle and the HIP library both use this generator so that masks can be
compared bit for bit.  The generator is a bijection of a 256-bit counter
under a 128-bit key:

  one round     (x0, x1, x2, x3), key (k0, k1):
                  hi0:lo0 = M0 * x0,  hi1:lo1 = M1 * x2   (full 128-bit products)
                  -> (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0)
  key schedule  after every round but the last: k0 += W0, k1 += W1 (mod 2^64)
  rounds        10

with multipliers M0, M1 and Weyl increments W0 (golden ratio) and W1
(sqrt(3) - 1) as published.

Everything is vectorised over numpy uint64 arrays; the 128-bit product is
assembled from 32-bit limbs (schoolbook multiplication).
"""
from __future__ import annotations

import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15
W1 = 0xBB67AE8584CAA73B
ROUNDS = 10

_MASK32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def mulhilo64(a, b):
    """Return (hi, lo) of the 128-bit product a*b for uint64 arrays/scalars."""
    a = np.asarray(a, dtype=np.uint64)
    b = np.asarray(b, dtype=np.uint64)
    a0, a1 = a & _MASK32, a >> _S32
    b0, b1 = b & _MASK32, b >> _S32
    p00 = a0 * b0
    p01 = a0 * b1
    p10 = a1 * b0
    p11 = a1 * b1
    # middle column: carries out of bit 64 of the low half
    mid = (p00 >> _S32) + (p01 & _MASK32) + (p10 & _MASK32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    lo = a * b  # wraps modulo 2^64
    return hi, lo


def philox4x64(counter, key, rounds: int = ROUNDS):
    """Apply Philox4x64-`rounds` to counters.

    counter: uint64 array of shape (..., 4); key: pair of uint64 (or arrays
    broadcastable to counter[..., 0]).  Returns uint64 array of shape (..., 4).
    """
    with np.errstate(over="ignore"):
        ctr = np.asarray(counter, dtype=np.uint64)
        x0, x1, x2, x3 = (ctr[..., i].copy() for i in range(4))
        k0 = np.asarray(key[0], dtype=np.uint64) + np.zeros_like(x0)
        k1 = np.asarray(key[1], dtype=np.uint64) + np.zeros_like(x0)
        m0, m1 = np.uint64(M0), np.uint64(M1)
        w0, w1 = np.uint64(W0), np.uint64(W1)
        for r in range(rounds):
            hi0, lo0 = mulhilo64(m0, x0)
            hi1, lo1 = mulhilo64(m1, x2)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
            if r != rounds - 1:
                k0 = k0 + w0
                k1 = k1 + w1
        return np.stack([x0, x1, x2, x3], axis=-1)
