"""Case-III structured dropout masks (Sec. 3.1 and Fig. 1 caption): the
pattern is the same for every row of the batch (whole neurons are dropped)
and is drawn afresh at every time step.  Test infrastructure only.

The paper does not specify the random source.  Reading used here (and by the
HIP library, implemented independently):

  * one 64-bit uniform word per (stream, time step t, neuron k, training
    step): Philox4x64-10 with key (seed, 0) and counter
    (k // 4, t, stream, step); the word is lane k % 4 of the output block;
  * neuron k is dropped at t iff word < floor(p * 2**64), computed exactly
    with Python integers, so the drop decision is integer and bit-exact;
  * stream ids: the non-recurrent (NR) input of layer l uses 4*l; the
    recurrent (RH) input of layer l, direction d uses 4*l + 2 + d; the
    output (pre-FC) site of an L-layer stack uses 4*L, the NR stream a
    layer L would have (the FC layer is the next consumer of the output).

A keep list is the ascending list of kept neuron indices at one t; its
length is the keep count.  The paper calls packing the kept rows "matrix
compaction" (Sec. 4); the keep list is what that compaction gathers by.
"""
from __future__ import annotations

import numpy as np

from .philox import philox4x64


def drop_threshold(p: float) -> int:
    """floor(p * 2^64) as an exact integer, for 0 <= p < 1."""
    if not (0.0 <= p < 1.0):
        raise ValueError("dropout rate must be in [0, 1)")
    # p is a binary64 value; scaling by 2^64 is exact, floor is exact.
    from fractions import Fraction
    return int(Fraction(p) * (1 << 64))


def nr_stream(layer: int) -> int:
    return 4 * layer


def rh_stream(layer: int, direction: int) -> int:
    return 4 * layer + 2 + direction


def out_stream(num_layers: int) -> int:
    return 4 * num_layers


def uniform_words(seed: int, step: int, stream: int, T: int, K: int) -> np.ndarray:
    """The 64-bit words u[t][k] for one stream: shape [T][K], uint64."""
    seed &= (1 << 64) - 1
    nblk = (K + 3) // 4
    t_idx, b_idx = np.meshgrid(np.arange(T, dtype=np.uint64),
                               np.arange(nblk, dtype=np.uint64), indexing="ij")
    ctr = np.stack([b_idx, t_idx,
                    np.full_like(t_idx, np.uint64(stream)),
                    np.full_like(t_idx, np.uint64(step))], axis=-1)
    out = philox4x64(ctr, (np.uint64(seed), np.uint64(0)))  # [T][nblk][4]
    return out.reshape(T, nblk * 4)[:, :K]


def keep_mask(seed: int, step: int, stream: int, T: int, K: int, p: float) -> np.ndarray:
    """m[t][k] in {0, 1} (uint8): 1 = kept.  p == 0 keeps everything."""
    thr = drop_threshold(p)
    u = uniform_words(seed, step, stream, T, K)
    if thr == 0:
        return np.ones((T, K), dtype=np.uint8)
    drop = u < np.uint64(thr)
    return (~drop).astype(np.uint8)


def keep_mask_fixed(seed: int, step: int, stream: int, T: int, K: int, p: float) -> np.ndarray:
    """Case-IV (Sec. 3: structured in the batch and the same at every time
    step): the draw of t = 0 repeated at every t."""
    return np.repeat(keep_mask(seed, step, stream, 1, K, p), T, axis=0)


def keep_lists(mask: np.ndarray):
    """Ascending kept indices per t and their counts."""
    lists = [np.nonzero(mask[t])[0].astype(np.int32) for t in range(mask.shape[0])]
    counts = np.array([len(k) for k in lists], dtype=np.int32)
    return lists, counts


def all_masks(seed: int, step: int, num_layers: int, num_dirs: int, T: int,
              k_in, hidden: int, p_nr, p_rh, fixed: bool = False):
    """Masks for every site of a stacked (bi)LSTM.  p_nr and p_rh are one
    rate for every layer or a sequence of one rate per layer (each site then
    draws with its own layer's rate).

    Returns (nr, rh): nr[l] is [T][k_in(l)], rh[l][d] is [T][hidden].
    """
    draw = keep_mask_fixed if fixed else keep_mask
    rate = lambda p, l: float(p[l]) if isinstance(p, (list, tuple, np.ndarray)) else float(p)
    nr = [draw(seed, step, nr_stream(l), T, k_in(l), rate(p_nr, l)) for l in range(num_layers)]
    rh = [[draw(seed, step, rh_stream(l, d), T, hidden, rate(p_rh, l)) for d in range(num_dirs)]
          for l in range(num_layers)]
    return nr, rh
