"""Case-I ("NR+Random") comparator: unstructured dropout on every layer's
input, one keep bit per element (t, b, k), so no row of a product can be
skipped (Sec. 3 names the cases; the paper's NR+Random baselines, Sec. 4,
drop the non-recurrent inputs this way).  TEST INFRASTRUCTURE ONLY.

Random source (a reading, like the Case-III one): element (t, b, k) of the
input of layer l is dropped iff word k%4 of Philox4x64-10 with key (seed, 0)
and counter (k//4, t, 4l + 2^32 (b+1), step) is below floor(p * 2^64): the
Case-III generator with the batch row in the high word of the stream.

The step is the definition written out layer by layer: the input of layer l
is multiplied by its mask and by s = 1/(1-p), the layer runs without dropout
(the float64 LSTM of oracle.lstm with every mask 1), its output is the next
layer's input; the gradient of each layer's input goes back through the same
mask and scale.
"""
from __future__ import annotations

import numpy as np

from . import lstm, masks
from .philox import philox4x64


def element_mask(seed: int, step: int, stream: int, T: int, B: int, K: int, p: float) -> np.ndarray:
    """m[t][b][k] in {0, 1} (uint8)."""
    thr = masks.drop_threshold(p)
    if thr == 0:
        return np.ones((T, B, K), dtype=np.uint8)
    seed &= (1 << 64) - 1
    nblk = (K + 3) // 4
    t_i, b_i, q_i = np.meshgrid(np.arange(T, dtype=np.uint64), np.arange(B, dtype=np.uint64),
                                np.arange(nblk, dtype=np.uint64), indexing="ij")
    sw = np.uint64(stream) + ((b_i + np.uint64(1)) << np.uint64(32))
    ctr = np.stack([q_i, t_i, sw, np.full_like(t_i, np.uint64(step))], axis=-1)
    words = philox4x64(ctr, (np.uint64(seed), np.uint64(0))).reshape(T, B, nblk * 4)[:, :, :K]
    return (~(words < np.uint64(thr))).astype(np.uint8)


def all_element_masks(seed, step, num_layers, T, B, k_in, p):
    return [element_mask(seed, step, masks.nr_stream(l), T, B, k_in(l), p) for l in range(num_layers)]


def case1_step(W, U, b, x, h0, c0, num_layers, num_dirs, m, p, loss, target=None, lengths=None):
    """Forward, loss and backward of a stack under Case-I input dropout.
    W, U, b: per (l, d) as in oracle.lstm; m: per layer [T][B][K_in(l)].
    Returns y, loss, dx and the per-(l, d) dW, dU, db lists."""
    s = 1.0 / (1.0 - p)
    L, D = num_layers, num_dirs
    T = x.shape[0]
    H = U[0].shape[0]
    caches, inp = [], x.astype(np.float64)
    for l in range(L):
        xt = inp * m[l] * s
        P = lstm.params_from(W[l * D:(l + 1) * D], U[l * D:(l + 1) * D], b[l * D:(l + 1) * D], 1, D)
        ones_nr = [np.ones((T, xt.shape[2]), np.uint8)]
        ones_rh = [[np.ones((T, H), np.uint8) for _ in range(D)]]
        y, _, _, cache = lstm.forward(P, xt, h0[l * D:(l + 1) * D], c0[l * D:(l + 1) * D], ones_nr, ones_rh,
                                      0.0, 0.0, lengths)
        caches.append(cache)
        inp = y
    if loss == "sum":
        lv, dy = lstm.loss_sum(inp)
    else:
        lv, dy = lstm.loss_mse(inp, target, lengths)
    dW, dU, db = [None] * (L * D), [None] * (L * D), [None] * (L * D)
    for l in reversed(range(L)):
        g = lstm.backward(caches[l], dy)
        for d in range(D):
            dW[l * D + d], dU[l * D + d], db[l * D + d] = g["dW"][d], g["dU"][d], g["db"][d]
        dy = g["dx"] * m[l] * s
    return dict(y=inp, loss=lv, dx=dy, dW=dW, dU=dU, db=db)
