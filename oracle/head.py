"""Output head of an LSTM language model under structured dropout: the
pre-FC output dropout, the FC (vocabulary projection) layer and the softmax
cross-entropy loss.  TEST INFRASTRUCTURE ONLY, like the rest of this package.

The paper's timings cover the products of the LSTM and of the FC layers
after compaction (Sec. 4, experimental setup); its language models drop the
LSTM output before the FC layer (Sec. 4.1, the AWD-LSTM dropout vector) and
its translation models add dropout on the final encoder/decoder outputs,
the decoder's projection being sized by the vocabulary (Sec. 4.2).  The FC
layer is one linear map, so a Case-III mask on its input (one keep bit per
feature and time step, shared by the batch; Sec. 3.1) propagates as in
Sec. 3.2 (Eq. 7-11 applied to a single product): the forward product reads
only the kept input columns, the input gradient is non-zero only in the
kept columns, and the weight gradient only in the kept rows at each t.

Notation: y [T][B][F] the top LSTM output, m [T][F] the output keep mask,
s = 1/(1-p) the inverted-dropout scale, W [F][V] (input-major, as the LSTM
weights), c [V] the bias, z [T][B][V] the logits, tgt [T][B] the target
token ids.  Everything is float64.
"""
from __future__ import annotations

import numpy as np


def head_forward(y, W, c, m, p):
    """z[t][b] = (s * m[t] * y[t][b]) @ W + c."""
    s = 1.0 / (1.0 - p)
    yt = y.astype(np.float64) * (s * m.astype(np.float64))[:, None, :]
    return yt @ W.astype(np.float64) + c.astype(np.float64)


def valid_rows(tgt, V, lengths=None):
    """[T][B] bool: rows that carry loss: t < length and a target in [0, V)
    (other targets act as an ignore index)."""
    T, B = tgt.shape
    ok = (tgt >= 0) & (tgt < V)
    if lengths is not None:
        ok &= np.arange(T)[:, None] < np.asarray(lengths)[None, :]
    return ok


def softmax_xent(z, tgt, lengths=None):
    """Mean cross-entropy over the valid rows and its gradient:
    loss = (1/N) sum_rows (logsumexp(z_row) - z_row[tgt]),
    dz_row = (softmax(z_row) - onehot(tgt)) / N on valid rows, 0 elsewhere.
    N = number of valid rows (loss 0, dz 0 when there are none)."""
    z = z.astype(np.float64)
    T, B, V = z.shape
    ok = valid_rows(tgt, V, lengths)
    N = int(ok.sum())
    mx = z.max(axis=2, keepdims=True)
    e = np.exp(z - mx)
    se = e.sum(axis=2, keepdims=True)
    lse = (mx + np.log(se))[:, :, 0]
    prob = e / se
    dz = np.zeros_like(z)
    loss = 0.0
    if N:
        tt, bb = np.nonzero(ok)
        tv = tgt[tt, bb]
        loss = float((lse[tt, bb] - z[tt, bb, tv]).sum() / N)
        dz[tt, bb] = prob[tt, bb]
        dz[tt, bb, tv] -= 1.0
        dz /= N
    return loss, dz


def head_backward(y, W, m, p, dz):
    """Gradients of the head given dz = dL/dz:
    dy[t][b] = s * m[t] * (dz[t][b] @ W^T)      (zero in dropped columns)
    dW = s * sum_t (m[t] * y[t])^T @ dz[t]       (zero rows where never kept)
    dc = sum_t sum_b dz[t][b]."""
    s = 1.0 / (1.0 - p)
    mm = m.astype(np.float64)
    W = W.astype(np.float64)
    dy = s * mm[:, None, :] * (dz @ W.T)
    ym = y.astype(np.float64) * mm[:, None, :]
    dW = s * np.einsum("tbk,tbv->kv", ym, dz)
    dc = dz.sum(axis=(0, 1))
    return dy, dW, dc


def head_step(y, W, c, m, p, tgt, lengths=None):
    """Forward, loss and backward of the head: a dict with z, loss, dz, dy,
    dW, dc."""
    z = head_forward(y, W, c, m, p)
    loss, dz = softmax_xent(z, tgt, lengths)
    dy, dW, dc = head_backward(y, W, m, p, dz)
    return dict(z=z, loss=loss, dz=dz, dy=dy, dW=dW, dc=dc)
