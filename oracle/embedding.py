"""Embedding gradient of an LSTM language model's input, the step just below
the LSTM (TEST INFRASTRUCTURE ONLY, like the rest of this package).

The model's layer-0 input is x_t[b] = E[tok_t[b]], a row lookup in an
embedding table E [V][I].  The gradient of the loss with respect to E is
therefore, for every row v,

    dE[v] = sum over (t, b) with tok_t[b] = v of dx_t[b]

where dx is the input gradient of Eq. 10 for layer 0.  Under structured
dropout dx_t is zero in the columns dropped at t (output sparsity, Eq. 10),
so only the kept columns of each row carry gradient; the product
accumulates those alone.  The sum is taken in ascending (t, b) order and
added to the existing dE (gradients accumulate), in float64 here.
"""
from __future__ import annotations

import numpy as np


def embedding_grad(tokens, dx, m_nr0, d_emb):
    """d_emb [V][I] (float64, updated in place and returned) += the rows of
    dx [T][B][I] gathered by tokens [T][B], restricted to the columns kept at
    each t (m_nr0 [T][I], layer 0's input mask).  Tokens outside [0, V) are
    skipped."""
    T, B = tokens.shape
    V = d_emb.shape[0]
    for t in range(T):
        keep = m_nr0[t].astype(bool)
        for b in range(B):
            v = int(tokens[t, b])
            if 0 <= v < V:
                d_emb[v, keep] += dx[t, b, keep]
    return d_emb
