"""Pins of the embedding-gradient oracle: special cases with a closed form
(distinct tokens, one token everywhere), a library scatter-add on random
data, accumulation into the existing gradient, the dropped columns, and
tokens outside the table."""
import numpy as np

from oracle import embedding


def _data(T=4, B=3, I=7, V=11, seed=0, p=0.5):
    rng = np.random.default_rng(seed)
    tok = rng.integers(0, V, size=(T, B))
    m = (rng.random((T, I)) >= p).astype(np.uint8)
    dx = rng.normal(size=(T, B, I)) * m[:, None, :]      # dropped columns are zero (Eq. 10)
    return tok, dx, m


def test_distinct_tokens_copy_rows():
    T, B, I = 3, 4, 5
    tok = np.arange(T * B).reshape(T, B)
    _, dx, m = _data(T, B, I, V=T * B)
    d = embedding.embedding_grad(tok, dx, m, np.zeros((T * B, I)))
    assert np.array_equal(d, dx.reshape(T * B, I))


def test_one_token_sums_every_row():
    T, B, I = 5, 3, 6
    _, dx, m = _data(T, B, I)
    tok = np.full((T, B), 2)
    d = embedding.embedding_grad(tok, dx, m, np.zeros((4, I)))
    assert np.allclose(d[2], dx.sum(axis=(0, 1)), rtol=0, atol=1e-12)
    assert not d[[0, 1, 3]].any()


def test_matches_library_scatter_add():
    tok, dx, m = _data(T=9, B=7, I=13, V=17, seed=3)
    ref = np.zeros((17, 13))
    np.add.at(ref, tok.reshape(-1), dx.reshape(-1, 13))
    d = embedding.embedding_grad(tok, dx, m, np.zeros((17, 13)))
    assert np.allclose(d, ref, rtol=0, atol=1e-12)


def test_accumulates_and_skips_dropped_columns():
    tok, dx, m = _data(T=4, B=2, I=5, V=6, seed=5)
    base = np.random.default_rng(9).normal(size=(6, 5))
    # garbage in the dropped columns must not reach the gradient
    dx_noisy = dx + (1 - m[:, None, :]) * 1e6
    d = embedding.embedding_grad(tok, dx_noisy, m, base.copy())
    ref = base.copy()
    np.add.at(ref, tok.reshape(-1), dx.reshape(-1, 5))
    assert np.allclose(d, ref, rtol=0, atol=1e-9)


def test_out_of_range_tokens_are_skipped():
    tok, dx, m = _data(T=3, B=2, I=4, V=5, seed=7)
    tok = tok.copy()
    tok[0, 0] = -1
    tok[1, 1] = 5
    d = embedding.embedding_grad(tok, dx, m, np.zeros((5, 4)))
    ok = (tok >= 0) & (tok < 5)
    ref = np.zeros((5, 4))
    np.add.at(ref, tok[ok], dx[ok])
    assert np.allclose(d, ref, rtol=0, atol=1e-12)
