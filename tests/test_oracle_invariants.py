"""Structural properties the paper states (Sec. 3.2), checked on the oracle:
output sparsity of the input gradients (Eq. 10), row sparsity of the weight
gradients (Eq. 11), the cell-state gradient not being sparse, and the
independence of batch rows under batch-shared masks."""
import numpy as np

from oracle import lstm
from tests._oracle_helpers import tiny_problem


def _run(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths=None, seed=4):
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    R = np.random.default_rng(seed).normal(size=y.shape)
    return y, lstm.backward(cache, R)


def test_never_kept_neuron_has_zero_weight_gradient_rows():
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=2, D=1, I=6, H=5, B=3, T=5, p_nr=0.5, p_rh=0.5)
    m_nr = [m.copy() for m in m_nr]
    m_rh = [[m.copy() for m in r] for r in m_rh]
    m_nr[0][:, 2] = 0
    m_nr[1][:, 4] = 0
    m_rh[1][0][:, 1] = 0
    _, g = _run(P, x, h0, c0, m_nr, m_rh, 0.5, 0.5)
    assert np.all(g["dW"][0][2] == 0.0)
    assert np.all(g["dW"][1][4] == 0.0)
    assert np.all(g["dU"][1][1] == 0.0)
    assert np.any(g["dW"][0][3] != 0.0)


def test_dropped_columns_of_input_gradient_are_zero():
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=2, D=2, I=6, H=4, B=3, T=5, p_nr=0.5, p_rh=0.5)
    _, g = _run(P, x, h0, c0, m_nr, m_rh, 0.5, 0.5)
    dropped = m_nr[0] == 0
    assert dropped.any()
    for t in range(x.shape[0]):
        assert np.all(g["dx"][t][:, dropped[t]] == 0.0)
        assert np.all(g["dx"][t][:, ~dropped[t]] != 0.0)
    # dh0 (the recurrent input of the first step) is zero where the first
    # step's RH mask dropped; forward direction starts at t=0, reverse at T-1
    T = x.shape[0]
    for l in range(2):
        for d in range(2):
            t0 = 0 if d == 0 else T - 1
            drop = m_rh[l][d][t0] == 0
            assert np.all(g["dh0"][l * 2 + d][:, drop] == 0.0)


def test_cell_gradient_not_sparse():
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=1, D=1, I=6, H=6, B=3, T=5, p_nr=0.5, p_rh=0.5)
    _, g = _run(P, x, h0, c0, m_nr, m_rh, 0.5, 0.5)
    drop = m_rh[0][0][0] == 0
    assert drop.any()
    assert np.all(g["dc0"][0][:, drop] != 0.0)


def test_batch_rows_independent():
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=2, D=2, I=5, H=4, B=6, T=4, p_nr=0.5, p_rh=0.3)
    lengths = np.array([4, 1, 3, 2, 4, 0])
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, 0.5, 0.3, lengths)
    rows = [1, 4, 5]
    y2, hT2, cT2, _ = lstm.forward(P, x[:, rows], h0[:, rows], c0[:, rows], m_nr, m_rh, 0.5, 0.3,
                                   lengths[rows])
    assert np.allclose(y[:, rows], y2, rtol=0, atol=1e-14)
    assert np.allclose(hT[:, rows], hT2, rtol=0, atol=1e-14)
    assert np.allclose(cT[:, rows], cT2, rtol=0, atol=1e-14)
    # gradient of a loss that only sees these rows equals the subset run's
    R = np.random.default_rng(1).normal(size=y.shape)
    Rz = np.zeros_like(R)
    Rz[:, rows] = R[:, rows]
    g = lstm.backward(cache, Rz)
    _, _, _, c2 = lstm.forward(P, x[:, rows], h0[:, rows], c0[:, rows], m_nr, m_rh, 0.5, 0.3, lengths[rows])
    g2 = lstm.backward(c2, R[:, rows])
    for k in range(4):
        assert np.allclose(g["dW"][k], g2["dW"][k], rtol=0, atol=1e-12)
        assert np.allclose(g["dU"][k], g2["dU"][k], rtol=0, atol=1e-12)
    assert np.allclose(g["dx"][:, rows], g2["dx"], rtol=0, atol=1e-13)


def test_zero_length_row_passes_state_through():
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=2, D=1, I=5, H=4, B=2, T=3, p_nr=0.5, p_rh=0.5)
    lengths = np.array([3, 0])
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, 0.5, 0.5, lengths)
    assert np.all(y[:, 1] == 0.0)
    assert np.array_equal(hT[:, 1], h0[:, 1]) and np.array_equal(cT[:, 1], c0[:, 1])
    dhT = np.random.default_rng(0).normal(size=hT.shape)
    dcT = np.random.default_rng(1).normal(size=cT.shape)
    g = lstm.backward(cache, np.zeros_like(y), dhT=dhT, dcT=dcT)
    assert np.array_equal(g["dh0"][:, 1], dhT[:, 1])
    assert np.array_equal(g["dc0"][:, 1], dcT[:, 1])
