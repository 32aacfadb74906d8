"""Pins the oracle against closed forms derived by hand.

With W = U = 0 and b = 0 every gate pre-activation is 0, so i = f = o = 1/2
and g = 0 whatever the input and the masks: c_t = c_{t-1}/2, h_t = tanh(c_t)/2.
For the loss L = sum_t sum h_t of a single-layer LSTM the backward pass then
reduces to scalar recursions (dU^T terms vanish):
    dc_t  = (1 - tanh^2 c_t)/2 + dc_{t+1}/2
    da_i  = 0 (g = 0),  da_f = dc_t c_{t-1}/4,  da_g = dc_t/2,  da_o = tanh(c_t)/4
    dc0   = dc_0/2,  dh0 = 0,  dx = 0."""
import numpy as np
import pytest

from oracle import lstm, masks


@pytest.mark.parametrize("p_nr,p_rh", [(0.0, 0.0), (0.5, 0.5), (0.7, 0.3)])
def test_zero_weights_closed_form(p_nr, p_rh):
    T, B, I, H = 6, 3, 4, 5
    rng = np.random.default_rng(1)
    P = lstm.params_from([np.zeros((I, 4 * H))], [np.zeros((H, 4 * H))], [np.zeros(4 * H)], 1, 1)
    x = rng.normal(size=(T, B, I))
    h0 = rng.normal(size=(1, B, H))
    c0 = rng.normal(size=(1, B, H))
    m_nr, m_rh = masks.all_masks(9, 0, 1, 1, T, lambda l: I, H, p_nr, p_rh)
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh)
    c = [c0[0] * 0.5 ** (t + 1) for t in range(T)]
    for t in range(T):
        assert np.allclose(y[t], 0.5 * np.tanh(c[t]), rtol=0, atol=1e-15)
    assert np.allclose(cT[0], c[-1], rtol=0, atol=1e-15)

    _, dy = lstm.loss_sum(y)
    g = lstm.backward(cache, dy)
    dc = [None] * T
    nxt = np.zeros((B, H))
    for t in range(T - 1, -1, -1):
        tc = np.tanh(c[t])
        dc[t] = 0.5 * (1 - tc ** 2) + 0.5 * nxt
        nxt = dc[t]
    db = np.zeros(4 * H)
    dW = np.zeros((I, 4 * H))
    s = 1.0 / (1.0 - p_nr) if p_nr > 0 else 1.0
    for t in range(T):
        cprev = c0[0] if t == 0 else c[t - 1]
        da = np.concatenate([np.zeros((B, H)), dc[t] * cprev / 4, dc[t] / 2, np.tanh(c[t]) / 4], axis=1)
        db += da.sum(0)
        dW += (x[t] * m_nr[0][t][None, :] * s).T @ da
    assert np.allclose(g["db"][0], db, rtol=0, atol=1e-13)
    assert np.allclose(g["dW"][0], dW, rtol=0, atol=1e-13)
    assert np.allclose(g["dc0"][0], 0.5 * dc[0], rtol=0, atol=1e-15)
    assert np.all(g["dh0"] == 0.0)
    assert np.all(g["dx"] == 0.0)
    # the i-gate columns of dW and dU get nothing because g == 0
    assert np.all(g["dW"][0][:, :H] == 0.0) and np.all(g["dU"][0][:, :H] == 0.0)
