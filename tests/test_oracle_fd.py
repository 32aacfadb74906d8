"""Pins the oracle's hand-written BPTT by central finite differences of its
own forward pass (float64, tiny shapes), masks fixed."""
import numpy as np
import pytest

from oracle import lstm
from tests._oracle_helpers import tiny_problem

EPS = 1e-6


def _loss(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths, R, kind):
    y, hT, cT, _ = lstm.forward(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    if kind == "lin":
        return float(np.sum(y * R) + 0.7 * np.sum(hT) - 0.4 * np.sum(cT))
    return lstm.loss_mse(y, R, lengths)[0]


def _check(f, arr, analytic, rel=1e-6):
    num = np.zeros_like(arr)
    it = np.nditer(arr, flags=["multi_index"])
    for _ in it:
        idx = it.multi_index
        old = arr[idx]
        arr[idx] = old + EPS
        fp = f()
        arr[idx] = old - EPS
        fm = f()
        arr[idx] = old
        num[idx] = (fp - fm) / (2 * EPS)
    err = np.linalg.norm(num - analytic) / max(np.linalg.norm(num), 1e-30)
    assert err < rel, err


@pytest.mark.parametrize("L,D,p_nr,p_rh,with_len,kind", [
    (1, 1, 0.5, 0.0, False, "lin"),
    (2, 1, 0.5, 0.5, False, "lin"),
    (1, 2, 0.3, 0.5, True, "lin"),
    (2, 2, 0.5, 0.3, True, "mse"),
    (2, 1, 0.0, 0.0, True, "mse"),
])
def test_fd_all_parameters(L, D, p_nr, p_rh, with_len, kind):
    T, B, I, H = 4, 3, 4, 3
    lengths = np.array([4, 2, 1]) if with_len else None
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=L, D=D, I=I, H=H, B=B, T=T, p_nr=p_nr, p_rh=p_rh,
                                               seed=31 + L + 3 * D, mask_seed=5)
    R = np.random.default_rng(2).normal(size=(T, B, D * H))
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    if kind == "lin":
        g = lstm.backward(cache, R, dhT=0.7 * np.ones_like(hT), dcT=-0.4 * np.ones_like(cT))
    else:
        _, dy = lstm.loss_mse(y, R, lengths)
        g = lstm.backward(cache, dy)
    f = lambda: _loss(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths, R, kind)
    _check(f, x, g["dx"])
    _check(f, h0, g["dh0"])
    _check(f, c0, g["dc0"])
    for k in range(L * D):
        _check(f, P.W[k], g["dW"][k])
        _check(f, P.U[k], g["dU"][k])
        _check(f, P.b[k], g["db"][k])


def test_loss_mse_gradient_fd():
    rng = np.random.default_rng(0)
    y = rng.normal(size=(3, 4, 2))
    tg = rng.normal(size=(3, 4, 2))
    lengths = np.array([3, 1, 2, 0])
    _, dy = lstm.loss_mse(y, tg, lengths)
    _check(lambda: lstm.loss_mse(y, tg, lengths)[0], y, dy)
