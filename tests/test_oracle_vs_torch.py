"""Pins the oracle against PyTorch's own LSTM (float64, CPU).

p = 0: the oracle must equal torch.nn.LSTM (a library routine) for the
forward outputs and, through autograd, every gradient; with sequence lengths
the comparison goes through torch's packed sequences.
p > 0: the structured masks are applied to the inputs of torch.nn.LSTMCell
(the non-recurrent input x * m * s and the copy of h_{t-1} that enters U),
and torch's cell arithmetic plus autograd supply the reference values."""
import numpy as np
import pytest
import torch

from oracle import lstm
from tests._oracle_helpers import tiny_problem

TOL = 1e-11


def _torch_lstm(P, I):
    L, D, H = P.num_layers, P.num_dirs, P.hidden
    m = torch.nn.LSTM(I, H, num_layers=L, bidirectional=(D == 2), dtype=torch.float64)
    with torch.no_grad():
        for l in range(L):
            for d in range(D):
                sfx = f"_l{l}" + ("_reverse" if d == 1 else "")
                k = l * D + d
                getattr(m, "weight_ih" + sfx).copy_(torch.from_numpy(P.W[k].T.copy()))
                getattr(m, "weight_hh" + sfx).copy_(torch.from_numpy(P.U[k].T.copy()))
                getattr(m, "bias_ih" + sfx).copy_(torch.from_numpy(P.b[k]))
                getattr(m, "bias_hh" + sfx).zero_()
    return m


def _grads_of_module(m, P, l, d):
    sfx = f"_l{l}" + ("_reverse" if d == 1 else "")
    return (getattr(m, "weight_ih" + sfx).grad.numpy().T,
            getattr(m, "weight_hh" + sfx).grad.numpy().T,
            getattr(m, "bias_ih" + sfx).grad.numpy())


@pytest.mark.parametrize("L,D", [(1, 1), (2, 1), (1, 2), (2, 2), (3, 1)])
@pytest.mark.parametrize("with_lengths", [False, True])
def test_p0_equals_torch_lstm(L, D, with_lengths):
    T, B, I, H = 5, 4, 6, 3
    lengths = np.array([5, 2, 4, 1]) if with_lengths else None
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=L, D=D, I=I, H=H, B=B, T=T, p_nr=0.0, p_rh=0.0,
                                               seed=L * 10 + D)
    R = np.random.default_rng(5).normal(size=(T, B, D * H))
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, 0.0, 0.0, lengths)
    g = lstm.backward(cache, R)

    m = _torch_lstm(P, I)
    xt = torch.tensor(x, requires_grad=True)
    h0t = torch.tensor(h0, requires_grad=True)
    c0t = torch.tensor(c0, requires_grad=True)
    if with_lengths:
        packed = torch.nn.utils.rnn.pack_padded_sequence(xt, torch.tensor(lengths), enforce_sorted=False)
        out, (hn, cn) = m(packed, (h0t, c0t))
        yt, _ = torch.nn.utils.rnn.pad_packed_sequence(out, total_length=T)
    else:
        yt, (hn, cn) = m(xt, (h0t, c0t))
    (yt * torch.from_numpy(R)).sum().backward()

    assert np.allclose(y, yt.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(hT, hn.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(cT, cn.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dx"], xt.grad.numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dh0"], h0t.grad.numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dc0"], c0t.grad.numpy(), atol=TOL, rtol=0)
    for l in range(L):
        for d in range(D):
            gW, gU, gb = _grads_of_module(m, P, l, d)
            k = l * D + d
            assert np.allclose(g["dW"][k], gW, atol=TOL, rtol=0)
            assert np.allclose(g["dU"][k], gU, atol=TOL, rtol=0)
            assert np.allclose(g["db"][k], gb, atol=TOL, rtol=0)


def _masked_cells(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths):
    """Masked stacked (bi)LSTM built from torch.nn.LSTMCell; returns the
    output and everything that needs a gradient."""
    L, D, H = P.num_layers, P.num_dirs, P.hidden
    T, B, I = x.shape
    per_layer = lambda p: list(p) if isinstance(p, (list, tuple)) else [p] * L
    s_nr = [1.0 / (1.0 - p) if p > 0 else 1.0 for p in per_layer(p_nr)]
    s_rh = [1.0 / (1.0 - p) if p > 0 else 1.0 for p in per_layer(p_rh)]
    xt = torch.tensor(x, requires_grad=True)
    h0t = torch.tensor(h0, requires_grad=True)
    c0t = torch.tensor(c0, requires_grad=True)
    valid = torch.ones(T, B, dtype=torch.bool) if lengths is None else \
        (torch.arange(T)[:, None] < torch.tensor(lengths)[None, :])
    cells = []
    inp = xt
    hT, cT = [], []
    for l in range(L):
        mn = torch.tensor(m_nr[l], dtype=torch.float64)
        xin = inp * mn[:, None, :] * s_nr[l]
        outs = []
        for d in range(D):
            k = l * D + d
            cell = torch.nn.LSTMCell(xin.shape[-1], H, dtype=torch.float64)
            with torch.no_grad():
                cell.weight_ih.copy_(torch.from_numpy(P.W[k].T.copy()))
                cell.weight_hh.copy_(torch.from_numpy(P.U[k].T.copy()))
                cell.bias_ih.copy_(torch.from_numpy(P.b[k]))
                cell.bias_hh.zero_()
            cells.append(cell)
            mr = torch.tensor(m_rh[l][d], dtype=torch.float64)
            h, c = h0t[k], c0t[k]
            ys = [None] * T
            order = range(T) if d == 0 else range(T - 1, -1, -1)
            for t in order:
                hn, cn = cell(xin[t], (h * mr[t][None, :] * s_rh[l], c))
                v = valid[t][:, None]
                ys[t] = torch.where(v, hn, torch.zeros_like(hn))
                h = torch.where(v, hn, h)
                c = torch.where(v, cn, c)
            outs.append(torch.stack(ys))
            hT.append(h)
            cT.append(c)
        inp = torch.cat(outs, dim=-1)
    return inp, torch.stack(hT), torch.stack(cT), xt, h0t, c0t, cells


@pytest.mark.parametrize("L,D,p_nr,p_rh", [(2, 1, 0.5, 0.0), (2, 1, 0.5, 0.5), (1, 2, 0.3, 0.7),
                                           (2, 2, 0.65, 0.65), (3, 1, 0.7, 0.3),
                                           # a rate per layer (the AWD-LSTM dropout vector of Sec. 4.1)
                                           (3, 1, [0.4, 0.25, 0.25], [0.5, 0.5, 0.5]),
                                           (2, 2, [0.3, 0.6], [0.0, 0.45])])
@pytest.mark.parametrize("with_lengths", [False, True])
def test_masked_equals_torch_cells(L, D, p_nr, p_rh, with_lengths):
    T, B, I, H = 6, 4, 7, 5
    lengths = np.array([6, 3, 1, 5]) if with_lengths else None
    P, x, h0, c0, m_nr, m_rh, _ = tiny_problem(L=L, D=D, I=I, H=H, B=B, T=T, p_nr=p_nr, p_rh=p_rh,
                                               seed=7 + L + D, mask_seed=123)
    # the masks really drop something at these rates
    assert min(m.min() for m in m_nr) == 0
    R = np.random.default_rng(9).normal(size=(T, B, D * H))
    y, hT, cT, cache = lstm.forward(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    g = lstm.backward(cache, R, dhT=np.ones_like(hT) * 0.3, dcT=np.ones_like(cT) * -0.2)

    yt, hTt, cTt, xt, h0t, c0t, cells = _masked_cells(P, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    loss = (yt * torch.from_numpy(R)).sum() + 0.3 * hTt.sum() - 0.2 * cTt.sum()
    loss.backward()
    assert np.allclose(y, yt.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(hT, hTt.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(cT, cTt.detach().numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dx"], xt.grad.numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dh0"], h0t.grad.numpy(), atol=TOL, rtol=0)
    assert np.allclose(g["dc0"], c0t.grad.numpy(), atol=TOL, rtol=0)
    for k, cell in enumerate(cells):
        assert np.allclose(g["dW"][k], cell.weight_ih.grad.numpy().T, atol=TOL, rtol=0)
        assert np.allclose(g["dU"][k], cell.weight_hh.grad.numpy().T, atol=TOL, rtol=0)
        assert np.allclose(g["db"][k], cell.bias_ih.grad.numpy(), atol=TOL, rtol=0)
