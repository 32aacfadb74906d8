"""Pins of the Case-I ("NR+Random") comparator oracle: the per-element mask
against a one-counter recomputation of its definition, its drop fraction and
its variation over batch rows; and the whole step against torch.nn.LSTM
(float64, autograd), one single-layer module per layer with the layer input
multiplied by the mask and the scale."""
import numpy as np
import pytest
import torch

from oracle import case1, masks
from oracle.philox import philox4x64
from tests._oracle_helpers import tiny_problem


def test_element_mask_definition_and_statistics():
    T, B, K, p = 3, 5, 1000, 0.4
    m = case1.element_mask(9, 4, 8, T, B, K, p)
    thr = masks.drop_threshold(p)
    for (t, b, k) in [(0, 0, 0), (2, 4, 999), (1, 3, 517)]:
        ctr = np.array([[k // 4, t, 8 + ((b + 1) << 32), 4]], dtype=np.uint64)
        w = philox4x64(ctr, (np.uint64(9), np.uint64(0)))[0][k % 4]
        assert m[t, b, k] == (0 if int(w) < thr else 1)
    assert abs(1.0 - m.mean() - p) < 5 * np.sqrt(p * (1 - p) / m.size)
    assert not np.array_equal(m[0, 0], m[0, 1])          # rows of the batch differ (unstructured)
    assert np.array_equal(case1.element_mask(9, 4, 8, T, B, K, 0.0), np.ones((T, B, K), np.uint8))


def _torch_layer(W, U, b, D):
    I, H = W[0].shape[0], U[0].shape[0]
    mod = torch.nn.LSTM(I, H, num_layers=1, bidirectional=(D == 2), dtype=torch.float64)
    with torch.no_grad():
        for d in range(D):
            sfx = "_l0" + ("_reverse" if d == 1 else "")
            getattr(mod, "weight_ih" + sfx).copy_(torch.from_numpy(W[d].T.copy()))
            getattr(mod, "weight_hh" + sfx).copy_(torch.from_numpy(U[d].T.copy()))
            getattr(mod, "bias_ih" + sfx).copy_(torch.from_numpy(b[d]))
            getattr(mod, "bias_hh" + sfx).zero_()
    return mod


@pytest.mark.parametrize("L,D", [(2, 1), (1, 2), (3, 1)])
def test_step_equals_torch(L, D):
    P, x, h0, c0, _, _, _ = tiny_problem(L=L, D=D, I=6, H=4, B=3, T=5)
    p = 0.4
    kin = lambda l: 6 if l == 0 else D * 4
    m = case1.all_element_masks(21, 1, L, 5, 3, kin, p)
    target = np.random.default_rng(3).normal(size=(5, 3, D * 4))
    ref = case1.case1_step(P.W, P.U, P.b, x, h0, c0, L, D, m, p, "mse", target)
    xt = torch.tensor(x, requires_grad=True)
    inp, mods = xt, []
    for l in range(L):
        mod = _torch_layer(P.W[l * D:(l + 1) * D], P.U[l * D:(l + 1) * D], P.b[l * D:(l + 1) * D], D)
        mods.append(mod)
        xin = inp * torch.from_numpy(m[l].astype(np.float64)) / (1 - p)
        inp, _ = mod(xin, (torch.from_numpy(h0[l * D:(l + 1) * D]), torch.from_numpy(c0[l * D:(l + 1) * D])))
    loss = ((inp - torch.from_numpy(target)) ** 2).mean()
    loss.backward()
    assert ref["loss"] == pytest.approx(float(loss), rel=1e-12)
    assert np.allclose(ref["y"], inp.detach().numpy(), rtol=0, atol=1e-12)
    assert np.allclose(ref["dx"], xt.grad.numpy(), rtol=0, atol=1e-12)
    for l in range(L):
        for d in range(D):
            sfx = "_l0" + ("_reverse" if d == 1 else "")
            k = l * D + d
            assert np.allclose(ref["dW"][k], getattr(mods[l], "weight_ih" + sfx).grad.numpy().T, atol=1e-12)
            assert np.allclose(ref["dU"][k], getattr(mods[l], "weight_hh" + sfx).grad.numpy().T, atol=1e-12)
            assert np.allclose(ref["db"][k], getattr(mods[l], "bias_ih" + sfx).grad.numpy(), atol=1e-12)
