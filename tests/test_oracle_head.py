"""Pins of the output-head oracle (pre-FC structured dropout, FC layer,
softmax cross-entropy): a closed form at zero logits, central finite
differences of the whole head loss with respect to every input (y, W, c),
a brute-force product on tiny inputs, torch's cross-entropy as an
independent library routine, and the invariants of the dropped columns,
of a logit shift per row and of ignored rows."""
import numpy as np
import pytest

from oracle import head


def _data(T=3, B=2, F=5, V=7, p=0.4, seed=0):
    rng = np.random.default_rng(seed)
    y = rng.normal(size=(T, B, F))
    W = rng.normal(size=(F, V)) * 0.5
    c = rng.normal(size=(V,)) * 0.1
    m = (rng.random((T, F)) >= p).astype(np.uint8)
    m[0, 0], m[0, 1] = 0, 1                   # at least one dropped and one kept column
    tgt = rng.integers(0, V, size=(T, B))
    return y, W, c, m, tgt


def test_zero_logits_closed_form():
    T, B, V = 2, 3, 11
    z = np.zeros((T, B, V))
    tgt = np.arange(T * B).reshape(T, B) % V
    loss, dz = head.softmax_xent(z, tgt)
    assert loss == pytest.approx(np.log(V), rel=0, abs=1e-14)
    ref = np.full((T, B, V), 1.0 / V)
    for t in range(T):
        for b in range(B):
            ref[t, b, tgt[t, b]] -= 1.0
    assert np.allclose(dz, ref / (T * B), rtol=0, atol=1e-15)


def test_brute_force_forward():
    y, W, c, m, _ = _data(T=2, B=2, F=3, V=4, p=0.5, seed=1)
    p = 0.5
    z = head.head_forward(y, W, c, m, p)
    for t in range(2):
        for b in range(2):
            for v in range(4):
                acc = c[v]
                for k in range(3):
                    if m[t, k]:
                        acc += y[t, b, k] / (1 - p) * W[k, v]
                assert z[t, b, v] == pytest.approx(acc, rel=1e-13, abs=1e-13)


def _loss(y, W, c, m, p, tgt, lengths=None):
    return head.softmax_xent(head.head_forward(y, W, c, m, p), tgt, lengths)[0]


@pytest.mark.parametrize("p", [0.0, 0.4])
def test_finite_differences_of_the_head(p):
    y, W, c, m, tgt = _data(p=0.4, seed=2)
    if p == 0.0:
        m = np.ones_like(m)
    g = head.head_step(y, W, c, m, p, tgt)
    h = 1e-6
    for arr, grad in ((y, g["dy"]), (W, g["dW"]), (c, g["dc"])):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + h
            lp = _loss(y, W, c, m, p, tgt)
            arr[idx] = old - h
            lm = _loss(y, W, c, m, p, tgt)
            arr[idx] = old
            num[idx] = (lp - lm) / (2 * h)
        assert np.allclose(grad, num, rtol=1e-6, atol=1e-8), np.abs(grad - num).max()


def test_matches_torch_cross_entropy():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    T, B, V = 4, 5, 9
    z = rng.normal(size=(T, B, V)) * 3
    tgt = rng.integers(0, V, size=(T, B))
    tgt[1, 2] = -100                           # torch's default ignore index: outside [0, V)
    loss, dz = head.softmax_xent(z, tgt)
    zt = torch.tensor(z.reshape(-1, V), dtype=torch.float64, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(tgt.reshape(-1)), ignore_index=-100)
    lt.backward()
    assert loss == pytest.approx(float(lt), rel=1e-13)
    assert np.allclose(dz.reshape(-1, V), zt.grad.numpy(), rtol=0, atol=1e-15)


def test_dropped_columns_and_never_kept_rows():
    y, W, c, m, tgt = _data(T=4, B=3, F=6, V=5, seed=4)
    m[:, 3] = 0                                # feature 3 never kept
    p = 0.3
    g = head.head_step(y, W, c, m, p, tgt)
    y2 = y + (1 - m[:, None, :]) * 1e3         # garbage in the dropped columns
    g2 = head.head_step(y2, W, c, m, p, tgt)
    assert np.allclose(g["z"], g2["z"], rtol=0, atol=1e-12)
    assert not (g["dy"] * (1 - m[:, None, :])).any()
    assert not g["dW"][3].any()


def test_shift_invariance_and_large_logits():
    rng = np.random.default_rng(5)
    z = rng.normal(size=(2, 3, 6))
    tgt = rng.integers(0, 6, size=(2, 3))
    l0, d0 = head.softmax_xent(z, tgt)
    l1, d1 = head.softmax_xent(z + rng.normal(size=(2, 3, 1)) * 1e3, tgt)
    assert l1 == pytest.approx(l0, rel=1e-9)
    assert np.allclose(d1, d0, rtol=0, atol=1e-12)
    # two classes: loss = log(1 + e^{-(z_t - z_o)}), stable at large margins
    z2 = np.array([[[800.0, 0.0]]])
    l2, _ = head.softmax_xent(z2, np.array([[1]]))
    assert l2 == pytest.approx(800.0, rel=1e-15)


def test_lengths_and_ignored_targets_drop_rows():
    rng = np.random.default_rng(6)
    T, B, V = 5, 3, 4
    z = rng.normal(size=(T, B, V))
    tgt = rng.integers(0, V, size=(T, B))
    lengths = np.array([5, 2, 0])
    tgt[0, 0] = V                              # out of range: ignored
    loss, dz = head.softmax_xent(z, tgt, lengths)
    ok = head.valid_rows(tgt, V, lengths)
    assert ok.sum() == 5 + 2 - 1
    # the same loss over the valid rows alone, as a flat batch
    tt, bb = np.nonzero(ok)
    ls, ds = head.softmax_xent(z[tt, bb][None], tgt[tt, bb][None])
    assert loss == pytest.approx(ls, rel=1e-14)
    assert np.allclose(dz[tt, bb], ds[0], rtol=0, atol=1e-15)
    assert not dz[~ok].any()
    # no valid row at all: zero loss and gradient
    l0, d0 = head.softmax_xent(z, np.full((T, B), -1))
    assert l0 == 0.0 and not d0.any()
