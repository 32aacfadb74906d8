"""Pins the oracle's Case-III mask draw (Sec. 3.1): statistics, exact
thresholds, the counter layout, determinism and stream independence."""
import numpy as np
import pytest

from oracle import masks
from oracle.philox import philox4x64


def test_threshold_exact():
    assert masks.drop_threshold(0.0) == 0
    assert masks.drop_threshold(0.5) == 1 << 63
    assert masks.drop_threshold(0.25) == 1 << 62
    assert masks.drop_threshold(0.75) == 3 << 62
    # 0.3 is not dyadic: floor of the exact binary64 value times 2^64
    from fractions import Fraction
    assert masks.drop_threshold(0.3) == (Fraction(0.3) * (1 << 64)).__floor__()
    assert masks.drop_threshold(np.nextafter(1.0, 0.0)) == (1 << 64) - (1 << 11)
    for bad in (-0.1, 1.0, 1.5):
        with pytest.raises(ValueError):
            masks.drop_threshold(bad)


def test_counter_layout_brute_force():
    seed, step, stream, T, K = 1234567, 3, 6, 5, 11
    u = masks.uniform_words(seed, step, stream, T, K)
    for t in range(T):
        for k in range(K):
            blk = philox4x64(np.array([k // 4, t, stream, step], dtype=np.uint64),
                             (np.uint64(seed), np.uint64(0)))
            assert u[t, k] == blk[k % 4]


@pytest.mark.parametrize("p", [0.3, 0.5, 0.65, 0.7])
def test_drop_fraction(p):
    T, K = 1000, 1000
    m = masks.keep_mask(42, 0, 2, T, K, p)
    n = T * K
    drop = n - int(m.sum())
    sigma = np.sqrt(n * p * (1 - p))
    assert abs(drop - n * p) < 5 * sigma
    # each time step varies (Case-III randomised in time)
    assert len({m[t].tobytes() for t in range(20)}) == 20


def test_p_zero_keeps_all():
    m = masks.keep_mask(1, 0, 0, 7, 33, 0.0)
    assert m.all()


def test_drop_decision_matches_threshold():
    seed, step, stream, T, K, p = 99, 1, 4, 6, 50, 0.5
    u = masks.uniform_words(seed, step, stream, T, K)
    m = masks.keep_mask(seed, step, stream, T, K, p)
    # p = 0.5: dropped iff the top bit of the word is clear
    assert np.array_equal(m, (u >> np.uint64(63)).astype(np.uint8))


def test_determinism_and_fresh_steps():
    a = masks.keep_mask(5, 0, 0, 10, 100, 0.5)
    b = masks.keep_mask(5, 0, 0, 10, 100, 0.5)
    c = masks.keep_mask(5, 1, 0, 10, 100, 0.5)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)


def test_streams_independent():
    T, K = 200, 1000
    a = masks.keep_mask(7, 0, masks.nr_stream(0), T, K, 0.5).astype(np.float64).ravel()
    b = masks.keep_mask(7, 0, masks.rh_stream(0, 0), T, K, 0.5).astype(np.float64).ravel()
    c = masks.keep_mask(7, 0, masks.rh_stream(0, 1), T, K, 0.5).astype(np.float64).ravel()
    n = a.size
    for x, y in ((a, b), (a, c), (b, c)):
        r = np.corrcoef(x, y)[0, 1]
        assert abs(r) < 5 / np.sqrt(n)


def test_keep_lists():
    m = masks.keep_mask(3, 0, 0, 9, 37, 0.6)
    lists, counts = masks.keep_lists(m)
    for t in range(9):
        assert np.all(np.diff(lists[t]) > 0)
        assert counts[t] == m[t].sum()
        assert np.all(m[t][lists[t]] == 1)


def test_stream_ids_distinct():
    ids = set()
    for l in range(4):
        ids.add(masks.nr_stream(l))
        for d in range(2):
            ids.add(masks.rh_stream(l, d))
    assert len(ids) == 12


def test_case4_fixed_masks():
    """Case-IV (one mask for the whole sequence): every row is the t = 0 row of
    the Case-III draw, and the drop fraction over many neurons is near p."""
    from oracle import masks as M
    T, K, p = 7, 4000, 0.3
    f = M.keep_mask_fixed(5, 2, M.nr_stream(1), T, K, p)
    c3 = M.keep_mask(5, 2, M.nr_stream(1), T, K, p)
    assert f.shape == (T, K)
    assert all(np.array_equal(f[t], c3[0]) for t in range(T))
    assert not all(np.array_equal(c3[t], c3[0]) for t in range(T))   # Case-III does vary in t
    assert abs(1.0 - f[0].mean() - p) < 5 * np.sqrt(p * (1 - p) / K)
    nr, rh = M.all_masks(5, 2, 2, 2, T, lambda l: 16 if l == 0 else 24, 12, p, p, fixed=True)
    assert all(np.array_equal(m, np.repeat(m[:1], T, axis=0)) for m in nr + [r for x in rh for r in x])


def test_per_layer_rates():
    """A rate per layer (the AWD-LSTM dropout vector): each site draws from
    its own stream with its own layer's threshold; the brute-force drop
    decision word < floor(p * 2^64) holds site by site, and each site's drop
    fraction sits within 5 sigma of its own rate."""
    T, H, I, L = 300, 400, 300, 3
    p_nr, p_rh = [0.4, 0.25, 0.1], [0.5, 0.0, 0.7]
    k_in = lambda l: I if l == 0 else H
    nr, rh = masks.all_masks(99, 4, L, 1, T, k_in, H, p_nr, p_rh)
    for l in range(L):
        for m, stream, p in ((nr[l], masks.nr_stream(l), p_nr[l]), (rh[l][0], masks.rh_stream(l, 0), p_rh[l])):
            u = masks.uniform_words(99, 4, stream, T, m.shape[1])
            thr = (int(p * 2 ** 53) << 11) if p in (0.5, 0.25) else masks.drop_threshold(p)
            assert np.array_equal(m == 0, u < np.uint64(thr)) if thr else m.all()
            n = m.size
            drop = n - int(m.sum())
            assert abs(drop - n * p) <= 5 * np.sqrt(n * p * (1 - p)) + 1e-9
