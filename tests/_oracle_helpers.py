"""Small shared helpers for the oracle tests (random tiny problems)."""
import numpy as np

from oracle import lstm, masks


def tiny_problem(L=2, D=1, I=5, H=3, B=3, T=4, p_nr=0.5, p_rh=0.0, seed=0, lengths=None,
                 mask_seed=77, step=0, scale=0.5):
    rng = np.random.default_rng(seed)
    W, U, b = [], [], []
    for l in range(L):
        kin = I if l == 0 else D * H
        for _ in range(D):
            W.append(rng.normal(0, scale, (kin, 4 * H)))
            U.append(rng.normal(0, scale, (H, 4 * H)))
            b.append(rng.normal(0, scale, (4 * H,)))
    P = lstm.params_from(W, U, b, L, D)
    x = rng.normal(0, 1.0, (T, B, I))
    h0 = rng.normal(0, 0.5, (L * D, B, H))
    c0 = rng.normal(0, 0.5, (L * D, B, H))
    kin = lambda l: I if l == 0 else D * H
    m_nr, m_rh = masks.all_masks(mask_seed, step, L, D, T, kin, H, p_nr, p_rh)
    return P, x, h0, c0, m_nr, m_rh, lengths
