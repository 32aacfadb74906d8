"""Helpers of the GPU parity tests: oracle runs on the same seeded inputs and
normwise comparisons."""
import sys

import numpy as np

import workloads
from oracle import lstm, masks

TOL = {"f32": 1e-4, "bf16": 2e-2}


def mode_rates(cfg, mode, p):
    m = workloads.MODES[mode]
    return p, (p if m["rh"] else 0.0), (1 if m["compact"] else 0)


def oracle_masks(cfg, p_nr, p_rh, step=0, T=None):
    T = cfg.seq_len if T is None else T
    return masks.all_masks(cfg.mask_seed, step, cfg.num_layers, cfg.num_dirs, T, cfg.k_in,
                           cfg.hidden, p_nr, p_rh)


def site_list(cfg, m_nr, m_rh):
    """Masks in the library's site order: NR sites by layer, then RH by (l, d)."""
    out = list(m_nr)
    for l in range(cfg.num_layers):
        for d in range(cfg.num_dirs):
            out.append(m_rh[l][d])
    return out


def oracle_step(wl, p_nr, p_rh, m_nr, m_rh, dy=None):
    cfg = wl.cfg
    P = lstm.params_from(wl.W, wl.U, wl.b, cfg.num_layers, cfg.num_dirs)
    y, hT, cT, cache = lstm.forward(P, wl.x, wl.h0, wl.c0, m_nr, m_rh, p_nr, p_rh, wl.lengths)
    if dy is None:
        if cfg.loss == "sum":
            loss, dy = lstm.loss_sum(y)
        else:
            loss, dy = lstm.loss_mse(y, wl.target, wl.lengths)
    else:
        loss = None
    g = lstm.backward(cache, dy)
    return dict(y=y, hT=hT, cT=cT, loss=loss, dy=dy, **g)


def rel(a, r):
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    n = np.linalg.norm(r)
    if n == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - r) / n)


def compare(gpu, ref, keys=("y", "hT", "cT", "dx", "dh0", "dc0"), rows=None):
    errs = {}
    for k in keys:
        a, r = gpu[k], ref[k]
        if rows is not None:
            a = a[:, rows]
        errs[k] = rel(a, r)
    for k in ("dW", "dU", "db"):
        for i, (a, r) in enumerate(zip(gpu[k], ref[k])):
            errs[f"{k}{i}"] = rel(a, r)
    return errs


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def fwd_persist_launches(cfg, stacked=True):
    """Persistent launches per forward (or backward) pass: one for a
    unidirectional stack run in one launch, else one per layer."""
    if stacked and cfg.num_dirs == 1 and 1 < cfg.num_layers <= 4:
        return 1
    return cfg.num_layers
