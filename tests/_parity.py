"""Helpers of the GPU parity tests: oracle runs on the same seeded inputs and
normwise comparisons."""
import sys

import numpy as np

import workloads
from oracle import lstm, masks

TOL = {"f32": 1e-4, "bf16": 2e-2}


def mode_rates(cfg, mode, p):
    """(p_nr, p_rh, compact) of a mode: p on the NR sites (and the RH sites in
    the NR+RH modes), or the config's per-layer rate vectors when it has them."""
    m = workloads.MODES[mode]
    compact = 1 if m["compact"] else 0
    if cfg.p_nr_layers is not None:
        rh = list(cfg.p_rh_layers) if m["rh"] else 0.0
        return list(cfg.p_nr_layers), rh, compact
    return p, (p if m["rh"] else 0.0), compact


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


def rel_max(a, r):
    """max |a - r| / max |r| (elementwise error against the tensor's scale)."""
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    m = float(np.max(np.abs(r))) if r.size else 0.0
    d = float(np.max(np.abs(a - r))) if r.size else 0.0
    return d if m == 0 else d / m


BLK = 16     # the MFMA tile edge: a wrong or skipped tile shows up in one block


def rel_blocks(a, r, blk=BLK):
    """Largest normwise error over blk x blk blocks of the last two axes (blk
    runs of a 1-D tensor): ||a_blk - r_blk|| / max(||r_blk||, rms(r) sqrt(n_blk)).
    The floor keeps blocks of tiny reference values from dividing by ~0; a
    block that is wrong by its own size gives about 1 whatever its norm."""
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if r.size == 0:
        return 0.0
    if r.ndim == 1:
        a, r = a[None, :], r[None, :]
    lead = r.shape[:-2]
    R, C = r.shape[-2:]
    Rp, Cp = -(-R // blk) * blk, -(-C // blk) * blk
    pad = [(0, 0)] * len(lead) + [(0, Rp - R), (0, Cp - C)]
    d = np.pad(a - r, pad).reshape(*lead, Rp // blk, blk, Cp // blk, blk)
    rr = np.pad(r, pad).reshape(*lead, Rp // blk, blk, Cp // blk, blk)
    dn = np.sqrt((d ** 2).sum(axis=(-3, -1)))
    rn = np.sqrt((rr ** 2).sum(axis=(-3, -1)))
    rms = np.linalg.norm(r) / np.sqrt(r.size)
    if rms == 0:
        return float(dn.max())
    return float((dn / np.maximum(rn, rms * blk)).max())


def tensor_errors(name, a, r, out):
    """Three bounds per tensor: normwise, elementwise-max and per 16x16 block."""
    out[name] = rel(a, r)
    out[name + ".max"] = rel_max(a, r)
    out[name + ".blk"] = rel_blocks(a, r)


def compare(gpu, ref, keys=("y", "hT", "cT", "dx", "dh0", "dc0"), rows=None):
    errs = {}
    for k in keys:
        a, r = gpu[k], ref[k]
        if rows is not None:
            a = a[:, rows]
        tensor_errors(k, a, r, errs)
    for k in ("dW", "dU", "db"):
        for i, (a, r) in enumerate(zip(gpu[k], ref[k])):
            tensor_errors(f"{k}{i}", a, r, errs)
    return errs


def summary(errs):
    """The largest error of each kind (normwise, elementwise-max, block)."""
    kinds = {"norm": [v for k, v in errs.items() if "." not in k],
             "max": [v for k, v in errs.items() if k.endswith(".max")],
             "blk": [v for k, v in errs.items() if k.endswith(".blk")]}
    return {k: f"{max(v):.2e}" for k, v in kinds.items() if v}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def fwd_persist_launches(cfg, stacked=True):
    """Persistent launches per forward (or backward) pass: one for a
    unidirectional stack run in one launch, else one per layer."""
    if stacked and cfg.num_dirs == 1 and 1 < cfg.num_layers <= 4:
        return 1
    return cfg.num_layers
