"""Dense float64 LSTM with structured (batch-shared) dropout masks, and its
back-propagation through time, written out by hand.  Test infrastructure
only (see the package docstring); shares no code with the HIP library.

What is computed (row-vector convention of Eq. 1-4; gates stored as the
column blocks i | f | g | o of a [K][4H] weight, K-major):

  forward, layer l, direction d, time t (Eq. 1-6):
    x~_t     = x_t  * m_nr[l][t] * s_nr         input of layer l, masked
    h~_prev  = h_prev * m_rh[l][d][t] * s_rh    recurrent input, masked
    a_t      = x~_t W + h~_prev U + b
    i, f, o  = sigmoid(a_i, a_f, a_o);  g = tanh(a_g)
    c_t      = f * c_prev + i * g                (Eq. 5)
    h_t      = o * tanh(c_t)                     (Eq. 6)
  where s = 1/(1-p) (inverted dropout; the paper does not state the scale)
  and the masks are broadcast over the batch rows (Case-III, Sec. 3.1).
  Each rate is one number for every layer, or one per layer (a dropout
  vector with a rate per site, as the AWD-LSTM workload of Sec. 4.1 uses):
  layer l then takes p_nr[l] on its input and p_rh[l] on its recurrence.
  The recurrent mask touches only the copy of h_prev that enters U; the
  carried h and the cell state are never dropped (Sec. 3.2, FP paragraph).
  The reverse direction runs t = T-1 .. 0 with h_prev = h_{t+1}.  Layer
  output is the concatenation over directions.  Rows past their sequence
  length keep h and c frozen and output 0.

  backward (Eq. 7-11, in the direction's reverse time order):
    dh      = dy_t + (gradient carried from the next step)
    do      = dh * tanh(c_t)                     (Eq. 7)
    dc      = dh * o * (1 - tanh^2 c_t) + f_{t+1} * dc_{t+1}
    df      = dc * c_prev, di = dc * g, dg = dc * i, dc_prev = dc * f  (Eq. 8-9)
    da      = (di i(1-i), df f(1-f), dg (1-g^2), do o(1-o))
    dh_prev = (da U^T) * m_rh * s_rh             (Eq. 10; output masked)
    dx_t    = (da W^T) * m_nr * s_nr             (Eq. 10)
    dW += x~_t^T da,  dU += h~_prev^T da,  db += sum_b da   (Eq. 11, summed over t)
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np


def _sigmoid(z):
    # exact rewrite of 1/(1+exp(-z)) that does not overflow for large |z|
    e = np.exp(-np.abs(z))
    return np.where(z >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def _scale(p: float) -> float:
    return 1.0 / (1.0 - p) if p > 0.0 else 1.0


def layer_rate(p, l: int) -> float:
    """The rate of layer l: p itself, or p[l] for a per-layer sequence."""
    return float(p[l]) if isinstance(p, (list, tuple, np.ndarray)) else float(p)


@dataclasses.dataclass
class Params:
    """Weights per (layer, direction), index l*D + d, all float64."""
    W: List[np.ndarray]   # [K_in][4H]
    U: List[np.ndarray]   # [H][4H]
    b: List[np.ndarray]   # [4H]
    num_layers: int
    num_dirs: int

    @property
    def hidden(self):
        return self.U[0].shape[0]


@dataclasses.dataclass
class Cache:
    params: Params
    p_nr: float
    p_rh: float
    m_nr: list
    m_rh: list
    lengths: Optional[np.ndarray]
    layer_in: list          # per layer: x~ (masked, scaled input), [T][B][K]
    steps: list             # per (l, d): dict of per-t arrays
    y: np.ndarray


def _valid(lengths, T, B):
    if lengths is None:
        return np.ones((T, B), dtype=bool)
    return np.arange(T)[:, None] < np.asarray(lengths)[None, :]


def forward(params: Params, x, h0, c0, m_nr, m_rh, p_nr: float, p_rh: float,
            lengths=None):
    """Returns (y [T][B][D*H], hT [L*D][B][H], cT [L*D][B][H], cache)."""
    L, D, H = params.num_layers, params.num_dirs, params.hidden
    x = np.asarray(x, dtype=np.float64)
    T, B, _ = x.shape
    valid = _valid(lengths, T, B)
    hT = np.zeros((L * D, B, H))
    cT = np.zeros((L * D, B, H))
    inp = x
    layer_in, steps = [], []
    for l in range(L):
        s_nr, s_rh = _scale(layer_rate(p_nr, l)), _scale(layer_rate(p_rh, l))
        xt = inp * (np.asarray(m_nr[l], dtype=np.float64)[:, None, :] * s_nr)
        layer_in.append(xt)
        outs = []
        for d in range(D):
            k = l * D + d
            W, U, b = params.W[k], params.U[k], params.b[k]
            h = np.asarray(h0[k], dtype=np.float64).copy()
            c = np.asarray(c0[k], dtype=np.float64).copy()
            yd = np.zeros((T, B, H))
            rec = dict(order=[], i={}, f={}, g={}, o={}, c={}, c_prev={}, h_tilde={})
            order = range(T) if d == 0 else range(T - 1, -1, -1)
            mr = np.asarray(m_rh[l][d], dtype=np.float64)
            for t in order:
                h_tilde = h * (mr[t][None, :] * s_rh)
                a = xt[t] @ W + h_tilde @ U + b
                i = _sigmoid(a[:, 0:H])
                f = _sigmoid(a[:, H:2 * H])
                g = np.tanh(a[:, 2 * H:3 * H])
                o = _sigmoid(a[:, 3 * H:4 * H])
                c_new = f * c + i * g
                h_new = o * np.tanh(c_new)
                v = valid[t][:, None]
                rec["order"].append(t)
                for name, val in (("i", i), ("f", f), ("g", g), ("o", o), ("c", c_new),
                                  ("c_prev", c), ("h_tilde", h_tilde)):
                    rec[name][t] = val
                yd[t] = np.where(v, h_new, 0.0)
                h = np.where(v, h_new, h)
                c = np.where(v, c_new, c)
            hT[k], cT[k] = h, c
            outs.append(yd)
            steps.append(rec)
        inp = np.concatenate(outs, axis=-1)
    cache = Cache(params, p_nr, p_rh, m_nr, m_rh, lengths, layer_in, steps, inp)
    return inp, hT, cT, cache


def backward(cache: Cache, dy, dhT=None, dcT=None):
    """Gradients of a scalar loss given dL/dy (dy [T][B][D*H]).

    Returns dict with dx [T][B][I], dh0, dc0 [L*D][B][H], and lists dW, dU, db
    per (l, d)."""
    P = cache.params
    L, D, H = P.num_layers, P.num_dirs, P.hidden
    dy = np.asarray(dy, dtype=np.float64)
    T, B, _ = dy.shape
    valid = _valid(cache.lengths, T, B)
    dW = [None] * (L * D)
    dU = [None] * (L * D)
    db = [None] * (L * D)
    dh0 = np.zeros((L * D, B, H))
    dc0 = np.zeros((L * D, B, H))
    dout = dy                      # gradient w.r.t. the current layer's output
    for l in range(L - 1, -1, -1):
        s_nr, s_rh = _scale(layer_rate(cache.p_nr, l)), _scale(layer_rate(cache.p_rh, l))
        xt = cache.layer_in[l]
        dxt = np.zeros_like(xt)    # gradient w.r.t. x~ (masked input)
        for d in range(D):
            k = l * D + d
            rec = cache.steps[k]
            W, U = P.W[k], P.U[k]
            gW, gU, gb = np.zeros_like(W), np.zeros_like(U), np.zeros(4 * H)
            dh = np.zeros((B, H)) if dhT is None else np.asarray(dhT[k], dtype=np.float64).copy()
            dc = np.zeros((B, H)) if dcT is None else np.asarray(dcT[k], dtype=np.float64).copy()
            mr = np.asarray(cache.m_rh[l][d], dtype=np.float64)
            for t in reversed(rec["order"]):
                v = valid[t][:, None]
                i, f, g, o = rec["i"][t], rec["f"][t], rec["g"][t], rec["o"][t]
                c, c_prev = rec["c"][t], rec["c_prev"][t]
                dh_t = dh + np.where(v, dout[t][:, d * H:(d + 1) * H], 0.0)
                tc = np.tanh(c)
                do = dh_t * tc
                dct = dh_t * o * (1.0 - tc * tc) + dc
                df = dct * c_prev
                di = dct * g
                dg = dct * i
                dc_prev = dct * f
                da = np.concatenate([di * i * (1.0 - i), df * f * (1.0 - f),
                                     dg * (1.0 - g * g), do * o * (1.0 - o)], axis=1)
                da = np.where(v, da, 0.0)
                dh_prev = (da @ U.T) * (mr[t][None, :] * s_rh)
                dxt[t] += da @ W.T
                gW += xt[t].T @ da
                gU += rec["h_tilde"][t].T @ da
                gb += da.sum(axis=0)
                dh = np.where(v, dh_prev, dh_t)
                dc = np.where(v, dc_prev, dc)
            dW[k], dU[k], db[k] = gW, gU, gb
            dh0[k], dc0[k] = dh, dc
        mn = np.asarray(cache.m_nr[l], dtype=np.float64)
        dout = dxt * (mn[:, None, :] * s_nr)
    return dict(dx=dout, dh0=dh0, dc0=dc0, dW=dW, dU=dU, db=db)


# ----------------------------------------------------------------------------
# Losses used by the workloads (the paper's own losses need the datasets).

def loss_sum(y):
    """L = sum of every element of the top layer's output; dL/dy = 1."""
    return float(np.sum(y)), np.ones_like(np.asarray(y, dtype=np.float64))


def loss_mse(y, target, lengths=None):
    """L = mean over valid (t, b) and features of (y - target)^2."""
    y = np.asarray(y, dtype=np.float64)
    tg = np.asarray(target, dtype=np.float64)
    T, B, F = y.shape
    v = _valid(lengths, T, B)[:, :, None]
    n = float(v.sum()) * F
    diff = np.where(v, y - tg, 0.0)
    return float(np.sum(diff * diff) / n), 2.0 * diff / n


def params_from(W, U, b, num_layers, num_dirs) -> Params:
    f = lambda a: np.asarray(a, dtype=np.float64)
    return Params([f(w) for w in W], [f(u) for u in U], [f(v) for v in b],
                  num_layers, num_dirs)


def train_step(params: Params, x, h0, c0, m_nr, m_rh, p_nr, p_rh, loss, target=None,
               lengths=None):
    """Forward, loss, backward.  Returns (loss value, forward outputs, grads)."""
    y, hT, cT, cache = forward(params, x, h0, c0, m_nr, m_rh, p_nr, p_rh, lengths)
    if loss == "sum":
        lv, dy = loss_sum(y)
    else:
        lv, dy = loss_mse(y, target, lengths)
    grads = backward(cache, dy)
    return lv, dict(y=y, hT=hT, cT=cT, dy=dy), grads
