"""Seeded synthetic workloads shaped like the paper's LSTM experiments.

This module is the only code shared by the oracle side (tests) and the HIP
side (tests, bench, smoke).  It draws inputs, weights, initial states,
targets and sequence lengths from a seeded generator and holds none of the
method's arithmetic: no LSTM cell, no dropout mask, no gradient.  Dropout
masks are not drawn here; each side derives them from (seed, step) with its
own implementation of the same counter-based generator.

Shapes follow the paper's workloads (Sec. 4.1 Zaremba medium/large,
Sec. 4.2 Luong encoder, Sec. 4.3 BiLSTM tagger) plus a large stress shape.
The real datasets (PTB, IWSLT, CoNLL) are not used: token ids are drawn from
a truncated Zipf(1.1) law over the stated vocabulary and looked up in a
random embedding table.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = ["Config", "CONFIGS", "MODES", "Workload", "make_workload",
           "round_to_bf16", "get_config"]


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    num_layers: int
    num_dirs: int
    input_dim: int
    hidden: int
    batch: int
    seq_len: int
    p_values: tuple          # structured dropout rates the config is run at
    dtype: str               # "f32" or "bf16": storage type of x, W, U, h0
    loss: str                # "sum" (sum of top-layer y) or "mse"
    seed: int
    # input recipe
    input_kind: str          # "normal" or "embedding"
    input_std: float = 0.1
    vocab: int = 0
    weight_init: str = "normal"   # "normal" (N(0, weight_scale)) or "uniform" (U(+-weight_scale))
    weight_scale: float = 0.1
    min_len: Optional[int] = None  # if set, lengths ~ U{min_len..seq_len}
    input_init: str = "normal"     # embedding table: "normal" N(0, input_std) or "uniform" U(+-input_std)
    # a rate per layer (the dropout vector of a model with one rate per
    # site): NR of layer l's input, RH of layer l; None = p for every layer
    p_nr_layers: Optional[tuple] = None
    p_rh_layers: Optional[tuple] = None
    p_out: Optional[float] = None  # rate of the output (pre-FC) site, if the model fixes one

    @property
    def mask_seed(self) -> int:
        return 1000 + self.seed

    def k_in(self, layer: int) -> int:
        return self.input_dim if layer == 0 else self.num_dirs * self.hidden


def _cfgs():
    cs = [
        Config("tiny", 2, 1, 32, 64, 4, 8, (0.5,), "f32", "sum", 1,
               "normal", 0.1, 0, "normal", 0.1),
        Config("lm_medium", 2, 1, 650, 650, 20, 35, (0.5,), "bf16", "mse", 2,
               "embedding", 0.05, 10000, "uniform", 0.05),
        Config("lm_large", 2, 1, 1500, 1500, 20, 35, (0.65,), "bf16", "mse", 3,
               "embedding", 0.04, 10000, "uniform", 0.04),
        Config("seq2seq_enc", 2, 1, 500, 500, 64, 50, (0.3,), "bf16", "mse", 4,
               "embedding", 0.1, 20000, "uniform", 1.0 / np.sqrt(500), min_len=20),
        Config("tagger", 1, 2, 300, 256, 32, 40, (0.3, 0.5, 0.7), "bf16", "mse", 5,
               "normal", 1.0, 0, "uniform", 1.0 / np.sqrt(256)),
        Config("stress", 2, 1, 1024, 1024, 256, 64, (0.3, 0.5, 0.7), "bf16", "mse", 6,
               "normal", 1.0, 0, "uniform", 1.0 / np.sqrt(1024)),
        # AWD-LSTM shape (Sec. 4.1): 3 layers, embedding 400, every hidden
        # layer 1150, LSTM weights U(+-1/sqrt(H)), embeddings U(+-0.1); input
        # dropout 0.4 on layer 0, 0.25 between layers, 0.4 before the FC
        # layer, and 0.5 on the recurrent weights, which structured becomes
        # RH dropout on h_{t-1}.  Batch 20 and 70 steps per sequence are the
        # usual PTB settings of that model (the paper does not restate them).
        Config("awd_lstm", 3, 1, 400, 1150, 20, 70, (0.4,), "bf16", "mse", 7,
               "embedding", 0.1, 10000, "uniform", 1.0 / np.sqrt(1150), input_init="uniform",
               p_nr_layers=(0.4, 0.25, 0.25), p_rh_layers=(0.5, 0.5, 0.5), p_out=0.4),
    ]
    return {c.name: c for c in cs}


CONFIGS = _cfgs()

# Dropout modes: which sites carry structured dropout, and whether the
# kernels skip dropped rows ("compact") or run the same kernels over every
# row with the mask applied as a multiplier ("dense").
MODES = {
    "nr": dict(rh=False, compact=True),        # NR+ST
    "nrrh": dict(rh=True, compact=True),       # NR+RH+ST
    "nr_dense": dict(rh=False, compact=False),
    "nrrh_dense": dict(rh=True, compact=False),
}


def get_config(name: str) -> Config:
    return CONFIGS[name]


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned
    as float32.  Input quantisation only: both sides consume these values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out).astype(np.float32)


@dataclasses.dataclass
class Workload:
    cfg: Config
    x: np.ndarray            # [T][B][I] float32 (bf16-representable for bf16 configs)
    W: list                  # per (l, d): [K_in][4H]
    U: list                  # per (l, d): [H][4H]
    b: list                  # per (l, d): [4H] float32
    h0: np.ndarray           # [L*D][B][H]
    c0: np.ndarray           # [L*D][B][H] float32
    target: np.ndarray       # [T][B][D*H] float32 (MSE target)
    lengths: Optional[np.ndarray]  # [B] int32 or None
    tokens: Optional[np.ndarray] = None   # [T][B] int32 token ids of an embedding input, or None
    # output head of a language model (embedding inputs only): the next token
    # as target, an FC layer [D*H][V] (input-major) and its bias [V]
    targets: Optional[np.ndarray] = None  # [T][B] int32
    W_fc: Optional[np.ndarray] = None     # [D*H][V] float32 (bf16-representable for bf16 configs)
    b_fc: Optional[np.ndarray] = None     # [V] float32

    @property
    def batch(self):
        return self.x.shape[1]


def _zipf_ids(rng, vocab, shape, s=1.1):
    r = np.arange(1, vocab + 1, dtype=np.float64)
    pr = r ** (-s)
    pr /= pr.sum()
    return rng.choice(vocab, size=shape, p=pr)


def make_workload(cfg: Config, batch: Optional[int] = None) -> Workload:
    """Draw the seeded inputs of one config.  `batch` overrides the batch size
    (rows are drawn in the same order, so a smaller batch is a prefix of the
    full one only for the per-row arrays drawn last; callers that need
    row subsets slice a full workload instead)."""
    B = cfg.batch if batch is None else batch
    T, L, D, I, H = cfg.seq_len, cfg.num_layers, cfg.num_dirs, cfg.input_dim, cfg.hidden
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    bf = cfg.dtype == "bf16"
    q = round_to_bf16 if bf else (lambda a: np.asarray(a, dtype=np.float32))

    # layer input
    ids = None
    if cfg.input_kind == "embedding":
        if cfg.input_init == "uniform":
            table = rng.uniform(-cfg.input_std, cfg.input_std, size=(cfg.vocab, I)).astype(np.float32)
        else:
            table = rng.normal(0.0, cfg.input_std, size=(cfg.vocab, I)).astype(np.float32)
        ids = _zipf_ids(rng, cfg.vocab, (T, B))
        x = table[ids]
    else:
        x = rng.normal(0.0, cfg.input_std, size=(T, B, I)).astype(np.float32)

    W, U, bias = [], [], []
    for l in range(L):
        kin = cfg.k_in(l)
        for _d in range(D):
            if cfg.weight_init == "uniform":
                a = cfg.weight_scale
                w = rng.uniform(-a, a, size=(kin, 4 * H))
                u = rng.uniform(-a, a, size=(H, 4 * H))
                bb = rng.uniform(-a, a, size=(4 * H,))
            else:
                s = cfg.weight_scale
                w = rng.normal(0.0, s, size=(kin, 4 * H))
                u = rng.normal(0.0, s, size=(H, 4 * H))
                bb = rng.normal(0.0, s, size=(4 * H,))
            W.append(q(w.astype(np.float32)))
            U.append(q(u.astype(np.float32)))
            bias.append(bb.astype(np.float32))
    h0 = q(rng.normal(0.0, 0.1, size=(L * D, B, H)).astype(np.float32))
    c0 = rng.normal(0.0, 0.1, size=(L * D, B, H)).astype(np.float32)
    target = rng.normal(0.0, 1.0, size=(T, B, D * H)).astype(np.float32)
    lengths = None
    if cfg.min_len is not None:
        lengths = rng.integers(cfg.min_len, T + 1, size=(B,)).astype(np.int32)
        # padded positions carry zero input
        valid = np.arange(T)[:, None] < lengths[None, :]
        x = np.where(valid[:, :, None], x, 0.0).astype(np.float32)
    x = q(x)
    tokens = None if ids is None else np.ascontiguousarray(ids.astype(np.int32))
    targets = W_fc = b_fc = None
    if ids is not None:
        # drawn from a generator of their own, so the draws above do not move
        hr = np.random.Generator(np.random.PCG64([cfg.seed, 1]))
        nxt = _zipf_ids(hr, cfg.vocab, (1, B))
        targets = np.ascontiguousarray(np.concatenate([ids[1:], nxt]).astype(np.int32))
        a = cfg.weight_scale
        W_fc = q(hr.uniform(-a, a, size=(D * H, cfg.vocab)).astype(np.float32))
        b_fc = hr.uniform(-a, a, size=(cfg.vocab,)).astype(np.float32)
    return Workload(cfg, np.ascontiguousarray(x), W, U, bias, h0, c0, target, lengths, tokens, targets,
                    W_fc, b_fc)


def slice_rows(wl: Workload, rows) -> Workload:
    """The same workload restricted to a subset of batch rows (weights and
    every per-row array sliced consistently)."""
    rows = np.asarray(rows)
    return Workload(wl.cfg, np.ascontiguousarray(wl.x[:, rows]), wl.W, wl.U, wl.b,
                    np.ascontiguousarray(wl.h0[:, rows]), np.ascontiguousarray(wl.c0[:, rows]),
                    np.ascontiguousarray(wl.target[:, rows]),
                    None if wl.lengths is None else np.ascontiguousarray(wl.lengths[rows]),
                    None if wl.tokens is None else np.ascontiguousarray(wl.tokens[:, rows]),
                    None if wl.targets is None else np.ascontiguousarray(wl.targets[:, rows]),
                    wl.W_fc, wl.b_fc)
