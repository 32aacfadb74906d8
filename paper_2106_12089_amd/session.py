"""Device-resident state of one LSTM training step driven through the C ABI.

PyTorch only allocates device memory here and supplies the stream; every
computation is a call into liblstm_sd.so.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import binding as B_


class Session:
    """Buffers and calls for one (config, dropout mode) pair.

    wl:      a workload (x, W, U, b, h0, c0, target, lengths as numpy arrays)
    p_nr, p_rh: dropout rates of the two sites; compact: 1 = method, 0 = dense
    """

    def __init__(self, wl, p_nr: float, p_rh: float, compact: int, device: str = "cuda:0",
                 loss: Optional[str] = None):
        cfg = wl.cfg
        self.cfg, self.wl = cfg, wl
        self.device = torch.device(device)
        self.L, self.D, self.H = cfg.num_layers, cfg.num_dirs, cfg.hidden
        self.T, self.B, self.I = wl.x.shape[0], wl.x.shape[1], wl.x.shape[2]
        self.bf16 = cfg.dtype == "bf16"
        self.loss_kind = loss or cfg.loss
        dt = torch.bfloat16 if self.bf16 else torch.float32
        self.dims = B_.make_dims(self.L, self.I, self.H, self.B, self.T, self.D,
                                 B_.DTYPE_BF16 if self.bf16 else B_.DTYPE_F32, compact, p_nr, p_rh)
        dev = self.device
        f = lambda a, t=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(t)
        self.W = [f(w, dt) for w in wl.W]
        self.U = [f(u, dt) for u in wl.U]
        self.b = [f(v) for v in wl.b]
        self.x = f(wl.x, dt)
        self.h0 = f(wl.h0, dt)
        self.c0 = f(wl.c0)
        self.target = f(wl.target)
        self.lengths = None if wl.lengths is None else f(wl.lengths, torch.int32)
        u8 = torch.uint8
        self.mask_buf = torch.zeros(B_.lstm_sd_mask_bytes(self.dims), dtype=u8, device=dev)
        self.reserve = torch.zeros(B_.lstm_sd_reserve_bytes(self.dims), dtype=u8, device=dev)
        self.workspace = torch.zeros(B_.lstm_sd_workspace_bytes(self.dims), dtype=u8, device=dev)
        F = self.D * self.H
        z = lambda *s: torch.zeros(*s, dtype=torch.float32, device=dev)
        self.y = z(self.T, self.B, F)
        self.hT = z(self.L * self.D, self.B, self.H)
        self.cT = z(self.L * self.D, self.B, self.H)
        self.dy = z(self.T, self.B, F)
        self.loss = z(1)
        self.dx = z(self.T, self.B, self.I)
        self.dh0 = z(self.L * self.D, self.B, self.H)
        self.dc0 = z(self.L * self.D, self.B, self.H)
        self.dW = [z(*w.shape) for w in self.W]
        self.dU = [z(*u.shape) for u in self.U]
        self.db = [z(*v.shape) for v in self.b]
        if self.loss_kind == "sum":
            self.dy.fill_(1.0)      # d(sum y)/dy, constant

    # -- calls ---------------------------------------------------------------
    def masks(self, seed: int, step: int, fixed: bool = False):
        """Case-III masks (fresh at every t), or with fixed the Case-IV ones
        (one draw for the whole sequence)."""
        if fixed:
            B_.lstm_sd_mask_generate_fixed(self.dims, seed, step, self.mask_buf)
        else:
            B_.lstm_sd_mask_generate(self.dims, seed, step, self.mask_buf)

    def masks_compact(self):
        B_.lstm_sd_mask_compact(self.dims, self.mask_buf)

    def forward(self):
        B_.lstm_sd_forward(self.dims, self.W, self.U, self.b, self.x, self.lengths, self.h0, self.c0,
                           self.mask_buf, self.y, self.hT, self.cT, self.reserve, self.workspace)

    def loss_grad(self):
        if self.loss_kind == "mse":
            B_.lstm_sd_mse_grad(self.dims, self.y, self.target, self.lengths, self.dy, self.loss,
                                self.workspace)

    def backward(self, dy=None, dhT=None, dcT=None, want_dx=True):
        B_.lstm_sd_backward(self.dims, self.W, self.U, self.b, self.x, self.lengths, self.h0, self.c0,
                            self.mask_buf, self.reserve, self.dy if dy is None else dy, dhT, dcT,
                            self.dx if want_dx else None, self.dh0, self.dc0, self.dW, self.dU, self.db,
                            self.workspace)

    def embedding_backward(self, tokens, vocab: int, d_emb=None):
        """Embedding-table gradient from this step's dx (lstm_sd_embedding_backward):
        accumulated into d_emb [vocab][I] (a new zero tensor when None), returned."""
        if d_emb is None:
            d_emb = torch.zeros(vocab, self.I, dtype=torch.float32, device=self.dx.device)
        B_.lstm_sd_embedding_backward(self.dims, tokens, vocab, self.dx, self.mask_buf, d_emb)
        return d_emb

    def step(self, seed: int, step: int):
        self.masks(seed, step)
        self.forward()
        self.loss_grad()
        self.backward()

    # -- host views (tests) -------------------------------------------------------
    def mask_views(self):
        """Decode the mask buffer: (mask, keep, pos, count, drop, dcount) numpy
        arrays with shapes [sites][T][kmax] or [sites][T]."""
        lay = B_.lstm_sd_mask_layout_get(self.dims)
        raw = self.mask_buf.cpu().numpy()
        S, T, K = lay.sites, lay.seq_len, lay.kmax
        i32 = lambda off, n: raw[off:off + n * 4].view(np.int32)
        mask = raw[lay.mask_off:lay.mask_off + S * T * K].reshape(S, T, K)
        keep = i32(lay.keep_off, S * T * K).reshape(S, T, K)
        pos = i32(lay.pos_off, S * T * K).reshape(S, T, K)
        count = i32(lay.count_off, S * T).reshape(S, T)
        drop = i32(lay.drop_off, S * T * K).reshape(S, T, K)
        dcount = i32(lay.dcount_off, S * T).reshape(S, T)
        self.last_segments = (i32(lay.kseg_off, S * T * 17).reshape(S, T, 17),
                              i32(lay.dseg_off, S * T * 17).reshape(S, T, 17))
        return mask, keep, pos, count, drop, dcount

    def write_masks(self, mask_u8: np.ndarray):
        """Overwrite the mask bytes ([sites][T][kmax]) and rebuild keep lists."""
        lay = B_.lstm_sd_mask_layout_get(self.dims)
        flat = torch.from_numpy(np.ascontiguousarray(mask_u8, dtype=np.uint8).ravel()).to(self.device)
        self.mask_buf[lay.mask_off:lay.mask_off + flat.numel()].copy_(flat)
        self.masks_compact()

    def site_k(self, s):
        return (self.I if s == 0 else self.D * self.H) if s < self.L else self.H

    def outputs(self):
        g = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
        return dict(y=g(self.y), hT=g(self.hT), cT=g(self.cT), dx=g(self.dx), dh0=g(self.dh0),
                    dc0=g(self.dc0), dW=[g(t) for t in self.dW], dU=[g(t) for t in self.dU],
                    db=[g(t) for t in self.db], loss=float(self.loss.item()), dy=g(self.dy))


class HeadSession:
    """Buffers and calls of a language model's output head (pre-FC structured
    output dropout, FC layer, softmax cross-entropy) on the top output of an
    L-layer stack.

    wl:      a workload with W_fc [F][V], b_fc [V] and targets [T][B]
    p_out:   output dropout rate; compact: 1 = method, 0 = dense
    """

    def __init__(self, wl, p_out: float, compact: int, device: str = "cuda:0"):
        cfg = wl.cfg
        self.cfg, self.wl = cfg, wl
        dev = torch.device(device)
        self.T, self.B = wl.x.shape[0], wl.x.shape[1]
        self.F, self.V = wl.W_fc.shape
        bf16 = cfg.dtype == "bf16"
        dt = torch.bfloat16 if bf16 else torch.float32
        self.hd = B_.make_head_dims(self.F, self.V, self.B, self.T, B_.DTYPE_BF16 if bf16 else B_.DTYPE_F32,
                                    compact, 4 * cfg.num_layers, p_out)
        f = lambda a, t=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(t)
        self.W_fc = f(wl.W_fc, dt)
        self.b_fc = f(wl.b_fc)
        self.targets = f(wl.targets, torch.int32)
        self.lengths = None if wl.lengths is None else f(wl.lengths, torch.int32)
        u8 = torch.uint8
        self.mask_buf = torch.zeros(B_.lstm_sd_head_mask_bytes(self.hd), dtype=u8, device=dev)
        self.workspace = torch.zeros(B_.lstm_sd_head_workspace_bytes(self.hd), dtype=u8, device=dev)
        z = lambda *s: torch.zeros(*s, dtype=torch.float32, device=dev)
        self.logits = z(self.T, self.B, self.V)
        self.loss = z(1)
        self.dy = z(self.T, self.B, self.F)
        self.dW = z(self.F, self.V)
        self.db = z(self.V)

    def masks(self, seed: int, step: int):
        B_.lstm_sd_head_mask_generate(self.hd, seed, step, self.mask_buf)

    def forward(self, y):
        B_.lstm_sd_head_forward(self.hd, self.W_fc, self.b_fc, y, self.mask_buf, self.logits, self.workspace)

    def backward(self):
        B_.lstm_sd_head_backward(self.hd, self.W_fc, self.targets, self.lengths, self.mask_buf, self.logits,
                                 self.loss, self.dy, self.dW, self.db, self.workspace)

    def mask_view(self):
        """The output mask bytes [T][F] (1 = kept)."""
        lay = B_.lstm_sd_head_mask_layout_get(self.hd)
        raw = self.mask_buf.cpu().numpy()
        return raw[lay.mask_off:lay.mask_off + self.T * self.F].reshape(self.T, self.F)

    def outputs(self):
        g = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
        return dict(z=g(self.logits), loss=float(self.loss.item()), dy=g(self.dy), dW=g(self.dW),
                    dc=g(self.db))


class Case1Session:
    """The Case-I ("NR+Random") comparator: per-element dropout on every
    layer's input (lstm_sd_case1_dropout), each layer a single-layer step
    without dropout (identity keep lists, every row multiplied), the input
    gradients taken back through the same masks.

    wl: a workload; p: the input dropout rate of every layer."""

    def __init__(self, wl, p: float, device: str = "cuda:0"):
        import dataclasses
        import types
        cfg = wl.cfg
        self.cfg, self.wl, self.p = cfg, wl, p
        self.L, self.D, self.H = cfg.num_layers, cfg.num_dirs, cfg.hidden
        self.T, self.B = wl.x.shape[0], wl.x.shape[1]
        self.bf16 = cfg.dtype == "bf16"
        self.layers = []
        for l in range(self.L):
            kin = cfg.k_in(l)
            lcfg = dataclasses.replace(cfg, num_layers=1, input_dim=kin)
            sl = slice(l * self.D, (l + 1) * self.D)
            lwl = types.SimpleNamespace(cfg=lcfg, x=wl.x if l == 0 else np.zeros((self.T, self.B, kin), np.float32),
                                        W=wl.W[sl], U=wl.U[sl], b=wl.b[sl], h0=wl.h0[sl], c0=wl.c0[sl],
                                        target=wl.target, lengths=wl.lengths)
            s = Session(lwl, 0.0, 0.0, 1, device)
            s.masks(0, 0)                      # p = 0: identity keep lists, the same at every step
            self.layers.append(s)
        self.x0 = self.layers[0].x.clone()
        dev = self.layers[0].x.device
        self.drop_masks = [torch.zeros(self.T, self.B, cfg.k_in(l), dtype=torch.uint8, device=dev)
                           for l in range(self.L)]
        self.dx = torch.zeros(self.T, self.B, cfg.input_dim, dtype=torch.float32, device=dev)
        self.y = self.layers[-1].y

    def step(self, seed: int, step: int):
        dt = B_.DTYPE_BF16 if self.bf16 else B_.DTYPE_F32
        for l, s in enumerate(self.layers):
            src, sdt = (self.x0, dt) if l == 0 else (self.layers[l - 1].y, B_.DTYPE_F32)
            B_.lstm_sd_case1_dropout(self.T, self.B, s.I, sdt, src, dt, s.x, self.drop_masks[l], seed, step, 4 * l,
                                     self.p)
            s.forward()
        self.layers[-1].loss_grad()
        for l in reversed(range(self.L)):
            s = self.layers[l]
            s.backward(dy=None if l == self.L - 1 else self.layers[l].dy)
            out = self.dx if l == 0 else self.layers[l - 1].dy
            B_.lstm_sd_case1_dropout_backward(self.T, self.B, s.I, s.dx, self.drop_masks[l], self.p, out)

    def outputs(self):
        g = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
        top = self.layers[-1]
        return dict(y=g(top.y), loss=float(top.loss.item()), dx=g(self.dx),
                    dW=[g(t) for s in self.layers for t in s.dW], dU=[g(t) for s in self.layers for t in s.dU],
                    db=[g(t) for s in self.layers for t in s.db])
