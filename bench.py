"""Benchmark of one structured-dropout LSTM training step on one MI355X.

A step is one pass of the whole path over one batch of synthetic input that
is already resident in HBM: draw the Case-III masks and build the keep lists
(fresh masks every step), forward unroll, MSE loss gradient, BPTT with the
weight gradients.  The headline workload is the 2-layer, 650-unit
language-model shape (batch 20, 35 steps, bf16 storage with fp32
accumulation, structured dropout p = 0.5 on the non-recurrent inputs).
Every other workload (LM-large, the Luong encoder, the BiLSTM tagger, the
2-layer 1024-unit batch-256 stress shape, the AWD-LSTM shape) is measured in
the same run under "configs".  Prints one JSON line.

  value      effective TFLOP/s: algorithmic FLOPs of the step (products over
             the rows actually kept, three products per gate GEMM) / step time
  speedup    the same kernels run dense (compact = 0) / the method
  phases     per-step time of each kernel class (FP-x input product, FP-rec
             recurrence, BP-rec recurrence backward, BP-dx input gradient,
             WG weight gradients, mask draw), from HIP events around every
             launch of that class on its launch stream, in a separate pass
  roofline   the kernel class with the largest share of the step.  The
             recurrent classes at batch <= 64 are priced on the bytes of the
             kept rows of U they stream every time step (K'_h * 4H * element
             size per (layer, direction, t)) against HBM; every other class on
             its algorithmic MFMA FLOPs against the dense matrix peak of its
             data type
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "lm_medium"
METRIC = "LSTM fwd+BPTT step time & eff. TFLOP/s; speedup vs dense at p=0.5"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
KERNELS = ("mask_build", "transpose", "fx", "fwd_persist", "step", "bwd_persist", "bwd", "dx", "wgrad")
GEMM_KERNELS = ("fx", "fwd_persist", "step", "bwd_persist", "bwd", "dx", "wgrad")
RECURRENT = ("fwd_persist", "step", "bwd_persist", "bwd")
# kernel classes of each phase of the step (the paper's FP / BP / WG split)
PHASES = {"mask": ("mask_build",), "fp_x": ("fx",), "fp_rec": ("fwd_persist", "step"),
          "bp_rec": ("bwd_persist", "bwd"), "bp_dx": ("dx",), "wg": ("wgrad",), "other": ("transpose",)}
CONFIG_RUNS = ("lm_large", "seq2seq_enc", "tagger", "stress", "awd_lstm")
KERNEL_SRC_DIR = os.path.join(ROOT, "paper_2106_12089_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_src_hash():
    """Hash of every HIP source and header the kernels are built from."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(KERNEL_SRC_DIR)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(KERNEL_SRC_DIR, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# Work accounting from the kept counts (counts: [sites][T]; sites = NR of
# each layer, then RH of each (layer, direction)).

def algorithmic_flops(counts, cfg, lengths=None):
    """Sum over layers, directions and t of 3 * 2 * B_t * 4H * (n_x + n_h):
    the forward product, the input-gradient product and the weight-gradient
    product of every gate GEMM, over kept rows only (B_t = valid rows)."""
    L, D, H, T, B = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.batch
    bt = np.full(T, B) if lengths is None else \
        (np.arange(T)[:, None] < np.asarray(lengths)[None, :]).sum(1)
    tot = 0.0
    for l in range(L):
        for d in range(D):
            nx, nh = np.asarray(counts[l]), np.asarray(counts[L + l * D + d])
            tot += float(np.sum(3 * 2 * bt * 4 * H * (nx + nh)))
    return tot


def dense_counts(cfg):
    L, D, H, T, I = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.input_dim
    return [np.full(T, I if l == 0 else D * H) for l in range(L)] + [np.full(T, H)] * (L * D)


def kernel_work(kind, counts, cfg, stacked=False):
    """(flops, bytes, launches) of one step for a kernel class; bytes are the
    algorithmic minimum: every operand read once and every output written
    once per launch (kept rows only).  stacked: the unidirectional stack ran
    as one persistent launch per pass, whose slots also form the input
    product of every layer above the first (forward) and the input gradient
    of every layer below the top (backward); the separate passes then cover
    layer 0 only."""
    L, D, H, T, B = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.batch
    G = 4 * H
    e = 2 if cfg.dtype == "bf16" else 4
    fl = by = 0.0
    upper = range(1, L) if stacked else range(0)     # layers whose input product / gradient moved
    if kind == "step":                      # one launch per (layer, step), directions fused
        for l in range(L):
            for d in range(D):
                nh = np.asarray(counts[L + l * D + d], dtype=np.float64)
                fl += float(np.sum(2 * B * G * nh))
                by += float(np.sum(nh * G * e + B * nh * e))           # kept U rows, kept h columns
                by += T * B * (G * 4 + H * 8 + G * 4 + H * 4 + 2 * H * e + H * 8)
                by += T * B * H * (4 if l == L - 1 else 4 * e)
        return fl, by, L * T
    if kind == "fwd_persist":               # one launch per layer runs every step (both directions)
        for l in range(L):
            for d in range(D):
                nh = np.asarray(counts[L + l * D + d], dtype=np.float64)
                fl += float(np.sum(2 * B * G * nh))
                by += H * G * e                                        # U slice, read once per launch
                by += T * B * (G * 4 + G * 4 + H * 4 + 2 * H * e)      # gx, gates, c, h^T + exchange
                by += T * B * H * (4 if l == L - 1 else 2 * e) + B * H * 16
        for l in upper:                     # input product: W slice, x~ exchange, gx written and read
            n = np.asarray(counts[l], dtype=np.float64)
            fl += float(np.sum(2 * B * G * n))
            by += cfg.k_in(l) * G * e + float(np.sum(B * n * e)) + T * B * G * 8
        return fl, by, 1 if stacked else L
    if kind == "bwd_persist":               # one launch per layer runs every BPTT step (both directions)
        for l in range(L):
            for d in range(D):
                nh = np.asarray(counts[L + l * D + d], dtype=np.float64)
                fl += float(np.sum(2 * B * G * nh))
                by += H * G * e                                        # U rows, read once per launch
                by += T * B * G * e                                    # DA of each step, read once
                by += T * B * H * (16 + 4 + 4 + 4 + 8 * e)             # gates, c, c_prev, dy; DA + DA^T
                by += B * H * 16
        for l in upper:                     # input gradient of layer l: W rows, kept columns written and read
            n = np.asarray(counts[l], dtype=np.float64)
            fl += float(np.sum(2 * B * G * n))
            by += cfg.k_in(l) * G * e + float(np.sum(B * n * 8))
        return fl, by, 1 if stacked else L
    if kind == "bwd":                       # T pointwise steps + one final pass per layer
        for l in range(L):
            for d in range(D):
                nh = np.asarray(counts[L + l * D + d], dtype=np.float64)
                fl += float(np.sum(2 * B * G * nh))
                by += float(np.sum(nh * G * e + B * G * e))            # kept U rows, DA of that step
                by += T * B * H * (16 + 4 + 4 + 8 + 8 + 4 + 8 * e)
        return fl, by, L * (T + 1)
    if kind == "wgrad":                     # dW and dU of every (layer, direction)
        for l in range(L):
            kin = cfg.input_dim if l == 0 else D * H
            for d in range(D):
                for n, K in ((np.asarray(counts[l], np.float64), kin),
                             (np.asarray(counts[L + l * D + d], np.float64), H)):
                    fl += float(np.sum(2 * n * B * G))
                    by += float(np.sum(n * B * e + G * B * e)) + K * G * 4
        return fl, by, 2 * L * D
    if kind == "fx":
        for l in range(1 if stacked else L):
            kin = cfg.input_dim if l == 0 else D * H
            n = np.asarray(counts[l], np.float64)
            for d in range(D):
                fl += float(np.sum(2 * B * G * n))
                by += kin * G * e + float(np.sum(B * n * e)) + T * B * G * 4
        return fl, by, (1 if stacked else L) * D
    if kind == "dx":
        for l in range(1 if stacked else L):
            kin = cfg.input_dim if l == 0 else D * H
            n = np.asarray(counts[l], np.float64)
            fl += float(np.sum(2 * B * G * n)) * D
            by += D * (kin * G * e + T * B * G * e) + float(np.sum(B * n * 4))
        return fl, by, 1 if stacked else L
    raise ValueError(kind)


# ---------------------------------------------------------------------------

def run_mode(wl, p_nr, p_rh, compact, steps, warmup, timed_kernels=(), fixed=False, kernel_steps=None):
    import torch
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    cfg = wl.cfg
    s = Session(wl, p_nr, p_rh, compact)
    for i in range(warmup):
        s.step(cfg.mask_seed, 10_000 + i)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    if fixed:                                  # Case-IV: one mask draw for the whole sequence
        s.masks = lambda seed, step, _m=s.masks: _m(seed, step, fixed=True)
    # the timed pass: K whole steps between two events, nothing else recorded
    e_start, e_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e_start.record()
    for i in range(steps):
        s.step(cfg.mask_seed, i)
    e_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = e_start.elapsed_time(e_end)
    # a second pass with an event between the phases, for the breakdown only
    for i in range(steps):
        e = ev[i]
        e[0].record()
        s.masks(cfg.mask_seed, i)
        e[1].record()
        s.forward()
        e[2].record()
        s.loss_grad()
        e[3].record()
        s.backward()
        e[4].record()
    torch.cuda.synchronize()
    phases = np.zeros(4)
    for e in ev:
        for k in range(4):
            phases[k] += e[k].elapsed_time(e[k + 1])
    phases /= steps
    per_step = np.array([e[0].elapsed_time(e[4]) for e in ev])   # the instrumented pass, per step
    # kept counts of every timed step (masks regenerated outside the timed region)
    counts_all = []
    for i in range(steps):
        s.masks(cfg.mask_seed, i)
        counts_all.append(s.mask_views()[3].astype(np.float64))
    counts = np.mean(counts_all, axis=0)
    # per-kernel timing: a second timed pass per kernel class, events on the launch stream
    ktime = {}
    ks = steps if kernel_steps is None else kernel_steps
    for kname in timed_kernels:
        B_.lstm_sd_kernel_timer_start(kname)
        for i in range(ks):
            s.step(cfg.mask_seed, i)
        ms, n = B_.lstm_sd_kernel_timer_stop()
        torch.cuda.synchronize()
        ktime[kname] = dict(total_ms=ms / ks, launches=n / ks, avg_us=1e3 * ms / max(n, 1))
    return dict(ms=total_ms / steps, wall_ms=wall * 1e3 / steps, counts=counts,
                flops=float(np.mean([algorithmic_flops(c, cfg, wl.lengths) for c in counts_all])),
                phases=dict(mask=phases[0], forward=phases[1], loss=phases[2], backward=phases[3]),
                ktime=ktime, pct=[float(np.percentile(per_step, q)) for q in (10, 50, 90)])


def run_case1(wl, p, steps, warmup):
    """The Case-I ("NR+Random") comparator's whole step (per-element input
    dropout on every layer, each layer dense), timed with events."""
    import torch
    from paper_2106_12089_amd.session import Case1Session
    cfg = wl.cfg
    c = Case1Session(wl, p)
    for i in range(warmup):
        c.step(cfg.mask_seed, 10_000 + i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        c.step(cfg.mask_seed, i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def run_embedding(wl, p_nr, steps, warmup):
    """Embedding-table gradient after the step (lstm_sd_embedding_backward) on
    a language-model workload: its kernel's average duration (HIP events on
    its launch stream) and algorithmic bytes per launch (token ids, the kept
    columns of dx, one read and one write of each touched row of d_emb)."""
    import torch
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    cfg = wl.cfg
    s = Session(wl, p_nr, 0.0, 1)
    tok = torch.from_numpy(wl.tokens.astype(np.int32)).cuda()
    d_emb = torch.zeros(cfg.vocab, s.I, dtype=torch.float32, device="cuda")
    for i in range(warmup):
        s.step(cfg.mask_seed, 10_000 + i)
        s.embedding_backward(tok, cfg.vocab, d_emb)
    torch.cuda.synchronize()
    B_.lstm_sd_kernel_timer_start("emb_grad")
    nbytes = []
    rows = len(np.unique(wl.tokens))
    for i in range(steps):
        s.step(cfg.mask_seed, i)
        s.embedding_backward(tok, cfg.vocab, d_emb)
        kept = s.mask_views()[3][0].astype(np.int64)      # layer-0 NR kept count per step t
        nbytes.append(wl.tokens.size * 4 + int(kept.sum()) * s.B * 4 + rows * s.I * 8)
    ms, n = B_.lstm_sd_kernel_timer_stop()
    torch.cuda.synchronize()
    us = 1e3 * ms / max(n, 1)
    b = float(np.mean(nbytes))
    a = b / (us * 1e-6) / 1e9
    return {"avg_us": round(us, 3), "launches_per_step": n / steps, "vocab": cfg.vocab, "rows_touched": rows,
            "roofline": {"bound": "hbm", "achieved": round(a, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(a / PEAK_HBM_GBS, 5), "kernel": "emb_grad",
                         "algorithmic_bytes_per_launch": int(b), "traffic": None}}


def run_head(wl, p, steps, warmup, compact):
    """The output head (pre-FC structured dropout, FC layer, softmax
    cross-entropy) alone, and the whole LM step with it (LSTM forward, head,
    LSTM backward fed by the head's dy), timed with events on the stream;
    FC FLOPs counted over the kept input columns (forward, dX and dW
    products: 3 * 2 * B * V per kept (t, column))."""
    import torch
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import HeadSession, Session
    cfg = wl.cfg
    h = HeadSession(wl, p, compact)
    s = Session(wl, p, 0.0, compact)
    s.masks(cfg.mask_seed, 0)
    s.forward()
    torch.cuda.synchronize()

    def head_step(i):
        h.masks(cfg.mask_seed, i)
        h.forward(s.y)
        h.backward()

    def lm_step(i):
        s.masks(cfg.mask_seed, i)
        h.masks(cfg.mask_seed, i)
        s.forward()
        h.forward(s.y)
        h.backward()
        s.backward(dy=h.dy)

    out = {}
    for name, fn in (("head", head_step), ("lm_step", lm_step)):
        for i in range(warmup):
            fn(10_000 + i)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        out[name] = e0.elapsed_time(e1) / steps
    kept = []
    for i in range(steps):
        h.masks(cfg.mask_seed, i)
        kept.append(int(h.mask_view().sum()) if compact else h.T * h.F)
    out["flops"] = 6.0 * h.B * h.V * float(np.mean(kept))
    ktime = {}
    for kname in ("fx", "dx", "wgrad", "ce"):
        B_.lstm_sd_kernel_timer_start(kname)
        for i in range(steps):
            head_step(i)
        ms, n = B_.lstm_sd_kernel_timer_stop()
        torch.cuda.synchronize()
        ktime[kname] = round(1e3 * ms / steps, 2)
    out["kernels_us_per_step"] = ktime
    # algorithmic work per launch (each operand once, each result once)
    es = 2 if cfg.dtype == "bf16" else 4
    T, B, F, V = h.T, h.B, h.F, h.V
    kf = out["flops"] / 3.0                    # one FC product over the kept columns
    out["work"] = {
        "fx": dict(bytes=T * B * F * es + F * V * es + V * 4 + T * B * V * 4, flops=kf),
        "dx": dict(bytes=T * B * V * es + F * V * es + T * B * F * 4, flops=kf),
        "wgrad": dict(bytes=T * F * B * es + T * V * B * es + F * V * 4 + V * 4, flops=kf),
        "ce": dict(bytes=T * B * V * 4 + 2 * T * B * V * es + T * B * 4, flops=0.0),
    }
    return out


def head_roofline(hc, cfg):
    """Roofline of the head's dominant kernel (by time): HBM-bound when its
    arithmetic intensity is below the ridge point, else MFMA-bound."""
    k = max(hc["kernels_us_per_step"], key=hc["kernels_us_per_step"].get)
    us = hc["kernels_us_per_step"][k]
    w = hc["work"][k]
    peak_f = PEAK_TFLOPS["bf16" if cfg.dtype == "bf16" else "f32"]
    ridge = peak_f * 1e12 / (PEAK_HBM_GBS * 1e9)
    if w["flops"] / w["bytes"] >= ridge:
        a = w["flops"] / (us * 1e-6) / 1e12
        r = dict(bound="mfma", achieved=round(a, 3), peak=peak_f, unit="TFLOP/s", frac=round(a / peak_f, 5))
    else:
        a = w["bytes"] / (us * 1e-6) / 1e9
        r = dict(bound="hbm", achieved=round(a, 1), peak=PEAK_HBM_GBS, unit="GB/s", frac=round(a / PEAK_HBM_GBS, 5))
    r.update(kernel=k, launch_us=us, algorithmic_bytes_per_launch=int(w["bytes"]),
             algorithmic_flops_per_launch=w["flops"], traffic=None)
    return r


def head_cpu_baseline(wl, p):
    """The head's float64 oracle (forward, loss, backward) timed once on the
    host on the same workload."""
    from oracle import head, masks
    cfg = wl.cfg
    y = np.random.default_rng(0).normal(0.0, 0.5, size=(cfg.seq_len, cfg.batch, wl.W_fc.shape[0]))
    m = masks.keep_mask(cfg.mask_seed, 0, masks.out_stream(cfg.num_layers), cfg.seq_len, wl.W_fc.shape[0], p)
    t0 = time.perf_counter()
    head.head_step(y, wl.W_fc, wl.b_fc, m, p, wl.targets, wl.lengths)
    return dict(ms_per_step=round((time.perf_counter() - t0) * 1e3, 1), kind="oracle",
                sample="one head step (forward, loss, backward) of the same workload, float64 NumPy")


def embedding_cpu_baseline(wl, p):
    from oracle import embedding, masks
    cfg = wl.cfg
    dx = np.random.default_rng(0).normal(size=(cfg.seq_len, cfg.batch, cfg.input_dim))
    m = masks.keep_mask(cfg.mask_seed, 0, masks.nr_stream(0), cfg.seq_len, cfg.input_dim, p)
    t0 = time.perf_counter()
    embedding.embedding_grad(wl.tokens, dx, m, np.zeros((cfg.vocab, cfg.input_dim)))
    return dict(ms_per_step=round((time.perf_counter() - t0) * 1e3, 2), kind="oracle",
                sample="one embedding-gradient call of the same workload, float64 NumPy loop")


def recurrent_u_bytes(counts, cfg):
    """Bytes of U a recurrence streams per step of work: the kept rows
    U[K'_h, :] of every (layer, direction, t), K'_h * 4H * element size."""
    L, D, H = cfg.num_layers, cfg.num_dirs, cfg.hidden
    e = 2 if cfg.dtype == "bf16" else 4
    return float(sum(np.sum(np.asarray(counts[L + l * D + d], np.float64)) * 4 * H * e
                     for l in range(L) for d in range(D)))


def is_stacked(res, cfg):
    """One persistent launch per pass over a unidirectional stack."""
    kt = res["ktime"]
    return cfg.num_layers > 1 and all(kt.get(k, {}).get("launches", 0) == 1 for k in ("fwd_persist", "bwd_persist"))


def kernel_table(res, cfg):
    """Per kernel class: time per step, launches, algorithmic FLOPs and the
    MFMA fraction (FLOPs / summed launch time / dense peak of the data type);
    for the recurrences also the U-row bytes per launch and their HBM
    fraction."""
    kt = res["ktime"]
    stacked = is_stacked(res, cfg)
    peak_f = PEAK_TFLOPS["bf16" if cfg.dtype == "bf16" else "f32"]
    out = {}
    for k, v in kt.items():
        if v["total_ms"] <= 0:
            continue
        ent = {"ms_per_step": round(v["total_ms"], 4), "launches_per_step": v["launches"],
               "avg_us": round(v["avg_us"], 3)}
        if k in GEMM_KERNELS:
            fl, by, _ = kernel_work(k, res["counts"], cfg, stacked)
            tf = fl / (v["total_ms"] * 1e-3) / 1e12
            ent.update(gflop_per_step=round(fl / 1e9, 4), tflops=round(tf, 3), mfma_frac=round(tf / peak_f, 5),
                       min_bytes_per_launch=int(by / max(v["launches"], 1)))
            if k in RECURRENT:
                ub = recurrent_u_bytes(res["counts"], cfg) / max(v["launches"], 1)
                gbs = ub / (v["avg_us"] * 1e-6) / 1e9
                ent.update(u_bytes_per_launch=int(ub), u_gbs=round(gbs, 1), hbm_frac=round(gbs / PEAK_HBM_GBS, 5))
        out[k] = ent
    return out


def phase_times(res):
    """Per-step ms of each phase (sum of its kernel classes)."""
    kt = res["ktime"]
    return {ph: round(sum(kt.get(k, {}).get("total_ms", 0.0) for k in ks), 4) for ph, ks in PHASES.items()}


def roofline(res, cfg):
    """Roofline of the dominant kernel class (largest time per step)."""
    kt = res["ktime"]
    cand = [k for k in GEMM_KERNELS if kt.get(k, {}).get("total_ms", 0) > 0]
    name = max(cand, key=lambda k: kt[k]["total_ms"])
    stacked = is_stacked(res, cfg)
    fl, by, _ = kernel_work(name, res["counts"], cfg, stacked)
    launches = kt[name]["launches"]
    fl_l, by_l = fl / launches, by / launches
    dur = kt[name]["avg_us"] * 1e-6
    peak_f = PEAK_TFLOPS["bf16" if cfg.dtype == "bf16" else "f32"]
    traffic = None
    try:
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        ent = tr.get(name)
        if ent and ent.get("src_hash") == kernel_src_hash() and ent.get("workload") == cfg.name:
            traffic = ent["bytes_per_launch"]
    except (OSError, ValueError):
        pass
    if name in RECURRENT and cfg.batch <= 64:
        ub = recurrent_u_bytes(res["counts"], cfg) / launches
        out = dict(bound="hbm", achieved=ub / dur / 1e9, peak=PEAK_HBM_GBS, unit="GB/s",
                   formula="sum over (layer, direction, t) of K'_h * 4H * element bytes, per launch / launch time")
        out["algorithmic_bytes_per_launch"] = ub
    else:
        out = dict(bound="mfma", achieved=fl_l / dur / 1e12, peak=peak_f, unit="TFLOP/s",
                   formula="algorithmic FLOPs (2 * B * 4H * K' per product over kept rows) per launch / launch time")
        out["algorithmic_bytes_per_launch"] = by_l
    out["frac"] = out["achieved"] / out["peak"]
    out["traffic"] = traffic
    out["mfma_frac"] = fl_l / dur / 1e12 / peak_f
    out.update(kernel=name, launch_avg_us=kt[name]["avg_us"], launches_per_step=launches,
               min_bytes_per_launch=by_l, algorithmic_flops_per_launch=fl_l,
               share_of_step=kt[name]["total_ms"] / res["ms"])
    for k in ("achieved", "frac", "mfma_frac", "share_of_step"):
        out[k] = round(out[k], 5)
    return out


def rates(cfg, p, rh):
    """(p_nr, p_rh) of a mode: p on every site, or the config's per-layer
    rate vectors when it has them."""
    if cfg.p_nr_layers is not None:
        return list(cfg.p_nr_layers), (list(cfg.p_rh_layers) if rh else 0.0)
    return p, (p if rh else 0.0)


def mode_summary(r, rd, cfg, wl):
    """One mode (compact r, dense rd) of a config."""
    out = {"ms_per_step": round(r["ms"], 4),
           "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 4),
           "gflop_per_step": round(r["flops"] / 1e9, 4),
           "step_ms_p10_p50_p90": [round(v, 4) for v in r["pct"]]}
    if rd is not None:
        out.update(dense_ms_per_step=round(rd["ms"], 4), speedup_vs_dense=round(rd["ms"] / r["ms"], 4),
                   dense_equiv_tflops=round(algorithmic_flops(dense_counts(cfg), cfg, wl.lengths)
                                            / (r["ms"] * 1e-3) / 1e12, 4))
    if r["ktime"]:
        ph = phase_times(r)
        out["phases_ms"] = ph
        out["kernels"] = kernel_table(r, cfg)
        if rd is not None and rd["ktime"]:
            phd = phase_times(rd)
            out["phases_ms_dense"] = phd
            out["phase_speedup"] = {k: round(phd[k] / ph[k], 4) for k in ph if ph[k] > 0 and phd[k] > 0}
    return out


def config_block(name, steps, warmup, cpu, no_dense=False, sweep=True):
    """Every mode of one config: NR+ST and NR+RH+ST, each against the same
    kernels run dense, with kernel-class times; the p sweep of configs that
    have one (speedups only); the oracle on the host."""
    import workloads
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = 0.5 if 0.5 in cfg.p_values else cfg.p_values[0]
    kst = max(5, min(steps, 20))            # steps of each per-kernel-class pass
    out = {"layers": cfg.num_layers, "dirs": cfg.num_dirs, "input_dim": cfg.input_dim, "hidden": cfg.hidden,
           "batch": cfg.batch, "seq_len": cfg.seq_len, "dtype": cfg.dtype}
    for mode, rh in (("nr_st", False), ("nr_rh_st", True)):
        pn, pr = rates(cfg, p, rh)
        r = run_mode(wl, pn, pr, 1, steps, warmup, timed_kernels=KERNELS, kernel_steps=kst)
        rd = None if no_dense else run_mode(wl, pn, pr, 0, steps, warmup, timed_kernels=KERNELS, kernel_steps=kst)
        out[mode] = dict(p_nr=pn, p_rh=pr, **mode_summary(r, rd, cfg, wl))
        if mode == "nr_st":
            out["roofline"] = roofline(r, cfg)
    if sweep and len(cfg.p_values) > 1 and not no_dense:
        sw = {}
        for q in cfg.p_values:
            if q == p:
                continue
            ent = {}
            for mode, rh in (("nr_st", False), ("nr_rh_st", True)):
                pn, pr = rates(cfg, q, rh)
                r = run_mode(wl, pn, pr, 1, steps, warmup)
                rd = run_mode(wl, pn, pr, 0, steps, warmup)
                ent[mode] = {"ms_per_step": round(r["ms"], 4), "dense_ms_per_step": round(rd["ms"], 4),
                             "speedup_vs_dense": round(rd["ms"] / r["ms"], 4),
                             "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 4)}
            sw[str(q)] = ent
        out["p_sweep"] = sw
    if cpu:
        rows = None if cfg.batch <= 64 else np.arange(32)
        out["cpu_baseline"] = cpu_baseline(wl, *rates(cfg, p, False), budget_s=2.0, max_steps=3, rows=rows)
    return out


def cpu_baseline(wl, p_nr, p_rh, budget_s=12.0, max_steps=50, rows=None):
    """The float64 oracle as it stands, timed on the host on whole training
    steps of the same workload until about budget_s seconds of CPU work (at
    most max_steps steps).  rows: time the oracle on these batch rows only
    (the same workload's first rows; FLOPs counted for those rows)."""
    import workloads
    from oracle import lstm, masks
    cfg = wl.cfg
    B = cfg.batch
    if rows is not None:
        wl = workloads.slice_rows(wl, rows)
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count() or 1
    P = lstm.params_from(wl.W, wl.U, wl.b, cfg.num_layers, cfg.num_dirs)
    n, t_tot, flops = 0, 0.0, 0.0
    while t_tot < budget_s and n < max_steps:
        t0 = time.perf_counter()
        m_nr, m_rh = masks.all_masks(cfg.mask_seed, n, cfg.num_layers, cfg.num_dirs, cfg.seq_len,
                                     cfg.k_in, cfg.hidden, p_nr, p_rh)
        lstm.train_step(P, wl.x, wl.h0, wl.c0, m_nr, m_rh, p_nr, p_rh, cfg.loss, wl.target, wl.lengths)
        t_tot += time.perf_counter() - t0
        counts = [m.sum(1) for m in m_nr] + [m_rh[l][d].sum(1) for l in range(cfg.num_layers)
                                              for d in range(cfg.num_dirs)]
        flops += algorithmic_flops(counts, cfg, wl.lengths) * (wl.x.shape[1] / B)
        n += 1
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return dict(value=round(flops / t_tot / 1e12, 6), unit="TFLOP/s", cores=int(threads), kind="oracle",
                cpu_count=os.cpu_count(), cpu_model=model,
                sample=f"{n} whole training steps of the {cfg.name} workload"
                       + ("" if rows is None else f" on its first {len(rows)} of {B} batch rows")
                       + f" (NR+ST, masks of steps 0..{n - 1}), float64 NumPy oracle, {t_tot / n * 1e3:.0f} ms/step",
                ms_per_step=round(t_tot / n * 1e3, 3))


KERNEL_SYMBOLS = {"fwd_persist": ("lsd::k_fwd_persist<", "lsd::k_fwd_big<"), "step": ("lsd::k_step<",),
                  "bwd_persist": ("lsd::k_bwd_persist<", "lsd::k_bwd_big"), "bwd": ("lsd::k_bwd<",),
                  "wgrad": ("lsd::k_wgrad",),            # the row-sparse, the full and the large-batch kernel
                  "fx": ("lsd::k_fx<", "lsd::k_fx_big"), "dx": ("lsd::k_dx<", "lsd::k_dx_big"),
                  "mask_build": ("lsd::k_mask_build",), "transpose": ("lsd::k_trans",)}
SIMDS = 256 * 4             # MI355X: 256 compute units of 4 SIMDs
XCDS = 8                    # GRBM_GUI_ACTIVE is counted once per XCD
MFMA_BF16_FLOP_PER_MOP = 512


def kernel_class(name):
    for k, syms in KERNEL_SYMBOLS.items():
        if any(sym in name for sym in syms):
            return k
    return None


def summarize_pmc(paths, command):
    """Markdown summary of rocprofv3 --pmc counter runs (one CSV per pass)
    per kernel class: dispatches, average duration, MFMA busy fraction
    (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE per XCD times the SIMD
    count), MFMA rate from the bf16 MOPS count, and every other counter's
    mean per dispatch."""
    import csv
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(dict)
    names = collections.defaultdict(set)
    for path in paths:
        for r in csv.DictReader(open(path)):
            k = kernel_class(r["Kernel_Name"])
            if k is None:
                continue
            names[k].add(r["Kernel_Name"].split("(")[0].replace("void ", ""))
            vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
            dur[k][(path, r["Dispatch_Id"])] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
    lines = ["| class | kernels | dispatches | avg us | MFMA busy | MFMA TFLOP/s (bf16 MOPS) | counters (mean per dispatch) |",
             "|---|---|---|---|---|---|---|"]
    for k in KERNEL_SYMBOLS:
        if k not in vals:
            continue
        v = {c: float(np.mean(x)) for c, x in vals[k].items()}
        us = float(np.mean(list(dur[k].values())))
        busy = ""
        if "SQ_VALU_MFMA_BUSY_CYCLES" in v and "GRBM_GUI_ACTIVE" in v and v["GRBM_GUI_ACTIVE"] > 0:
            busy = f"{100.0 * v['SQ_VALU_MFMA_BUSY_CYCLES'] / (v['GRBM_GUI_ACTIVE'] / XCDS * SIMDS):.1f}%"
        rate = ""
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in v and us > 0:
            rate = f"{v['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * MFMA_BF16_FLOP_PER_MOP / (us * 1e-6) / 1e12:.1f}"
        others = ", ".join(f"{c} {x:.4g}" for c, x in sorted(v.items()))
        lines.append(f"| {k} | {' '.join(sorted(names[k]))} | {len(dur[k])} | {us:.1f} | {busy} | {rate} | {others} |")
    return "\n".join([f"Command: `{command}`", ""] + lines)


def summarize_stats(path, command):
    """Markdown table of a rocprofv3 --stats kernel summary (library kernels
    first, by total time)."""
    import csv
    rows = list(csv.DictReader(open(path)))
    lines = [f"Command: `{command}`", "", "| kernel | class | calls | total ms | avg us | min us | max us | % |",
             "|---|---|---|---|---|---|---|---|"]
    for r in rows:
        k = kernel_class(r["Name"])
        lines.append(f"| {r['Name'].split('(')[0].replace('void ', '')[:70]} | {k or ''} | {r['Calls']} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines)


def summarize_trace(path, command):
    """Markdown table of a rocprofv3 --kernel-trace CSV grouped by kernel and
    grid (workgroups x, y, z), so that launches of one kernel on different
    problems (the LSTM's and the output head's) stand apart.  Microseconds."""
    import csv
    import collections
    agg = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"].split("(")[0].replace("void ", "")
        if not name.startswith("lsd::"):
            continue
        grid = tuple(int(r[f"Grid_Size_{a}"]) // max(1, int(r[f"Workgroup_Size_{a}"])) for a in "XYZ")
        agg[(name, grid)].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    lines = [f"Command: `{command}`", "", "| Kernel | Grid (workgroups) | Calls | Average | Min | Max |",
             "|---|---|---:|---:|---:|---:|"]
    for (name, grid), v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"| `{name[:70]}` | {grid[0]} x {grid[1]} x {grid[2]} | {len(v)} | {sum(v) / len(v):.2f} | "
                     f"{min(v):.2f} | {max(v):.2f} |")
    return "\n".join(lines)


def summarize_counters(fetch_csv, write_csv, copy_bytes, workload, command):
    """Turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; KiB per
    dispatch) into HBM bytes per launch of each kernel class.  Each counter is
    scaled by what it reads for a plain device copy of copy_bytes bytes (the
    largest copy dispatch in the same run).  Writes profiles/traffic.json."""
    import csv
    import collections

    def per_kernel(path):
        agg = collections.defaultdict(list)
        copy = 0.0
        for r in csv.DictReader(open(path)):
            v = float(r["Counter_Value"])
            name = r["Kernel_Name"]
            if "copyBuffer" in name or "copy_kernel" in name:
                copy = max(copy, v)
            k = kernel_class(name)
            if k is not None:
                agg[k].append(v)
        return agg, copy

    fetch, fcopy = per_kernel(fetch_csv)
    write, wcopy = per_kernel(write_csv)
    ffac = copy_bytes / (fcopy * 1024.0)
    wfac = copy_bytes / (wcopy * 1024.0)
    out = {"_calibration": {"copy_bytes": copy_bytes, "fetch_kib_of_copy": fcopy, "write_kib_of_copy": wcopy,
                            "fetch_factor": ffac, "write_factor": wfac, "command": command}}
    for k in KERNEL_SYMBOLS:
        if k in fetch and k in write:
            f = float(np.mean(fetch[k])) * 1024.0 * ffac
            w = float(np.mean(write[k])) * 1024.0 * wfac
            out[k] = {"workload": workload, "src_hash": kernel_src_hash(), "fetch_kib": float(np.mean(fetch[k])),
                      "write_kib": float(np.mean(write[k])), "bytes_per_launch": f + w,
                      "fetch_bytes": f, "write_bytes": w, "dispatches": len(fetch[k])}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as fo:
        json.dump(out, fo, indent=1)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-nrrh", action="store_true", help="skip the NR+RH+ST runs")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense comparison runs (counter passes)")
    ap.add_argument("--no-head", action="store_true", help="skip the language-model output head runs")
    ap.add_argument("--no-case4", action="store_true", help="skip the Case-IV (fixed-in-time mask) runs")
    ap.add_argument("--no-case1", action="store_true", help="skip the Case-I (NR+Random) comparator run")
    ap.add_argument("--configs", default="all",
                    help="other workloads to measure in the same run: 'all', 'none' or a comma list")
    ap.add_argument("--no-sweep", action="store_true", help="skip the p sweep of the tagger and stress workloads")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic.json from two rocprofv3 --pmc runs and exit (no GPU)")
    ap.add_argument("--counter-command", default="", help="command recorded with the summaries")
    ap.add_argument("--summarize-pmc", nargs="+", metavar="CSV",
                    help="print a markdown summary of rocprofv3 --pmc counter CSVs per kernel class and exit (no GPU)")
    ap.add_argument("--summarize-trace", metavar="CSV",
                    help="print a markdown table of a rocprofv3 kernel-trace CSV by kernel and grid, and exit")
    ap.add_argument("--summarize-stats", metavar="CSV",
                    help="print a markdown table of a rocprofv3 --stats kernel summary and exit (no GPU)")
    args = ap.parse_args(argv)
    if args.summarize_pmc:
        print(summarize_pmc(args.summarize_pmc, args.counter_command))
        return 0
    if args.summarize_stats:
        print(summarize_stats(args.summarize_stats, args.counter_command))
        return 0
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.counter_command))
        return 0
    if args.summarize_counters:
        out = summarize_counters(*args.summarize_counters, copy_bytes=args.calibrate_copy * (1 << 20),
                                 workload=args.workload, command=args.counter_command)
        print(json.dumps(out, indent=1))
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU (asked for --gpus {args.gpus}): this build has no "
              "multi-GPU path; the data-parallel design is described but not built.", file=sys.stderr)
        return 2
    import torch
    import workloads
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    cfg = workloads.get_config(args.workload)
    wl = workloads.make_workload(cfg)
    p = 0.5 if 0.5 in cfg.p_values else cfg.p_values[0]
    kst = max(5, min(args.steps, 20))
    head = run_mode(wl, p, 0.0, 1, args.steps, args.warmup, timed_kernels=KERNELS, kernel_steps=kst)
    dense = None if args.no_dense else run_mode(wl, p, 0.0, 0, args.steps, args.warmup, timed_kernels=KERNELS,
                                                kernel_steps=kst)
    ms = mode_summary(head, dense, cfg, wl)
    out = {
        "metric": METRIC,
        "value": round(head["flops"] / (head["ms"] * 1e-3) / 1e12, 4),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "layers": cfg.num_layers, "dirs": cfg.num_dirs,
                   "input_dim": cfg.input_dim, "hidden": cfg.hidden, "batch": cfg.batch,
                   "seq_len": cfg.seq_len, "p_nr": p, "p_rh": 0.0, "mode": "NR+ST"},
        "value_kind": "effective TFLOP/s over kept-row FLOPs",
        "speedup_vs_dense": ms.get("speedup_vs_dense"),
        "dense_ms_per_step": ms.get("dense_ms_per_step"),
        "gflop_per_step": ms["gflop_per_step"],
        "dense_equiv_tflops": ms.get("dense_equiv_tflops"),
        "step_ms_p10_p50_p90": ms["step_ms_p10_p50_p90"],
        "step_ms_p10_p50_p90_note": "per-step times of the pass with phase events (about 19 us above the clean pass)",
        "host_phases_ms": {k: round(v, 4) for k, v in head["phases"].items()},
        "phases_ms": ms.get("phases_ms"),
        "phases_ms_dense": ms.get("phases_ms_dense"),
        "phase_speedup": ms.get("phase_speedup"),
        "kernels": ms.get("kernels"),
        "roofline": roofline(head, cfg),
    }
    if not args.no_nrrh:
        r = run_mode(wl, p, p, 1, args.steps, args.warmup, timed_kernels=KERNELS, kernel_steps=kst)
        rd = None if args.no_dense else run_mode(wl, p, p, 0, args.steps, args.warmup, timed_kernels=KERNELS,
                                                 kernel_steps=kst)
        out["nrrh"] = dict(p_nr=p, p_rh=p, **mode_summary(r, rd, cfg, wl))
    if not args.no_case1:
        c1 = run_case1(wl, p, args.steps, args.warmup)
        out["case1"] = {"what": "Case-I (NR+Random) comparator: per-element input dropout, every layer dense",
                        "ms_per_step": round(c1, 4), "speedup_of_nr_st": round(c1 / head["ms"], 4)}
    if not args.no_case4:
        c4 = run_mode(wl, p, 0.0, 1, args.steps, args.warmup, fixed=True)
        c4r = run_mode(wl, p, p, 1, args.steps, args.warmup, fixed=True)
        out["case4"] = {"what": "Case-IV masks (one draw per site for the whole sequence), same kernels",
                        "ms_per_step": round(c4["ms"], 4), "nrrh_ms_per_step": round(c4r["ms"], 4)}
    if wl.tokens is not None:
        out["embedding_backward"] = run_embedding(wl, p, args.steps, args.warmup)
        if not args.no_cpu:
            out["embedding_backward"]["cpu_baseline"] = embedding_cpu_baseline(wl, p)
    if wl.W_fc is not None and not args.no_head:
        hc = run_head(wl, p, args.steps, args.warmup, 1)
        hd = None if args.no_dense else run_head(wl, p, args.steps, args.warmup, 0)
        out["head"] = {"vocab": int(wl.W_fc.shape[1]), "p_out": p, "ms_per_step": round(hc["head"], 4),
                       "dense_ms_per_step": round(hd["head"], 4) if hd else None,
                       "speedup_vs_dense": round(hd["head"] / hc["head"], 4) if hd else None,
                       "tflops": round(hc["flops"] / (hc["head"] * 1e-3) / 1e12, 2),
                       "gflop_per_step": round(hc["flops"] / 1e9, 3),
                       "kernels_us_per_step": hc["kernels_us_per_step"],
                       "kernels_us_per_step_dense": hd["kernels_us_per_step"] if hd else None,
                       "roofline": head_roofline(hc, cfg)}
        if not args.no_cpu:
            out["head"]["cpu_baseline"] = head_cpu_baseline(wl, p)
        out["lm_step_with_head"] = {"ms_per_step": round(hc["lm_step"], 4),
                                    "dense_ms_per_step": round(hd["lm_step"], 4) if hd else None,
                                    "speedup_vs_dense": round(hd["lm_step"] / hc["lm_step"], 4) if hd else None}
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = n * 4
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, p, 0.0)
    names = [] if args.configs in ("", "none") else \
        [c for c in (CONFIG_RUNS if args.configs == "all" else args.configs.split(",")) if c != cfg.name]
    if names:
        out["configs"] = {}
        for name in names:
            print(f"[bench] config {name}", file=sys.stderr, flush=True)
            out["configs"][name] = config_block(name, args.steps, args.warmup, not args.no_cpu, args.no_dense,
                                                not args.no_sweep)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
