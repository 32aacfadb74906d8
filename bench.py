"""Benchmark of one structured-dropout LSTM training step on one MI355X.

A step is one pass of the whole path on one batch of synthetic input that
is already resident in HBM: draw the Case-III masks and build the keep lists
(fresh masks every step), forward unroll, MSE loss gradient, BPTT with the
weight gradients.  The workload is the 2-layer, 650-unit language-model
shape (batch 20, 35 steps, bf16 storage with fp32 accumulation, structured
dropout p = 0.5 on the non-recurrent inputs).  Prints one JSON line.

  value      effective TFLOP/s: algorithmic FLOPs of the step (products over
             the actually kept rows, 3 products per gate GEMM) / step time
  speedup    same kernels run dense (compact = 0) / method
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "lm_medium"
METRIC = "LSTM fwd+BPTT step time & eff. TFLOP/s; speedup vs dense at p=0.5"


def algorithmic_flops(counts, cfg, lengths=None):
    """Sum over layers, directions and t of 3 * 2 * B_t * 4H * (n_x + n_h):
    the forward product, the input-gradient product and the weight-gradient
    product of every gate GEMM, over kept rows only (B_t = valid rows)."""
    L, D, H, T, B = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.batch
    if lengths is None:
        bt = np.full(T, B)
    else:
        bt = (np.arange(T)[:, None] < np.asarray(lengths)[None, :]).sum(1)
    tot = 0.0
    for l in range(L):
        for d in range(D):
            nx = counts[l]
            nh = counts[L + l * D + d]
            tot += float(np.sum(3 * 2 * bt * 4 * H * (nx + nh)))
    return tot


def dense_flops(cfg, lengths=None):
    L, D, H, T, B, I = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.batch, cfg.input_dim
    counts = []
    for l in range(L):
        counts.append(np.full(T, I if l == 0 else D * H))
    for _ in range(L * D):
        counts.append(np.full(T, H))
    return algorithmic_flops(counts, cfg, lengths)


def time_mode(wl, p_nr, p_rh, compact, steps, warmup, seed0):
    import torch
    from paper_2106_12089_amd.session import Session
    s = Session(wl, p_nr, p_rh, compact)
    cfg = wl.cfg
    for i in range(warmup):
        s.step(cfg.mask_seed, 10_000 + i)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    phase = np.zeros(4)
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        ev[0].record()
        s.masks(cfg.mask_seed, seed0 + i)
        ev[1].record()
        s.forward()
        ev[2].record()
        s.loss_grad()
        ev[3].record()
        s.backward()
        ev[4].record()
        if i == steps - 1:
            break
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(end)
    for k in range(4):
        phase[k] = ev[k].elapsed_time(ev[k + 1])   # last step's phases
    # kept counts of every timed step (regenerated; outside the timed region)
    flops = 0.0
    lay = None
    from paper_2106_12089_amd import binding as B_
    lay = B_.lstm_sd_mask_layout_get(s.dims)
    for i in range(steps):
        s.masks(cfg.mask_seed, seed0 + i)
        count = s.mask_views()[3]
        flops += algorithmic_flops(count, cfg, wl.lengths)
    return dict(ms=total_ms / steps, wall_ms=wall * 1e3 / steps, flops=flops / steps,
                phases_last_ms=dict(mask=phase[0], forward=phase[1], loss=phase[2], backward=phase[3]),
                session=s)


def cpu_baseline(wl, p_nr, p_rh, budget_s=12.0):
    """The float64 oracle (untuned), timed on the host on whole steps of the
    same workload until about budget_s seconds of CPU work are done."""
    from oracle import lstm, masks
    cfg = wl.cfg
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count() or 1
    P = lstm.params_from(wl.W, wl.U, wl.b, cfg.num_layers, cfg.num_dirs)
    n, t_tot, flops = 0, 0.0, 0.0
    while t_tot < budget_s and n < 50:
        t0 = time.perf_counter()
        m_nr, m_rh = masks.all_masks(cfg.mask_seed, n, cfg.num_layers, cfg.num_dirs, cfg.seq_len,
                                     cfg.k_in, cfg.hidden, p_nr, p_rh)
        lstm.train_step(P, wl.x, wl.h0, wl.c0, m_nr, m_rh, p_nr, p_rh, cfg.loss, wl.target, wl.lengths)
        t_tot += time.perf_counter() - t0
        counts = [m.sum(1) for m in m_nr] + [m_rh[l][d].sum(1) for l in range(cfg.num_layers)
                                              for d in range(cfg.num_dirs)]
        flops += algorithmic_flops(counts, cfg, wl.lengths)
        n += 1
    return dict(value=flops / t_tot / 1e12, unit="TFLOP/s", cores=int(threads), kind="oracle",
                sample=f"{n} whole training steps of the {cfg.name} workload (float64 NumPy oracle, "
                       f"{t_tot / n * 1e3:.0f} ms/step)",
                ms_per_step=t_tot / n * 1e3)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--all-modes", action="store_true", help="also time NR+RH+ST and its dense run")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              "data-parallel path is not part of this build.", file=sys.stderr)
        return 2
    import torch
    import workloads
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    cfg = workloads.get_config(args.workload)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0] if 0.5 not in cfg.p_values else 0.5
    res = {}
    modes = [("nr", p, 0.0)] + ([("nrrh", p, p)] if args.all_modes else [])
    for name, pn, pr in modes:
        res[name] = time_mode(wl, pn, pr, 1, args.steps, args.warmup, 0)
        res[name + "_dense"] = time_mode(wl, pn, pr, 0, args.steps, args.warmup, 0)
    head = res["nr"]
    dense = res["nr_dense"]
    out = {
        "metric": METRIC,
        "value": round(head["flops"] / (head["ms"] * 1e-3) / 1e12, 4),
        "unit": "TFLOP/s (effective, kept-row FLOPs)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": cfg.name, "layers": cfg.num_layers, "dirs": cfg.num_dirs,
                   "input_dim": cfg.input_dim, "hidden": cfg.hidden, "batch": cfg.batch,
                   "seq_len": cfg.seq_len, "p_nr": p, "p_rh": 0.0, "mode": "NR+ST"},
        "speedup_vs_dense": round(dense["ms"] / head["ms"], 4),
        "dense_ms_per_step": round(dense["ms"], 4),
        "gflop_per_step": round(head["flops"] / 1e9, 4),
        "dense_equiv_tflops": round(dense_flops(cfg, wl.lengths) / (head["ms"] * 1e-3) / 1e12, 4),
        "phases_ms": {k: round(v, 4) for k, v in head["phases_last_ms"].items()},
    }
    if args.all_modes:
        r, rd = res["nrrh"], res["nrrh_dense"]
        out["nrrh"] = {"ms_per_step": round(r["ms"], 4), "dense_ms_per_step": round(rd["ms"], 4),
                       "speedup_vs_dense": round(rd["ms"] / r["ms"], 4),
                       "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 4)}
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, p, 0.0)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
