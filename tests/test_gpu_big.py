"""The large-batch kernels (the persistent forward with its U slice held in
registers, the contraction split over the waves and summed through LDS; the
input products, input gradients and weight gradients on 256-row tiles) on
ragged shapes,
forced with LSTM_SD_BIG=2 (it otherwise runs only where the row-group
tiling of the other persistent forward does not fit, as at the stress
shape): hidden sizes that are not multiples of the 32-neuron chunk or of the
16-unit tile, batches that are not multiples of the 64-row group or of the
16-row MFMA tile, both directions, per-row lengths, and both modes; the
weight gradients on the default GEMM and on the row-sparse kernel."""
import dataclasses

import numpy as np
import pytest

import workloads
from tests._parity import TOL, compare, oracle_step, say, summary

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(cfg, wl, p_nr, p_rh, compact):
    from oracle import masks as om
    from paper_2106_12089_amd.session import Session
    s = Session(wl, p_nr, p_rh, compact)
    s.masks(cfg.mask_seed, 0)
    s.forward()
    s.loss_grad()
    s.backward()
    torch.cuda.synchronize()
    m_nr, m_rh = om.all_masks(cfg.mask_seed, 0, cfg.num_layers, cfg.num_dirs, cfg.seq_len, cfg.k_in,
                              cfg.hidden, p_nr, p_rh)
    return s.outputs(), oracle_step(wl, p_nr, p_rh, m_nr, m_rh)


@pytest.mark.parametrize("shape", [
    dict(num_layers=2, num_dirs=1, input_dim=70, hidden=45, batch=70, seq_len=5),
    dict(num_layers=1, num_dirs=2, input_dim=129, hidden=100, batch=19, seq_len=4),
    dict(num_layers=2, num_dirs=1, input_dim=64, hidden=1000, batch=130, seq_len=3),
    dict(num_layers=1, num_dirs=1, input_dim=33, hidden=512, batch=64, seq_len=6, min_len=0),
    dict(num_layers=2, num_dirs=2, input_dim=200, hidden=72, batch=300, seq_len=3),
    dict(num_layers=1, num_dirs=2, input_dim=48, hidden=40, batch=1030, seq_len=3),
])
@pytest.mark.parametrize("mode", [(0.5, 0.5, 1), (0.5, 0.5, 0), (0.3, 0.0, 1)])
def test_big_forward_ragged(shape, mode, monkeypatch):
    monkeypatch.setenv("LSTM_SD_BIG", "2")
    base = workloads.get_config("tiny")
    cfg = dataclasses.replace(base, name="big", dtype="bf16", loss="mse", **shape)
    wl = workloads.make_workload(cfg)
    p_nr, p_rh, compact = mode
    say(f"[gpu] big forward {shape} p_nr={p_nr} p_rh={p_rh} compact={compact}")
    gpu, ref = _run(cfg, wl, p_nr, p_rh, compact)
    errs = compare(gpu, ref)
    say("   errs", summary(errs))
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    assert not bad, bad
    if cfg.min_len is not None:
        valid = np.arange(cfg.seq_len)[:, None] < wl.lengths[None, :]
        assert np.all(gpu["y"][~valid] == 0.0)


@pytest.mark.parametrize("shape", [
    dict(num_layers=2, num_dirs=1, input_dim=70, hidden=45, batch=70, seq_len=5),
    dict(num_layers=2, num_dirs=2, input_dim=200, hidden=72, batch=300, seq_len=3),
])
@pytest.mark.parametrize("mode", [(0.5, 0.5, 1), (0.5, 0.5, 0)])
def test_big_wgrad_rowsparse_kernel(shape, mode, monkeypatch):
    """The large-batch row-sparse weight-gradient kernel (per-step gathered
    rows; LSTM_SD_WGRAD_GEMM=0) in place of the default mask-multiplied
    GEMM."""
    monkeypatch.setenv("LSTM_SD_BIG", "2")
    monkeypatch.setenv("LSTM_SD_WGRAD_GEMM", "0")
    base = workloads.get_config("tiny")
    cfg = dataclasses.replace(base, name="big", dtype="bf16", loss="mse", **shape)
    wl = workloads.make_workload(cfg)
    p_nr, p_rh, compact = mode
    say(f"[gpu] big row-sparse wgrad {shape} p_nr={p_nr} p_rh={p_rh} compact={compact}")
    gpu, ref = _run(cfg, wl, p_nr, p_rh, compact)
    errs = compare(gpu, ref)
    say("   errs", summary(errs))
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    assert not bad, bad


@pytest.mark.parametrize("mode", [(0.3, 0.0, 1), (0.5, 0.5, 1), (0.5, 0.5, 0)])
def test_big_repeats_bit_identical(mode, monkeypatch):
    """The same step on the same masks gives the same bits every time: the
    large-batch kernels' exchanges and the weight gradient's accumulator
    (whose rows move between waves from step to step) leave no room for a
    race.  A hidden size around the 32-row tile boundary at keep rate 0.7
    puts rows in both tiles."""
    from paper_2106_12089_amd.session import Session
    monkeypatch.setenv("LSTM_SD_BIG", "2")
    base = workloads.get_config("tiny")
    cfg = dataclasses.replace(base, name="big", dtype="bf16", loss="mse", num_layers=2, num_dirs=1, input_dim=70,
                              hidden=45, batch=70, seq_len=5)
    wl = workloads.make_workload(cfg)
    p_nr, p_rh, compact = mode
    say(f"[gpu] big repeats p_nr={p_nr} p_rh={p_rh} compact={compact}")
    ref = None
    for it in range(6):
        s = Session(wl, p_nr, p_rh, compact)
        s.masks(cfg.mask_seed, 0)
        s.forward()
        s.loss_grad()
        s.backward()
        torch.cuda.synchronize()
        o = s.outputs()
        cur = {k: np.concatenate([np.ravel(a) for a in v]) if isinstance(v, list) else np.ravel(v)
               for k, v in o.items() if v is not None and k != "loss"}
        if ref is None:
            ref = cur
            continue
        diff = [k for k in ref if not np.array_equal(ref[k], cur[k])]
        assert not diff, (it, diff)
