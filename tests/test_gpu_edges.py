"""Edge cases of the HIP path against the oracle: ragged sizes that are not
multiples of any tile, contractions at the size limit, a single row and step, zero-length rows, rates of 0,
forced mask patterns (a neuron never kept, a step with everything dropped,
everything kept) and the dense/compact equivalence."""
import dataclasses

import numpy as np
import pytest

import workloads
from tests._parity import TOL, compare, fwd_persist_launches, oracle_step, say, site_list

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def make(name, **kw):
    base = workloads.get_config("tiny")
    cfg = dataclasses.replace(base, name=name, **kw)
    return cfg, workloads.make_workload(cfg)


def run_both(cfg, wl, p_nr, p_rh, compact, forced=None, dhT=False):
    from paper_2106_12089_amd.session import Session
    from oracle import masks as om
    s = Session(wl, p_nr, p_rh, compact)
    s.masks(cfg.mask_seed, 0)
    m_nr, m_rh = om.all_masks(cfg.mask_seed, 0, cfg.num_layers, cfg.num_dirs, cfg.seq_len, cfg.k_in,
                              cfg.hidden, p_nr, p_rh)
    if forced is not None:
        m_nr, m_rh = forced(m_nr, m_rh)
        mask = s.mask_views()[0]
        mask = mask.copy()
        for i, m in enumerate(site_list(cfg, m_nr, m_rh)):
            mask[i, :, :m.shape[1]] = m
        s.write_masks(mask)
    s.forward()
    s.loss_grad()
    s.backward()
    torch.cuda.synchronize()
    gpu = s.outputs()
    ref = oracle_step(wl, p_nr, p_rh, m_nr, m_rh)
    return gpu, ref, m_nr, m_rh


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [
    dict(num_layers=2, num_dirs=2, input_dim=37, hidden=45, batch=19, seq_len=3),
    dict(num_layers=1, num_dirs=1, input_dim=5, hidden=3, batch=1, seq_len=1),
    dict(num_layers=3, num_dirs=1, input_dim=70, hidden=33, batch=35, seq_len=5),
    dict(num_layers=1, num_dirs=2, input_dim=129, hidden=100, batch=70, seq_len=4),
])
@pytest.mark.parametrize("mode", ["nrrh", "nrrh_dense"])
def test_ragged_shapes(shape, dtype, mode):
    cfg, wl = make("ragged", dtype=dtype, loss="mse", **shape)
    compact = 0 if mode.endswith("dense") else 1
    say(f"[gpu] ragged {shape} {dtype} {mode}")
    gpu, ref, _, _ = run_both(cfg, wl, 0.5, 0.5, compact)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL[dtype], errs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [
    dict(num_layers=2, num_dirs=2, input_dim=2048, hidden=1024, batch=5, seq_len=2),
    dict(num_layers=1, num_dirs=1, input_dim=40, hidden=2048, batch=3, seq_len=2),
    dict(num_layers=2, num_dirs=2, input_dim=2048, hidden=1024, batch=64, seq_len=2),
    dict(num_layers=1, num_dirs=1, input_dim=64, hidden=2048, batch=64, seq_len=2),
])
def test_contractions_at_the_size_limit(shape, dtype):
    """Every contraction length at the library's limit of 2048: the input
    width and the stacked layer's input D*H, the recurrent H; at a small
    batch and at 64 rows (the large-batch kernels, and for H = 2048 the
    per-step recurrence that serves shapes past their register budget)."""
    cfg, wl = make("kmax", dtype=dtype, loss="mse", **shape)
    say(f"[gpu] size limit {shape} {dtype}")
    gpu, ref, _, _ = run_both(cfg, wl, 0.5, 0.5, 1)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL[dtype], errs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_long_sequence(dtype):
    """257 steps, two stacked bidirectional layers: many barrier generations
    of the persistent recurrences, and rounding carried through a long
    forward and BPTT."""
    cfg, wl = make("long", dtype=dtype, loss="mse", num_layers=2, num_dirs=2, input_dim=80, hidden=96,
                   batch=21, seq_len=257)
    say(f"[gpu] long sequence {dtype}")
    gpu, ref, _, _ = run_both(cfg, wl, 0.5, 0.5, 1)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL[dtype], errs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lengths_with_zero_rows(dtype):
    cfg, wl = make("lens", dtype=dtype, loss="mse", num_layers=2, num_dirs=2, input_dim=24, hidden=20,
                   batch=6, seq_len=7, min_len=0)
    wl.lengths[:] = np.array([7, 0, 3, 1, 6, 0], dtype=np.int32)
    valid = np.arange(cfg.seq_len)[:, None] < wl.lengths[None, :]
    wl.x[~valid] = 0.0
    say(f"[gpu] lengths {dtype}")
    gpu, ref, _, _ = run_both(cfg, wl, 0.5, 0.5, 1)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL[dtype], errs
    assert np.all(gpu["y"][~valid] == 0.0)


def test_rate_zero_is_plain_lstm():
    cfg, wl = make("p0", dtype="f32", loss="mse")
    say("[gpu] p = 0")
    gpu, ref, m_nr, _ = run_both(cfg, wl, 0.0, 0.0, 1)
    assert all(m.all() for m in m_nr)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL["f32"], errs


@pytest.mark.parametrize("compact", [1, 0])
def test_forced_patterns(compact):
    cfg, wl = make("forced", dtype="f32", loss="mse", num_layers=2, input_dim=40, hidden=24, batch=5,
                   seq_len=6)

    def force(m_nr, m_rh):
        m_nr = [m.copy() for m in m_nr]
        m_rh = [[m.copy() for m in r] for r in m_rh]
        m_nr[1][1, :] = 1          # everything kept at t = 1 (but neuron 3, below)
        m_nr[0][:, 7] = 0          # never kept: zero dW row
        m_nr[1][:, 3] = 0
        m_rh[1][0][:, 5] = 0       # never kept: zero dU row
        m_nr[0][2, :] = 0          # everything dropped at t = 2
        m_rh[0][0][4, :] = 0
        return m_nr, m_rh

    say(f"[gpu] forced patterns compact={compact}")
    gpu, ref, m_nr, m_rh = run_both(cfg, wl, 0.5, 0.5, compact, forced=force)
    errs = compare(gpu, ref)
    assert max(errs.values()) <= TOL["f32"], errs
    assert np.all(gpu["dW"][0][7] == 0.0)
    assert np.all(gpu["dW"][1][3] == 0.0)
    assert np.all(gpu["dU"][1][5] == 0.0)
    assert np.all(gpu["dx"][2] == 0.0)


def test_dense_equals_compact():
    cfg = workloads.get_config("lm_medium")
    wl = workloads.make_workload(cfg)
    from paper_2106_12089_amd.session import Session
    say("[gpu] dense vs compact lm_medium")
    outs = []
    for compact in (1, 0):
        s = Session(wl, 0.5, 0.5, compact)
        s.step(cfg.mask_seed, 1)
        torch.cuda.synchronize()
        outs.append(s.outputs())
    errs = compare(outs[0], outs[1])
    assert max(errs.values()) <= 1e-2, errs


def test_mse_kernel_matches_oracle():
    from oracle import lstm
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config("seq2seq_enc")
    wl = workloads.make_workload(cfg)
    s = Session(wl, 0.3, 0.0, 1)
    say("[gpu] mse kernel")
    y = np.random.default_rng(0).normal(size=s.y.shape).astype(np.float32)
    valid = np.arange(cfg.seq_len)[:, None] < wl.lengths[None, :]
    y[~valid] = 0.0
    s.y.copy_(torch.from_numpy(y))
    s.loss_grad()
    torch.cuda.synchronize()
    loss, dy = lstm.loss_mse(y, wl.target, wl.lengths)
    assert abs(s.loss.item() - loss) / loss < 1e-5
    assert np.allclose(s.dy.cpu().numpy(), dy, rtol=1e-5, atol=1e-9)


@pytest.mark.parametrize("name,mode", [("lm_medium", "nrrh"), ("tagger", "nr"), ("tiny", "nrrh_dense"),
                                       ("seq2seq_enc", "nrrh")])
def test_persistent_and_per_step_paths_agree(name, mode, monkeypatch):
    """The persistent recurrent kernels and the per-step kernels give the same
    step (to the bf16 bar), and the persistent kernels really run."""
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    from tests._parity import mode_rates
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0]
    p_nr, p_rh, compact = mode_rates(cfg, mode, p)
    say(f"[gpu] persistent vs per-step {name} {mode}")
    outs = []
    for flag in ("1", "0"):
        monkeypatch.setenv("LSTM_SD_PERSIST", flag)
        s = Session(wl, p_nr, p_rh, compact)
        s.masks(cfg.mask_seed, 2)
        B_.lstm_sd_kernel_timer_start("fwd_persist")
        s.forward()
        _, n = B_.lstm_sd_kernel_timer_stop()
        assert n == (fwd_persist_launches(cfg) if flag == "1" else 0)
        s.loss_grad()
        B_.lstm_sd_kernel_timer_start("bwd_persist")
        s.backward()
        _, n = B_.lstm_sd_kernel_timer_stop()
        assert n == (fwd_persist_launches(cfg) if flag == "1" else 0)
        torch.cuda.synchronize()
        outs.append(s.outputs())
    errs = compare(outs[0], outs[1])
    assert max(errs.values()) <= TOL[cfg.dtype], errs
    assert np.isfinite(outs[0]["hT"]).all()


@pytest.mark.parametrize("name,mode", [("lm_medium", "nrrh"), ("lm_medium", "nr_dense"), ("tiny", "nr"),
                                       ("seq2seq_enc", "nrrh")])
def test_stacked_and_per_layer_agree(name, mode, monkeypatch):
    """A unidirectional stack run as one persistent launch per pass (forward:
    an input-product worker per layer above the first forms its input product
    from what the layer below published, or, without workers, each layer
    forms its own; backward: a worker forms each layer's input gradient from
    the DA the layer publishes) gives the same step as one launch per layer
    with the separate input-product and input-gradient passes."""
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    from tests._parity import mode_rates
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0]
    p_nr, p_rh, compact = mode_rates(cfg, mode, p)
    say(f"[gpu] stacked vs per-layer {name} {mode}")
    outs = []
    for flag, workers in (("1", "1"), ("1", "0"), ("0", "1")):
        monkeypatch.setenv("LSTM_SD_STACK", flag)
        monkeypatch.setenv("LSTM_SD_FWD_WORKERS", workers)
        s = Session(wl, p_nr, p_rh, compact)
        s.masks(cfg.mask_seed, 4)
        B_.lstm_sd_kernel_timer_start("fwd_persist")
        s.forward()
        _, n = B_.lstm_sd_kernel_timer_stop()
        assert n == fwd_persist_launches(cfg, stacked=flag == "1")
        s.loss_grad()
        B_.lstm_sd_kernel_timer_start("bwd_persist")
        s.backward()
        _, n = B_.lstm_sd_kernel_timer_stop()
        assert n == fwd_persist_launches(cfg, stacked=flag == "1")
        torch.cuda.synchronize()
        outs.append(s.outputs())
    for o in outs[:2]:
        errs = compare(o, outs[2])
        assert max(errs.values()) <= TOL[cfg.dtype], errs
        for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
            assert np.isfinite(o[k]).all(), k


def test_mse_loss_repeated_calls():
    """Repeated loss calls on the same outputs give the same bits (a fixed
    summation order), and the loss matches the oracle's."""
    from paper_2106_12089_amd.session import Session
    cfg, wl = make("mse", loss="mse", dtype="f32", batch=19, seq_len=5)
    say("[gpu] mse repeated calls")
    s = Session(wl, 0.5, 0.0, 1)
    s.masks(cfg.mask_seed, 0)
    s.forward()
    vals = []
    for _ in range(3):
        s.loss_grad()
        torch.cuda.synchronize()
        vals.append(s.loss.item())
    assert vals[0] == vals[1] == vals[2]
    from oracle import masks as om
    m_nr, m_rh = om.all_masks(cfg.mask_seed, 0, cfg.num_layers, cfg.num_dirs, cfg.seq_len, cfg.k_in, cfg.hidden,
                              0.5, 0.0)
    ref = oracle_step(wl, 0.5, 0.0, m_nr, m_rh)
    assert abs(vals[0] - ref["loss"]) <= TOL["f32"] * abs(ref["loss"])
