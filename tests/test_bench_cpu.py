"""Work accounting of bench.py (host only): the FLOP and byte formulas on
dense keep counts against their closed forms, and the one-GPU guard."""
import numpy as np

import bench
import workloads


def test_dense_flops_closed_form():
    for name in ("lm_medium", "tagger", "awd_lstm"):
        cfg = workloads.get_config(name)
        L, D, H, T, B = cfg.num_layers, cfg.num_dirs, cfg.hidden, cfg.seq_len, cfg.batch
        want = sum(3 * 2 * B * 4 * H * (cfg.k_in(l) + H) * T * D for l in range(L))
        assert bench.algorithmic_flops(bench.dense_counts(cfg), cfg) == want


def test_flops_count_valid_rows_only():
    cfg = workloads.get_config("seq2seq_enc")
    lengths = np.full(cfg.batch, cfg.seq_len)
    lengths[:10] = 20
    full = bench.algorithmic_flops(bench.dense_counts(cfg), cfg)
    part = bench.algorithmic_flops(bench.dense_counts(cfg), cfg, lengths)
    frac = (np.minimum(np.arange(cfg.seq_len)[:, None] < lengths[None, :], 1).sum()) / (cfg.seq_len * cfg.batch)
    assert abs(part / full - frac) < 1e-12


def test_recurrent_u_bytes():
    cfg = workloads.get_config("lm_medium")
    L, H, T = cfg.num_layers, cfg.hidden, cfg.seq_len
    assert bench.recurrent_u_bytes(bench.dense_counts(cfg), cfg) == L * T * H * 4 * H * 2
    c = [np.full(T, cfg.k_in(l)) for l in range(L)] + [np.full(T, H // 2)] * L
    assert bench.recurrent_u_bytes(c, cfg) == L * T * (H // 2) * 4 * H * 2


def test_rates_per_layer():
    cfg = workloads.get_config("awd_lstm")
    assert bench.rates(cfg, 0.4, False) == ([0.4, 0.25, 0.25], 0.0)
    assert bench.rates(cfg, 0.4, True) == ([0.4, 0.25, 0.25], [0.5, 0.5, 0.5])
    cfg = workloads.get_config("tagger")
    assert bench.rates(cfg, 0.3, True) == (0.3, 0.3)


def test_one_gpu_only():
    assert bench.main(["--gpus", "2"]) == 2
