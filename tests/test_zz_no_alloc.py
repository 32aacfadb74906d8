"""lstm_sd_forward_static (the forward pass with the library's own
workspace, for callers that cannot allocate) against lstm_sd_forward with a
caller workspace: the same outputs and the same reserve, on two calls in a
row, the second on a smaller problem (the static workspace then holds the
first call's values), and a backward fed by the static call's reserve."""
import numpy as np
import pytest

import workloads
from tests._parity import TOL, compare, mode_rates, oracle_masks, oracle_step, say, summary

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(name, mode):
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p_nr, p_rh, compact = mode_rates(cfg, mode, 0.5)
    say(f"[gpu] static-workspace forward {name} {mode}")
    assert B_.lstm_sd_workspace_bytes(B_.make_dims(cfg.num_layers, cfg.input_dim, cfg.hidden, cfg.batch,
                                                   cfg.seq_len, cfg.num_dirs)) <= B_.STATIC_WORKSPACE_MAX
    a = Session(wl, p_nr, p_rh, compact)          # caller workspace
    s = Session(wl, p_nr, p_rh, compact)          # static workspace
    for x in (a, s):
        x.masks(cfg.mask_seed, 2)
    a.forward()
    B_.lstm_sd_forward_static(s.dims, s.W, s.U, s.b, s.x, s.lengths, s.h0, s.c0, s.mask_buf, s.y, s.hT, s.cT,
                              s.reserve)
    torch.cuda.synchronize()
    for k in ("y", "hT", "cT"):
        assert torch.equal(getattr(a, k), getattr(s, k)), k
    assert torch.equal(a.reserve, s.reserve), "reserve"
    # the static call's reserve feeds the backward as usual
    s.loss_grad()
    s.backward()
    torch.cuda.synchronize()
    gpu = s.outputs()
    m_nr, m_rh = oracle_masks(cfg, p_nr, p_rh, step=2)
    ref = oracle_step(wl, p_nr, p_rh, m_nr, m_rh)
    errs = compare(gpu, ref)
    say("   errs", summary(errs))
    bad = {k: v for k, v in errs.items() if not v <= TOL[cfg.dtype]}
    assert not bad, bad


def test_static_forward_two_calls_second_smaller():
    _run("lm_medium", "nrrh")    # 27.7 MiB of workspace
    _run("tiny", "nrrh")         # 0.8 MiB: the rest of the array still holds the first call's values


def test_static_forward_rejects_oversized_dims():
    from paper_2106_12089_amd import binding as B_
    cfg = workloads.get_config("stress")
    d = B_.make_dims(cfg.num_layers, cfg.input_dim, cfg.hidden, cfg.batch, cfg.seq_len, cfg.num_dirs)
    assert B_.lstm_sd_workspace_bytes(d) > B_.STATIC_WORKSPACE_MAX
    lib = B_.load()
    import ctypes
    fake = 4096   # never dereferenced: the size check fails first
    arr = (ctypes.c_void_p * 2)(fake, fake)
    w = B_.lstm_sd_weights(arr, arr, arr)
    rc = lib.lstm_sd_forward_static(ctypes.byref(d), ctypes.byref(w), *([fake] * 5), 1 << 40, fake, fake, fake,
                                    fake, 1 << 40, None)
    assert rc == B_.EUNSUPPORTED and "STATIC_WORKSPACE_MAX" in B_.lstm_sd_last_error()
