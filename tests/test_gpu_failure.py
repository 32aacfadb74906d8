"""The failure path of the persistent kernels, forced from the host: with a
zero barrier time-out every grid-barrier wait gives up at once, so every
workgroup leaves through the time-out path (no kernel spins or faults).  The
step must then report the failure through lstm_sd_status, write NaN into
every output it names, and a clean step on the same buffers afterwards must
match the oracle again.  The seq2seq encoder (batch 64) takes the large-batch
input products and gradients and the GEMM weight gradient; the stress shape
(batch 256) the large-batch recurrences, whose clean step after the failure
is checked bit for bit against a fresh session's."""
import numpy as np
import pytest

import workloads
from tests._parity import TOL, compare, mode_rates, oracle_masks, oracle_step, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["lm_medium", "tagger", "seq2seq_enc"])
def test_forced_barrier_timeout_is_reported_then_recovers(name):
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = 0.5
    p_nr, p_rh, compact = mode_rates(cfg, "nrrh", p)
    s = Session(wl, p_nr, p_rh, compact)
    say(f"[gpu] forced barrier time-out {name}")
    B_.lstm_sd_set_barrier_timeout(0.0)
    try:
        s.masks(cfg.mask_seed, 0)
        s.forward()
        s.loss_grad()
        s.backward()
        with pytest.raises(B_.LstmSdError) as e:
            B_.lstm_sd_status(s.dims, s.workspace)
    finally:
        B_.lstm_sd_set_barrier_timeout(-1.0)
    assert e.value.code == B_.EHIP
    msg = str(e.value)
    assert "forward" in msg and "backward" in msg, msg
    out = s.outputs()
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        assert np.isnan(out[k]).all(), k
    for k in ("dW", "dU", "db"):
        for i, a in enumerate(out[k]):
            assert np.isnan(a).all(), (k, i)

    say(f"[gpu] clean step after the failure {name}")
    s.masks(cfg.mask_seed, 0)
    s.forward()
    s.loss_grad()
    s.backward()
    B_.lstm_sd_status(s.dims, s.workspace)          # no error now
    torch.cuda.synchronize()
    gpu = s.outputs()
    m_nr, m_rh = oracle_masks(cfg, p_nr, p_rh)
    ref = oracle_step(wl, p_nr, p_rh, m_nr, m_rh)
    errs = compare(gpu, ref)
    say("   errs max", max(errs.values()))
    bad = {k: v for k, v in errs.items() if not v <= TOL[cfg.dtype]}
    assert not bad, bad


def test_forced_barrier_timeout_large_batch_recurrences():
    from paper_2106_12089_amd import binding as B_
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config("stress")
    wl = workloads.make_workload(cfg)
    p_nr, p_rh, compact = mode_rates(cfg, "nrrh", 0.5)
    s = Session(wl, p_nr, p_rh, compact)
    say("[gpu] forced barrier time-out stress")
    B_.lstm_sd_set_barrier_timeout(0.0)
    try:
        s.masks(cfg.mask_seed, 0)
        s.forward()
        s.loss_grad()
        s.backward()
        with pytest.raises(B_.LstmSdError) as e:
            B_.lstm_sd_status(s.dims, s.workspace)
    finally:
        B_.lstm_sd_set_barrier_timeout(-1.0)
    assert e.value.code == B_.EHIP
    out = s.outputs()
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        assert np.isnan(out[k]).all(), k
    for k in ("dW", "dU", "db"):
        for i, a in enumerate(out[k]):
            assert np.isnan(a).all(), (k, i)

    say("[gpu] clean step after the failure stress")
    s.masks(cfg.mask_seed, 0)
    s.forward()
    s.loss_grad()
    s.backward()
    B_.lstm_sd_status(s.dims, s.workspace)
    torch.cuda.synchronize()
    got = s.outputs()
    f = Session(wl, p_nr, p_rh, compact)
    f.masks(cfg.mask_seed, 0)
    f.forward()
    f.loss_grad()
    f.backward()
    torch.cuda.synchronize()
    ref = f.outputs()
    for k in ("y", "hT", "cT", "dx", "dh0", "dc0"):
        assert np.array_equal(got[k], ref[k]), k
    for k in ("dW", "dU", "db"):
        for i, (a, b) in enumerate(zip(got[k], ref[k])):
            assert np.array_equal(a, b), (k, i)
