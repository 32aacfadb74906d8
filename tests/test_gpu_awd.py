"""The AWD-LSTM shape of Sec. 4.1 on the GPU: three layers, embedding 400,
hidden 1150, a dropout rate per site (input 0.4 on layer 0, 0.25 between
layers) and the structured form of its recurrent weight drop (0.5 on h_{t-1}
of every layer).  Masks bit-exact against the oracle; the whole step within
the bf16 bound, in the method's mode and the same kernels run dense, and in
the NR-only mode."""
import numpy as np
import pytest

import workloads
from tests._parity import TOL, compare, mode_rates, oracle_masks, oracle_step, say, summary
from tests.test_gpu_parity import check_masks

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

_WL = {}


def workload():
    if "awd" not in _WL:
        _WL["awd"] = workloads.make_workload(workloads.get_config("awd_lstm"))
    return _WL["awd"]


@pytest.mark.parametrize("mode", ["nrrh", "nrrh_dense", "nr"])
def test_awd_step_parity(mode):
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config("awd_lstm")
    wl = workload()
    p_nr, p_rh, compact = mode_rates(cfg, mode, None)
    assert p_nr == [0.4, 0.25, 0.25]
    say(f"[gpu] awd_lstm mode={mode} p_nr={p_nr} p_rh={p_rh}")
    sess = Session(wl, p_nr, p_rh, compact)
    sess.masks(cfg.mask_seed, 0)
    m_nr, m_rh = oracle_masks(cfg, p_nr, p_rh)
    torch.cuda.synchronize()
    check_masks(sess, cfg, m_nr, m_rh, compact)
    # each site dropped at its own rate
    for l in range(cfg.num_layers):
        frac = 1.0 - m_nr[l].mean()
        assert abs(frac - p_nr[l]) < 0.05, (l, frac)
    sess.forward()
    sess.loss_grad()
    sess.backward()
    torch.cuda.synchronize()
    gpu = sess.outputs()
    ref = oracle_step(wl, p_nr, p_rh, m_nr, m_rh)
    errs = compare(gpu, ref)
    errs["loss"] = abs(gpu["loss"] - ref["loss"]) / abs(ref["loss"])
    say("   errs", summary(errs))
    bad = {k: v for k, v in errs.items() if not v <= TOL[cfg.dtype]}
    assert not bad, bad
    drop = m_nr[0] == 0
    for t in range(cfg.seq_len):
        assert np.all(gpu["dx"][t][:, drop[t]] == 0.0)
