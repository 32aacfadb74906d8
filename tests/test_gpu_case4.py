"""Case-IV masks (one draw per site for the whole sequence) on the GPU: the
masks and keep lists bit-exact against the oracle, and whole training steps
with them against the oracle (LM-medium NR+RH+ST, and the bidirectional
tagger)."""
import numpy as np
import pytest

import workloads
from oracle import masks as om
from tests._parity import TOL, compare, oracle_step, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["lm_medium", "tagger"])
def test_fixed_masks_step(name):
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = 0.5
    say(f"[gpu] case-IV {name} p={p}")
    s = Session(wl, p, p, 1)
    s.masks(cfg.mask_seed, 3, fixed=True)
    m_nr, m_rh = om.all_masks(cfg.mask_seed, 3, cfg.num_layers, cfg.num_dirs, cfg.seq_len, cfg.k_in, cfg.hidden,
                              p, p, fixed=True)
    mask, keep, pos, count, drop, dcount = s.mask_views()
    sites = list(m_nr) + [m_rh[l][d] for l in range(cfg.num_layers) for d in range(cfg.num_dirs)]
    for i, m in enumerate(sites):
        K = m.shape[1]
        assert np.array_equal(mask[i, :, :K], m), i
        for t in range(cfg.seq_len):
            kl = np.nonzero(m[t])[0]
            assert count[i, t] == len(kl) and np.array_equal(keep[i, t, :len(kl)], kl)
    s.forward()
    s.loss_grad()
    s.backward()
    torch.cuda.synchronize()
    errs = compare(s.outputs(), oracle_step(wl, p, p, m_nr, m_rh))
    say("   max err", max(errs.values()))
    assert max(errs.values()) <= TOL[cfg.dtype], errs
