"""The Case-I ("NR+Random") comparator on the GPU against its oracle: the
per-element masks bit-exact, and the whole step (every layer's input
dropped per element, each layer run dense) normwise within the step's
tolerance, at LM-medium and on the bidirectional tagger and the seq2seq
encoder (lengths)."""
import numpy as np
import pytest

import workloads
from oracle import case1
from tests._parity import TOL, rel, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["lm_medium", "tagger", "seq2seq_enc"])
def test_case1_step(name):
    from paper_2106_12089_amd.session import Case1Session
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0]
    say(f"[gpu] case-I {name} p={p}")
    s = Case1Session(wl, p)
    s.step(cfg.mask_seed, 2)
    torch.cuda.synchronize()
    m = case1.all_element_masks(cfg.mask_seed, 2, cfg.num_layers, cfg.seq_len, cfg.batch, cfg.k_in, p)
    for l in range(cfg.num_layers):
        assert np.array_equal(s.drop_masks[l].cpu().numpy(), m[l]), l
    ref = case1.case1_step(wl.W, wl.U, wl.b, wl.x, wl.h0, wl.c0, cfg.num_layers, cfg.num_dirs, m, p, cfg.loss,
                           wl.target, wl.lengths)
    got = s.outputs()
    errs = {k: rel(got[k], ref[k]) for k in ("y", "dx")}
    errs["loss"] = abs(got["loss"] - ref["loss"]) / abs(ref["loss"])
    for k in ("dW", "dU", "db"):
        for i, (a, r) in enumerate(zip(got[k], ref[k])):
            errs[f"{k}{i}"] = rel(a, r)
    say("   max err", max(errs.values()))
    assert max(errs.values()) <= TOL[cfg.dtype], errs
