"""The language-model output head on the GPU (through the C ABI) against the
float64 oracle: output-site masks bit-exact; logits, loss and every gradient
normwise within the step's tolerance, for the head alone on seeded inputs
and for the whole LM step (LSTM forward, head, LSTM backward fed by the
head's dy) at LM-medium; ragged f32 shapes in compact and dense mode with
padded rows and ignored targets; the degenerate cases (every feature dropped
at some t, no row that counts)."""
import types

import numpy as np
import pytest

import workloads
from oracle import head, lstm, masks
from tests._parity import TOL, oracle_masks, rel, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _head(wl, p, compact, seed, step=0):
    from paper_2106_12089_amd.session import HeadSession
    h = HeadSession(wl, p, compact)
    h.masks(seed, step)
    return h


def _out_mask(cfg, F, p, step=0, T=None):
    return masks.keep_mask(cfg.mask_seed, step, masks.out_stream(cfg.num_layers), T or cfg.seq_len, F, p)


def _check(got, ref, tol, keys=("z", "dy", "dW", "dc")):
    errs = {k: rel(got[k], ref[k]) for k in keys}
    errs["loss"] = abs(got["loss"] - ref["loss"]) / max(abs(ref["loss"]), 1e-30)
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    assert max(errs.values()) <= tol, errs


def _synthetic(name, T, B, F, V, dtype="f32", lengths=None, seed=0, L=1):
    cfg = types.SimpleNamespace(name=name, dtype=dtype, num_layers=L, seq_len=T, mask_seed=seed + 11)
    rng = np.random.default_rng(seed)
    q = workloads.round_to_bf16 if dtype == "bf16" else (lambda a: np.asarray(a, np.float32))
    wl = types.SimpleNamespace(
        cfg=cfg, x=np.zeros((T, B, 1), np.float32), lengths=lengths,
        W_fc=q(rng.uniform(-0.3, 0.3, size=(F, V)).astype(np.float32)),
        b_fc=rng.uniform(-0.1, 0.1, size=(V,)).astype(np.float32),
        targets=rng.integers(0, V, size=(T, B)).astype(np.int32))
    y = q(rng.normal(0.0, 1.0, size=(T, B, F)).astype(np.float32))
    return cfg, wl, y


def _run_head(cfg, wl, y, p, compact):
    h = _head(wl, p, compact, cfg.mask_seed)
    h.forward(torch.from_numpy(y).cuda())
    h.backward()
    torch.cuda.synchronize()
    F = wl.W_fc.shape[0]
    m = _out_mask(cfg, F, p)
    if compact:
        assert np.array_equal(h.mask_view(), m)
    ref = head.head_step(y, wl.W_fc, wl.b_fc, m, p, wl.targets, wl.lengths)
    return h.outputs(), ref, m


@pytest.mark.parametrize("name,compact", [("lm_medium", 1), ("lm_medium", 0), ("lm_large", 1),
                                          ("seq2seq_enc", 1)])
def test_head_alone(name, compact):
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0]
    say(f"[gpu] head {name} alone compact={compact} p={p}")
    F = cfg.num_dirs * cfg.hidden
    y = workloads.round_to_bf16(np.random.default_rng(5).normal(0, 0.5, size=(cfg.seq_len, cfg.batch,
                                                                             F)).astype(np.float32))
    got, ref, m = _run_head(cfg, wl, y, p, compact)
    _check(got, ref, TOL["bf16"])
    never = m.sum(axis=0) == 0
    assert not got["dW"][never].any()
    assert not (got["dy"] * (1 - m[:, None, :])).any()


def test_lm_medium_full_step():
    """LSTM forward -> head -> LSTM backward with the head's dy, against the
    oracle's chain on the same masks (NR+ST, p = 0.5 at both sites)."""
    from paper_2106_12089_amd.session import Session
    cfg = workloads.get_config("lm_medium")
    wl = workloads.make_workload(cfg)
    say("[gpu] head lm_medium full step")
    s = Session(wl, 0.5, 0.0, 1)
    s.masks(cfg.mask_seed, 0)
    s.forward()
    h = _head(wl, 0.5, 1, cfg.mask_seed)
    h.forward(s.y)
    h.backward()
    s.backward(dy=h.dy)
    torch.cuda.synchronize()
    m_nr, m_rh = oracle_masks(cfg, 0.5, 0.0)
    P = lstm.params_from(wl.W, wl.U, wl.b, cfg.num_layers, cfg.num_dirs)
    y, _, _, cache = lstm.forward(P, wl.x, wl.h0, wl.c0, m_nr, m_rh, 0.5, 0.0, wl.lengths)
    m = _out_mask(cfg, cfg.hidden, 0.5)
    hs = head.head_step(y, wl.W_fc, wl.b_fc, m, 0.5, wl.targets, wl.lengths)
    g = lstm.backward(cache, hs["dy"])
    _check(h.outputs(), hs, TOL["bf16"])
    gpu = s.outputs()
    errs = {"dx": rel(gpu["dx"], g["dx"])}
    for k in ("dW", "dU", "db"):
        for i, (a, r) in enumerate(zip(gpu[k], g[k])):
            errs[f"{k}{i}"] = rel(a, r)
    say("   lstm errs", {k: f"{v:.2e}" for k, v in errs.items()})
    assert max(errs.values()) <= TOL["bf16"], errs


@pytest.mark.parametrize("compact", [1, 0])
@pytest.mark.parametrize("shape", [
    dict(T=3, B=19, F=37, V=52),
    dict(T=2, B=1, F=5, V=4),
    dict(T=4, B=35, F=70, V=260),
    dict(T=2, B=70, F=129, V=1000),
])
def test_ragged_f32(shape, compact):
    T, B = shape["T"], shape["B"]
    lengths = np.random.default_rng(1).integers(0, T + 1, size=(B,)).astype(np.int32)
    cfg, wl, y = _synthetic("ragged", lengths=lengths, seed=2, **shape)
    wl.targets[0, 0] = -1                     # ignored
    say(f"[gpu] head ragged {shape} compact={compact}")
    got, ref, _ = _run_head(cfg, wl, y, 0.4, compact)
    _check(got, ref, TOL["f32"])


def test_bf16_ragged_and_p0():
    cfg, wl, y = _synthetic("bf16", T=3, B=21, F=66, V=132, dtype="bf16", seed=3)
    say("[gpu] head bf16 ragged p=0.3 and p=0")
    got, ref, _ = _run_head(cfg, wl, y, 0.3, 1)
    _check(got, ref, TOL["bf16"])
    got, ref, _ = _run_head(cfg, wl, y, 0.0, 1)
    _check(got, ref, TOL["bf16"])


def test_every_feature_dropped_at_some_t():
    cfg, wl, y = _synthetic("alldrop", T=8, B=5, F=3, V=8, seed=4)
    m = _out_mask(cfg, 3, 0.9)
    assert (m.sum(axis=1) == 0).any()         # the case is exercised
    say("[gpu] head all features dropped at some t")
    got, ref, _ = _run_head(cfg, wl, y, 0.9, 1)
    _check(got, ref, TOL["f32"])


def test_no_row_counts():
    cfg, wl, y = _synthetic("norow", T=3, B=4, F=16, V=32, seed=5)
    wl.targets[:] = 32                        # every target outside [0, V)
    say("[gpu] head no counting row")
    got, ref, _ = _run_head(cfg, wl, y, 0.5, 1)
    assert got["loss"] == 0.0
    assert not got["dy"].any() and not got["dW"].any() and not got["dc"].any()
    assert rel(got["z"], ref["z"]) <= TOL["f32"]


def test_repeat_is_deterministic():
    cfg, wl, y = _synthetic("repeat", T=3, B=19, F=37, V=52, seed=6)
    outs = []
    for _ in range(2):
        h = _head(wl, 0.4, 1, cfg.mask_seed)
        h.forward(torch.from_numpy(y).cuda())
        h.backward()
        torch.cuda.synchronize()
        outs.append(h.outputs())
    for k in ("z", "dy", "dW", "dc"):
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert outs[0]["loss"] == outs[1]["loss"]


def test_bidirectional_stack_with_head():
    """The head on a bidirectional stack's output (F = 2H, the tagger's shape
    with a synthetic FC layer and targets), chained through the LSTM
    backward, against the oracle chain (NR+RH+ST at the stack, p_out = 0.5)."""
    from paper_2106_12089_amd.session import HeadSession, Session
    cfg = workloads.get_config("tagger")
    wl = workloads.make_workload(cfg)
    F, V, p = cfg.num_dirs * cfg.hidden, 96, 0.5
    rng = np.random.default_rng(8)
    wl.W_fc = workloads.round_to_bf16(rng.uniform(-0.1, 0.1, size=(F, V)).astype(np.float32))
    wl.b_fc = rng.uniform(-0.1, 0.1, size=(V,)).astype(np.float32)
    wl.targets = rng.integers(0, V, size=(cfg.seq_len, cfg.batch)).astype(np.int32)
    say("[gpu] head on the bidirectional tagger stack")
    s = Session(wl, p, p, 1)
    s.masks(cfg.mask_seed, 0)
    s.forward()
    h = HeadSession(wl, p, 1)
    h.masks(cfg.mask_seed, 0)
    h.forward(s.y)
    h.backward()
    s.backward(dy=h.dy)
    torch.cuda.synchronize()
    m_nr, m_rh = oracle_masks(cfg, p, p)
    P = lstm.params_from(wl.W, wl.U, wl.b, cfg.num_layers, cfg.num_dirs)
    y, _, _, cache = lstm.forward(P, wl.x, wl.h0, wl.c0, m_nr, m_rh, p, p, wl.lengths)
    m = _out_mask(cfg, F, p)
    assert np.array_equal(h.mask_view(), m)
    hs = head.head_step(y, wl.W_fc, wl.b_fc, m, p, wl.targets, wl.lengths)
    g = lstm.backward(cache, hs["dy"])
    _check(h.outputs(), hs, TOL["bf16"])
    gpu = s.outputs()
    errs = {"dx": rel(gpu["dx"], g["dx"])}
    for k in ("dW", "dU", "db"):
        for i, (a, r) in enumerate(zip(gpu[k], g[k])):
            errs[f"{k}{i}"] = rel(a, r)
    say("   lstm errs", {k: f"{v:.2e}" for k, v in errs.items()})
    assert max(errs.values()) <= TOL["bf16"], errs
