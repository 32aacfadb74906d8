"""The embedding-table gradient on the GPU (through the C ABI) against the
float64 oracle.

Full-size LM-medium step: the GPU's d_emb (from its own dx) against the
oracle's (from the oracle's dx), normwise within the step's tolerance.
Kernel-level cases on a seeded host dx (drawn here, not by the HIP path):
every row against the oracle within fp32 summation error, accumulation into
an existing gradient, tokens outside the table, one token everywhere, a
vocabulary that is not a multiple of the workgroup's token range, more
positions than one chunk, and bit-identical repeats."""
import dataclasses

import numpy as np
import pytest

import workloads
from oracle import embedding
from tests._parity import TOL, oracle_masks, oracle_step, rel, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _session(cfg, wl, p_nr, p_rh, compact=1):
    from paper_2106_12089_amd.session import Session
    s = Session(wl, p_nr, p_rh, compact)
    s.masks(cfg.mask_seed, 0)
    return s


@pytest.mark.parametrize("name,p_rh,compact", [("lm_medium", 0.0, 1), ("lm_medium", 0.5, 1), ("lm_medium", 0.5, 0),
                                               ("lm_large", 0.0, 1), ("seq2seq_enc", 0.0, 1)])
def test_step(name, p_rh, compact):
    cfg = workloads.get_config(name)
    wl = workloads.make_workload(cfg)
    p = cfg.p_values[0]
    p_rh = p if p_rh else 0.0
    say(f"[gpu] embedding {name} p={p} p_rh={p_rh} compact={compact}")
    s = _session(cfg, wl, p, p_rh, compact)
    s.forward()
    s.loss_grad()
    s.backward()
    tok = torch.from_numpy(wl.tokens).cuda()
    d = s.embedding_backward(tok, cfg.vocab)
    torch.cuda.synchronize()
    m_nr, m_rh = oracle_masks(cfg, p, p_rh)
    ref = oracle_step(wl, p, p_rh, m_nr, m_rh)
    want = embedding.embedding_grad(wl.tokens, ref["dx"], m_nr[0], np.zeros((cfg.vocab, cfg.input_dim)))
    err = rel(d.cpu().numpy(), want)
    say("   rel err", err)
    assert err <= TOL[cfg.dtype]
    # rows of tokens that never occur are untouched (zero here)
    seen = np.zeros(cfg.vocab, bool)
    seen[wl.tokens.ravel()] = True
    assert not d.cpu().numpy()[~seen].any()


def _kernel_case(T, B, I, V, tokens, seed=0, p=0.5, base=None):
    cfg = dataclasses.replace(workloads.get_config("tiny"), name="emb", num_layers=1, num_dirs=1, input_dim=I,
                              hidden=8, batch=B, seq_len=T, dtype="f32")
    wl = workloads.make_workload(cfg)
    s = _session(cfg, wl, p, 0.0)
    m_nr, _ = oracle_masks(cfg, p, 0.0)
    rng = np.random.default_rng(seed)
    dx = (rng.normal(size=(T, B, I)) * m_nr[0][:, None, :]).astype(np.float32)   # zero in dropped columns
    d0 = np.zeros((V, I), np.float32) if base is None else base.astype(np.float32)
    d = torch.from_numpy(d0.copy()).cuda()
    from paper_2106_12089_amd import binding as B_
    B_.lstm_sd_embedding_backward(s.dims, torch.from_numpy(tokens.astype(np.int32)).cuda(), V,
                                  torch.from_numpy(dx).cuda(), s.mask_buf, d)
    torch.cuda.synchronize()
    want = embedding.embedding_grad(tokens, dx.astype(np.float64), m_nr[0], d0.astype(np.float64))
    return d.cpu().numpy(), want, s, dx


def _close(got, want):
    # fp32 sums of at most a few thousand terms of unit size
    assert np.allclose(got, want, rtol=1e-5, atol=1e-4), float(np.abs(got - want).max())


def test_kernel_zipf_tokens_and_accumulation():
    T, B, I, V = 6, 5, 70, 300
    rng = np.random.default_rng(1)
    tok = rng.integers(0, V, size=(T, B))
    tok[:, 0] = 7                              # a hot row
    base = np.random.default_rng(2).normal(size=(V, I))
    got, want, _, _ = _kernel_case(T, B, I, V, tok, base=base)
    _close(got, want)


def test_kernel_out_of_range_one_token_and_ragged_vocab():
    T, B, I = 4, 3, 33
    tok = np.full((T, B), 5)
    tok[0, 0] = -3
    tok[1, 2] = 1000
    got, want, _, _ = _kernel_case(T, B, I, 67, tok, seed=3)
    _close(got, want)


def test_kernel_many_positions_and_repeats():
    T, B, I, V = 50, 100, 24, 130              # 5000 positions: three chunks
    rng = np.random.default_rng(4)
    tok = rng.integers(0, V, size=(T, B))
    got, want, s, dx = _kernel_case(T, B, I, V, tok, seed=5)
    _close(got, want)
    from paper_2106_12089_amd import binding as B_
    outs = []
    for _ in range(2):
        d = torch.zeros(V, I, dtype=torch.float32, device="cuda")
        B_.lstm_sd_embedding_backward(s.dims, torch.from_numpy(tok.astype(np.int32)).cuda(), V,
                                      torch.from_numpy(dx).cuda(), s.mask_buf, d)
        torch.cuda.synchronize()
        outs.append(d.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])


def test_errors():
    from paper_2106_12089_amd import binding as B_
    cfg = workloads.get_config("tiny")
    wl = workloads.make_workload(cfg)
    s = _session(cfg, wl, 0.5, 0.0)
    tok = torch.zeros(cfg.seq_len, cfg.batch, dtype=torch.int32, device="cuda")
    d = torch.zeros(4, cfg.input_dim, dtype=torch.float32, device="cuda")
    with pytest.raises(B_.LstmSdError):
        B_.lstm_sd_embedding_backward(s.dims, tok, 0, s.dx, s.mask_buf, d)
    with pytest.raises(B_.LstmSdError):
        B_.lstm_sd_embedding_backward(s.dims, tok, 4, s.dx, s.mask_buf[:8], d)
