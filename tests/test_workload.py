"""The synthetic workload generators: shapes, distributions, determinism."""

import math

import numpy as np
import torch

import oracle
from workload import CONFIGS, bf16_bits, hidden_states, response_lengths, uniforms, vocab_weights
from workload.gen import seeds
from workload.sampler import sample_tokens


def test_hidden_states_rms_normalised_and_seeded():
    h = hidden_states(300, 512, seed=5)
    assert h.dtype == torch.bfloat16 and h.shape == (300, 512)
    rms = h.float().square().mean(dim=1).sqrt()
    assert torch.allclose(rms, torch.ones_like(rms), atol=1e-2)
    assert torch.equal(h, hidden_states(300, 512, seed=5))
    assert not torch.equal(h, hidden_states(300, 512, seed=6))
    # chunked generation draws the same stream as one chunk
    assert torch.equal(h, hidden_states(300, 512, seed=5, chunk=300))


def test_vocab_weights_std():
    W = vocab_weights(2000, 256, std=0.02, seed=1)
    assert W.dtype == torch.bfloat16 and W.is_contiguous()
    assert abs(W.float().std().item() - 0.02) < 5e-4
    assert abs(W.float().mean().item()) < 5e-4


def test_bf16_rne_cast():
    x = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20])
    b = x.to(torch.bfloat16).float()
    assert b.tolist() == [1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7]  # ties to even, else nearest


def test_response_lengths():
    L = response_lengths(64, 512, 4096, seed=3)
    assert L.min() >= 512 and L.max() <= 4096 and len(L) == 64
    assert (L == response_lengths(64, 512, 4096, seed=3)).all()
    assert (response_lengths(8, 16384, 16384, 5) == 16384).all()


def test_config_shapes():
    assert CONFIGS["tiny"].tokens == 64
    assert CONFIGS["long"].tokens == 131072
    assert 7000 < CONFIGS["small"].tokens < 12000
    assert 120000 < CONFIGS["mid"].tokens < 175000
    assert len({seeds(c) for c in CONFIGS.values()}) == 4  # stress reuses mid's inputs


def test_sampler_matches_distribution():
    """Inverse-CDF draws follow softmax(z / tau): chi-square over a planted row."""
    V, d, n = 8, 32, 40000
    z = np.array([0.0, 1.0, -1.0, 2.0, 0.5, -3.0, 1.5, 0.25])
    h = torch.zeros(n, d, dtype=torch.bfloat16); h[:, 0] = 1.0
    W = torch.zeros(V, d, dtype=torch.bfloat16); W[:, 0] = torch.tensor(z)
    tau = 0.7
    tok = sample_tokens(h, W, tau, uniforms(n, 9)).numpy()
    p = np.exp(z / tau - np.log(np.exp(z / tau).sum()))
    counts = np.bincount(tok, minlength=V)
    chi2 = (((counts - n * p) ** 2) / (n * p)).sum()
    assert chi2 < 30.0  # 7 dof; p < 1e-4


def test_tiny_config_sampled_tokens_are_plausible():
    cfg = CONFIGS["tiny"]
    hs, ws, us = seeds(cfg)
    h = hidden_states(cfg.tokens, cfg.d, hs)
    W = vocab_weights(cfg.V, cfg.d, cfg.w_std, ws)
    tok = sample_tokens(h, W, cfg.temperature, uniforms(cfg.tokens, us))
    assert tok.dtype == torch.int32 and int(tok.min()) >= 0 and int(tok.max()) < cfg.V
    lp, H = oracle.logprobs(bf16_bits(h), bf16_bits(W), tok.numpy(), cfg.temperature)
    # logit std is 1 here, so H ~ log V - 1/2 and E[logp of a sampled token] = -E[H]
    assert abs(H.mean() - (math.log(cfg.V) - 0.5)) < 0.15
    assert abs(lp.mean() + H.mean()) < 4 * lp.std() / math.sqrt(cfg.tokens)
