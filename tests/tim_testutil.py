"""Helpers shared by the GPU tests: seeded inputs on the GPU, oracle calls on
host copies of the same inputs, and tolerance checks that print the observed
error so the logs carry it."""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from workload import bf16_bits, hidden_states, vocab_weights

# Tolerances against the fp64 oracle (absolute, nats).
TOL_LOGP = 1e-3
TOL_ENT = 1e-3
# Relative tolerance on importance weights.
TOL_W_REL = 1e-3


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    tim.load_library()


def inputs(T, d, V, seed, w_std=None, device="cuda"):
    """bf16 hidden states (RMS-normalised) and W on the GPU, seeded."""
    if w_std is None:
        w_std = 1.0 / math.sqrt(d)
    h = hidden_states(T, d, 1000 + seed, device=device)
    W = vocab_weights(V, d, w_std, 2000 + seed, device=device)
    return h, W


def random_tokens(T, V, seed, device="cuda"):
    g = torch.Generator(device="cpu").manual_seed(5000 + seed)
    return torch.randint(0, V, (T,), generator=g, dtype=torch.int32).to(device)


def oracle_rows(h, W, tok, tau, rows=None):
    """fp64 oracle (logp, entropy) for the given row indices (all when None)."""
    if rows is None:
        hb = bf16_bits(h)
        tb = tok.cpu().numpy()
    else:
        idx = torch.as_tensor(np.asarray(rows), device=h.device, dtype=torch.long)
        hb = bf16_bits(h.index_select(0, idx))
        tb = tok.index_select(0, idx).cpu().numpy()
    return oracle.logprobs(hb, bf16_bits(W), tb, tau)


def check_close(name, got, ref, atol, rows=None):
    got = got.detach().double().cpu().numpy() if torch.is_tensor(got) else np.asarray(got, dtype=np.float64)
    if rows is not None:
        got = got[np.asarray(rows)]
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape
    both_nan = np.isnan(got) & np.isnan(ref)
    err = np.where(both_nan, 0.0, np.abs(got - ref))
    mx = float(np.nanmax(err)) if err.size else 0.0
    print(f"[parity] {name}: n={got.size} max|err|={mx:.3e} tol={atol:.0e}")
    assert not np.isnan(err).any(), f"{name}: NaN mismatch"
    assert mx <= atol, f"{name}: max error {mx} > {atol}"
    return mx


def bits_equal(a, b):
    return torch.equal(a.view(torch.int32), b.view(torch.int32))
