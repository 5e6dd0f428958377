"""fp64 oracle: log-probability and entropy of each row's next-token distribution.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed. Section 2 of the paper defines, for a context s_t and the
sampled token a_t, the token log-probability log pi(a_t | s_t) that both the
rollout engine and the trainer evaluate (the two sides of Eq. 1). In a
decoder LM that distribution is the softmax over the vocabulary of the LM-head
logits of the final hidden state, divided by the sampling temperature; the
paper does not spell this decomposition out, so the textbook definitions are
used, all in fp64:

    z_v     = (sum_k h_k * w_{v,k}) / tau                        (LM head, temperature)
    LSE     = m + log sum_v exp(z_v - m),  m = max_v z_v          (log of the softmax normaliser)
    logp    = z_{a_t} - LSE                                       (gathered log-probability)
    H       = -sum_v p_v * (z_v - LSE),  p_v = exp(z_v - LSE)     (Shannon entropy, nats)

A token id outside [0, V) has no log-probability: its logp is NaN (its entropy
is still the row's entropy).

Pins (tests/test_oracle.py): exact rational dot products on small inputs; a
uniform row (logp = -log V, H = log V); V = 1 and V = 2 closed forms
(log-sigmoid and binary entropy); scipy's log_softmax and entropy on planted
logits; probabilities summing to one over every token; entropy equal to the
expected negative log-probability; a duplicated vocabulary shifting logp and H
by log 2; a one-hot-dominant row; and temperature/scale equivalence.
"""

from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen raw bf16 bit patterns (uint16) to fp64. Exact: a bf16 value is the
    fp32 value with the same top 16 bits and zero low bits."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def logits(h_bits: np.ndarray, w_bits: np.ndarray, temperature: float,
           vocab_chunk: int = 8192) -> np.ndarray:
    """fp64 z[T, V] = (h @ W^T) / tau. The fp64 matrix product is the library
    step; W is widened one vocabulary chunk at a time to bound memory."""
    h = bf16_to_f64(h_bits)
    T, d = h.shape
    V = w_bits.shape[0]
    assert w_bits.shape == (V, d)
    z = np.empty((T, V), dtype=np.float64)
    for v0 in range(0, V, vocab_chunk):
        v1 = min(V, v0 + vocab_chunk)
        z[:, v0:v1] = h @ bf16_to_f64(w_bits[v0:v1]).T
    z /= float(temperature)
    return z


def logprobs(h_bits: np.ndarray, w_bits: np.ndarray, tokens: np.ndarray, temperature: float,
             row_block: int = 256, vocab_chunk: int = 8192):
    """(logp[T], entropy[T]) in fp64 for every row of h against the full vocabulary.

    Rows are independent; they are processed ``row_block`` at a time only to
    bound memory (each block holds its full fp64 logit matrix)."""
    h_bits = np.ascontiguousarray(h_bits, dtype=np.uint16)
    w_bits = np.ascontiguousarray(w_bits, dtype=np.uint16)
    tokens = np.asarray(tokens, dtype=np.int64)
    T = h_bits.shape[0]
    V = w_bits.shape[0]
    assert tokens.shape == (T,)
    logp = np.empty(T, dtype=np.float64)
    ent = np.empty(T, dtype=np.float64)
    for r0 in range(0, T, row_block):
        r1 = min(T, r0 + row_block)
        z = logits(h_bits[r0:r1], w_bits, temperature, vocab_chunk)
        m = z.max(axis=1, keepdims=True)
        lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
        zc = z - lse                      # log p_v
        p = np.exp(zc)
        ent[r0:r1] = -(p * zc).sum(axis=1)
        tok = tokens[r0:r1]
        ok = (tok >= 0) & (tok < V)
        rows = np.arange(r1 - r0)
        lp = np.full(r1 - r0, np.nan)
        lp[ok] = zc[rows[ok], tok[ok]]
        logp[r0:r1] = lp
    return logp, ent
