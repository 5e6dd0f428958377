"""fp64 oracle: gradients of the token log-probability and entropy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed. The trainer differentiates the same per-token quantities
whose forward values the rollout engine and the trainer must agree on
(Section 2, the two sides of Eq. 1; the PPO/GRPO objectives of Section 4 use
log pi_train through the ratio). For upstream gradients g_t = dL/dlogp_t and
e_t = dL/dH_t of a scalar loss L, with the forward of oracle.logprobs,

    z_v   = (h . w_v) / tau,   lse = log sum_v exp(z_v),   q_v = z_v - lse = log p_v
    logp  = q_a                         (a = the row's token)
    H     = -sum_v p_v q_v

the chain rule gives, per row (the softmax Jacobian is diag(p) - p p^T):

    dlogp/dz_v =  [v = a] - p_v
    dH/dz_v    = -p_v (q_v + H)
    dz_v       =  g_t ([v = a] - p_v) - e_t p_v (q_v + H)
    dacc_v     =  dz_v / tau            (z = acc / tau, acc = h . w_v)
    dh         =  sum_v dacc_v w_v      (dL/dh_t,  [T, d])
    dW_v       =  sum_t dacc_{t,v} h_t  (dL/dw_v,  [V, d])

A row whose token is outside [0, V) has no log-probability; its logp term
contributes nothing (only e_t's entropy term, if any).

Pins (tests/test_oracle.py): central finite differences of the pinned forward
oracle; torch's autograd in float64 through the textbook forward; the softmax
gradient summing to zero over the vocabulary (so the columns of dW sum to zero
and dh ignores a common shift of every w_v); the uniform row (h = 0) in closed
form; the two-token vocabulary (logistic) in closed form; linearity in (g, e).
"""

from __future__ import annotations

import numpy as np

from .logprobs import bf16_to_f64, logits


def logit_grads(h_bits: np.ndarray, w_bits: np.ndarray, tokens: np.ndarray, temperature: float,
                grad_logp: np.ndarray, grad_entropy: np.ndarray | None = None,
                row_block: int = 256, vocab_chunk: int = 8192) -> np.ndarray:
    """dacc[T, V] = dL/d(h . w_v) in fp64: the gradient with respect to the
    untempered LM-head contraction of every row. Rows are independent; they are
    processed ``row_block`` at a time only to bound memory."""
    h_bits = np.ascontiguousarray(h_bits, dtype=np.uint16)
    w_bits = np.ascontiguousarray(w_bits, dtype=np.uint16)
    tokens = np.asarray(tokens, dtype=np.int64)
    T = h_bits.shape[0]
    V = w_bits.shape[0]
    g = np.asarray(grad_logp, dtype=np.float64)
    e = np.zeros(T) if grad_entropy is None else np.asarray(grad_entropy, dtype=np.float64)
    assert tokens.shape == (T,) and g.shape == (T,) and e.shape == (T,)
    dacc = np.empty((T, V), dtype=np.float64)
    for r0 in range(0, T, row_block):
        r1 = min(T, r0 + row_block)
        z = logits(h_bits[r0:r1], w_bits, temperature, vocab_chunk)
        m = z.max(axis=1, keepdims=True)
        lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
        q = z - lse
        p = np.exp(q)
        H = -(p * q).sum(axis=1, keepdims=True)
        tok = tokens[r0:r1]
        ok = (tok >= 0) & (tok < V)
        gb = np.where(ok, g[r0:r1], 0.0)[:, None]
        onehot = np.zeros_like(p)
        rows = np.arange(r1 - r0)
        onehot[rows[ok], tok[ok]] = 1.0
        dz = gb * (onehot - p) - e[r0:r1, None] * p * (q + H)
        dacc[r0:r1] = dz / float(temperature)
    return dacc


def logprob_grads(h_bits: np.ndarray, w_bits: np.ndarray, tokens: np.ndarray, temperature: float,
                  grad_logp: np.ndarray, grad_entropy: np.ndarray | None = None):
    """(dh[T, d], dW[V, d]) in fp64 for L = sum_t g_t logp_t + e_t H_t.
    The fp64 matrix products are the library steps."""
    dacc = logit_grads(h_bits, w_bits, tokens, temperature, grad_logp, grad_entropy)
    h = bf16_to_f64(h_bits)
    w = bf16_to_f64(w_bits)
    dh = dacc @ w
    dw = dacc.T @ h
    return dh, dw
