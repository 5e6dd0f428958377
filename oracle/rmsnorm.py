"""fp64 oracle: the final RMS normalisation in front of the LM head, and its gradients.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed. The batch-invariant kernels of Section 3.1 include RMSNorm
(Zhang and Sennrich's root-mean-square layer normalisation): a row a of d
values becomes a_k / RMS(a) * g_k with RMS(a) = sqrt(mean_k a_k^2), a small
eps added under the root in practice. The final norm feeds the LM head, so its
output is the hidden state the log-probabilities are taken of. The engine
follows a HuggingFace model implementation (Section 3.1), whose norm widens a
bf16 row to fp32, scales it, rounds it back to bf16 and then multiplies by the
bf16 weight, rounding again; the oracle takes the same two roundings, each
from the exact fp64 value (round to nearest, ties to even), so a GPU that
rounds from fp32 agrees except where the two straddle a rounding boundary:

    r_t    = 1 / sqrt(mean_k x_tk^2 + eps)                       (fp64)
    n_tk   = x_tk * r_t                                           (fp64, exact product)
    h_tk   = bf16(g_k * bf16(n_tk))   (or bf16(n_tk) without a weight)

Gradients, with the roundings passed straight through (as autograd treats the
casts) for a loss with upstream gradient G = dL/dh:

    dL/dx_tk = r_t g_k G_tk - r_t^3 x_tk (1/d) sum_j G_tj g_j x_tj
    dL/dg_k  = sum_t G_tk x_tk r_t

Pins (tests/test_oracle.py): the bf16 rounding against torch's fp32 -> bf16
cast, exact ties and values just off a tie; a constant row in closed form;
torch's float64 rms_norm (a library routine); central differences and float64
autograd for the gradients; the scale identity sum_k x_k dL/dx_k = 0 when
eps = 0 (the normalised row does not change with the row's scale).
"""

from __future__ import annotations

import numpy as np

from .logprobs import bf16_to_f64


def round_bf16(v: np.ndarray) -> np.ndarray:
    """fp64 values rounded to the nearest bf16 value (8 significant bits, ties
    to even), returned as fp64. Directly from fp64, with no fp32 step. Exact for
    bf16's normal range (|v| >= 2^-126); the values here are far from its ends."""
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)                       # v = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def f64_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Bit patterns (uint16) of fp64 values that are exactly bf16 values."""
    f = np.asarray(v, dtype=np.float64).astype(np.float32)
    assert np.array_equal(f.astype(np.float64), np.asarray(v, dtype=np.float64)), "not a bf16 value"
    b = f.view(np.uint32)
    assert not (b & np.uint32(0xFFFF)).any(), "not a bf16 value"
    return (b >> np.uint32(16)).astype(np.uint16)


def rmsnorm(x_bits: np.ndarray, gamma_bits: np.ndarray | None, eps: float):
    """(h bf16 bits [T, d], r fp64 [T], n fp64 [T, d]) of the final norm."""
    x = bf16_to_f64(x_bits)
    d = x.shape[1]
    r = 1.0 / np.sqrt((x * x).sum(axis=1) / d + float(eps))
    n = x * r[:, None]
    h = round_bf16(n)
    if gamma_bits is not None:
        h = round_bf16(bf16_to_f64(gamma_bits)[None, :] * h)
    return f64_to_bf16_bits(h), r, n


def rmsnorm_grads(x_bits: np.ndarray, gamma_bits: np.ndarray | None, eps: float, grad_h: np.ndarray):
    """(dL/dx fp64 [T, d], dL/dg fp64 [d]) for upstream G = dL/dh."""
    x = bf16_to_f64(x_bits)
    T, d = x.shape
    g = np.ones(d) if gamma_bits is None else bf16_to_f64(gamma_bits)
    G = np.asarray(grad_h, dtype=np.float64)
    r = 1.0 / np.sqrt((x * x).sum(axis=1) / d + float(eps))
    s = (G * g[None, :] * x).sum(axis=1)
    dx = r[:, None] * g[None, :] * G - (r ** 3 * s / d)[:, None] * x
    dg = (G * x * r[:, None]).sum(axis=0)
    return dx, dg
