"""fp64 oracle: token-level training-inference mismatch statistics.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Given the trainer's and the rollout engine's log-probabilities of the same
sampled tokens (``logp_a`` = trainer, ``logp_b`` = rollout):

    delta  = logp_a - logp_b                   Eq. 1 (Section 2): the TIM discrepancy
    r_corr = exp(delta)                        the correction ratio pi_train / pi_rollout (Section 4.2)
    k3     = (r_corr - 1) - log r_corr         the K3 estimator (Section 4.1), written with
           = expm1(delta) - delta              log(exp(delta)) = delta substituted exactly
    w      = min(r_corr, C)                    the truncated importance weight of Eq. 6,
                                               C = tau_tok (2 in the appendix's settings)

The inputs are the fp32 arrays the GPU receives, widened to fp64.

Pins (tests/test_oracle.py): the printed log-probabilities and discrepancies
of Table 1; delta = 0 giving k3 = 0 and w = min(1, C); the literal
(r - 1) - log r form at moderate delta; the Taylor series of k3 at small
delta; w = C at delta = log C; k3 >= 0.
"""

from __future__ import annotations

import numpy as np


def mismatch(logp_a, logp_b, C: float):
    """(log_ratio, k3, is_weight) in fp64."""
    a = np.asarray(logp_a, dtype=np.float64)
    b = np.asarray(logp_b, dtype=np.float64)
    delta = a - b
    k3 = np.expm1(delta) - delta
    w = np.minimum(np.exp(delta), float(C))
    return delta, k3, w
