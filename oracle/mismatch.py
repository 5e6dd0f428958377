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

Sequence level (``mismatch_seq``), for a packed stream of responses
[cu[j], cu[j+1]):

    S_j    = sum over response j of K(r_corr,t)   the sequence score of Section 4.2,
             K1(r) = -log r = -delta, K3 as above  with the Section 4.1 estimators
    keep_j = 1[S_j <= tau_seq]                     sequence-level rejection (Section 4.2;
                                                   tau_seq = 0.001 in the appendix)
    wt_t   = keep_j * min(r_corr,t, C)             the per-token coefficient of the PPO term
                                                   in the appendix's tis-srs objectives

Sums are exactly rounded (math.fsum).

Pins (tests/test_oracle.py): the printed log-probabilities and discrepancies
of Table 1; delta = 0 giving k3 = 0 and w = min(1, C); the literal
(r - 1) - log r form at moderate delta; the Taylor series of k3 at small
delta; w = C at delta = log C; k3 >= 0. Sequence level: a constant-delta
response scores L * K(delta); K1 scores telescope to sum(b) - sum(a); identical
inputs score exactly 0; empty responses score 0; the <= boundary of keep; a
brute-force token-by-token accumulation on small random streams; permuting
the responses permutes the scores.
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


def mismatch_seq(logp_a, logp_b, cu_seqlens, estimator: str, C: float, tau_seq: float):
    """(score fp64 [n], keep bool [n], weight fp64 [T]) of the n responses
    [cu_seqlens[j], cu_seqlens[j + 1]) of a packed stream; estimator "k1" or "k3".
    Tokens outside every response get weight 0."""
    import math

    if estimator not in ("k1", "k3"):
        raise ValueError(estimator)
    a = np.asarray(logp_a, dtype=np.float64)
    b = np.asarray(logp_b, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    delta = a - b
    per_token = -delta if estimator == "k1" else np.expm1(delta) - delta
    n = len(cu) - 1
    score = np.zeros(n, dtype=np.float64)
    keep = np.zeros(n, dtype=bool)
    weight = np.zeros(len(a), dtype=np.float64)
    for j in range(n):
        s0, s1 = int(cu[j]), int(cu[j + 1])
        score[j] = math.fsum(per_token[s0:s1].tolist())
        keep[j] = bool(score[j] <= tau_seq)
        if keep[j]:
            weight[s0:s1] = np.minimum(np.exp(delta[s0:s1]), float(C))
    return score, keep, weight
