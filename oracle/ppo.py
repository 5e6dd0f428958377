"""fp64 oracle: the clipped PPO/GRPO token loss, its gradient, and the
zero-centred loss contribution.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed (Section 4.1, Eqs. 2-5; the corrections of Section 4.2):

    r_t       = exp(logp_t - logp_old_t)                    PPO ratio (Eq. 3; the caller picks the
                                                            trainer's or the rollout's old log-probs)
    L_t       = -min(r_t A_t, clip(r_t, 1 - eps_low, 1 + eps_high) A_t)      (Eq. 2)
    C_t       = -(r_t - 1) A_t                              zero-centred contribution (Eq. 5)
    S_j       = sum over response j of w_t L_t              w_t: token weights, e.g. the truncated
                                                            and rejected correction weights of
                                                            Section 4.2 (1 when absent)
    L         = (1 / n) sum_j S_j                           summed over each response, averaged
                                                            over the n sampled responses
    dL/dlogp_t = (1 / n) w_t (-A_t r_t)  where the unclipped term is the minimum, else 0

The clip bounds may differ (eps_low, eps_high); the paper's Eq. 2 has one eps.
clipped_t marks tokens whose loss is the clipped term strictly (zero
gradient): A_t > 0 with r_t > 1 + eps_high, or A_t < 0 with r_t < 1 - eps_low.

Pins (tests/test_oracle.py): torch autograd in float64 through the textbook
loss (clamp, minimum, exp); closed forms at r = 1 and A = 0; C's gradient
equal to that of -r A and C(1) = 0; the batch loss the mean of the response
sums; the clip regions by sign of A.
"""

from __future__ import annotations

import math

import numpy as np


def ppo_loss(logp, logp_old, advantages, cu_seqlens, eps_low: float, eps_high: float, weight=None):
    """dict of fp64 arrays: token_loss [T] (w_t L_t), grad [T] (dL/dlogp_t),
    contribution [T] (C_t), clipped bool [T], seq_loss [n] (S_j), batch_loss
    (L). Tokens outside every response have zero token outputs."""
    lp = np.asarray(logp, dtype=np.float64)
    lo = np.asarray(logp_old, dtype=np.float64)
    A = np.asarray(advantages, dtype=np.float64)
    w = np.ones_like(lp) if weight is None else np.asarray(weight, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    n = len(cu) - 1
    T = lp.shape[0]
    r = np.exp(lp - lo)
    clip_r = np.clip(r, 1.0 - eps_low, 1.0 + eps_high)
    unclipped = r * A
    clipped_term = clip_r * A
    L = -np.minimum(unclipped, clipped_term)
    use_unclipped = unclipped <= clipped_term
    grad_tok = np.where(use_unclipped, -A * r, 0.0)
    clipped = ~use_unclipped
    C = -(r - 1.0) * A
    token_loss = np.zeros(T)
    grad = np.zeros(T)
    contrib = np.zeros(T)
    clip_mask = np.zeros(T, dtype=bool)
    seq = np.zeros(n)
    for j in range(n):
        s0, s1 = int(cu[j]), int(cu[j + 1])
        token_loss[s0:s1] = w[s0:s1] * L[s0:s1]
        grad[s0:s1] = w[s0:s1] * grad_tok[s0:s1] / n
        contrib[s0:s1] = C[s0:s1]
        clip_mask[s0:s1] = clipped[s0:s1]
        seq[j] = math.fsum(token_loss[s0:s1].tolist())
    batch = math.fsum(seq.tolist()) / n if n > 0 else 0.0
    return {"token_loss": token_loss, "grad": grad, "contribution": contrib, "clipped": clip_mask,
            "seq_loss": seq, "batch_loss": batch}
