"""Token draws for the synthetic workloads: the rollout engine's part.

In the paper's setting each token a_t is drawn by the rollout engine from its
next-token distribution (Section 2). The synthetic workloads do the same: row
i's token is drawn by inverse CDF, with that row's U[0, 1) uniform, from the
softmax of (h_i . w_v) / tau over the vocabulary. This module only produces
token ids; the logits it forms here are dropped and are never an input to the
oracle or to the GPU path, both of which recompute everything from h, W and
the token ids.

The draw runs in fp64 on the CPU for small workloads and in fp32 on a GPU for
the large ones (fp32 logits of the bf16 inputs, a tiny perturbation of the
distribution that does not matter for a workload).
"""

from __future__ import annotations

import numpy as np
import torch


def sample_tokens(h: torch.Tensor, W: torch.Tensor, temperature: float, u: np.ndarray,
                  dtype=torch.float64, row_chunk: int = 1024, vocab_chunk: int = 32768) -> torch.Tensor:
    """int32 [T] token ids on h's device, one inverse-CDF draw per row."""
    T, d = h.shape
    V = W.shape[0]
    dev = h.device
    out = torch.empty(T, dtype=torch.int32, device=dev)
    u_t = torch.as_tensor(np.asarray(u, dtype=np.float64), device=dev)
    Wd = W.to(dtype)
    for r0 in range(0, T, row_chunk):
        r1 = min(T, r0 + row_chunk)
        hb = h[r0:r1].to(dtype)
        z = torch.empty((r1 - r0, V), dtype=dtype, device=dev)
        for v0 in range(0, V, vocab_chunk):
            v1 = min(V, v0 + vocab_chunk)
            z[:, v0:v1] = torch.nn.functional.linear(hb, Wd[v0:v1])
        z /= temperature
        z -= z.max(dim=1, keepdim=True).values
        p = torch.exp(z)
        del z
        cdf = torch.cumsum(p, dim=1)
        del p
        target = (u_t[r0:r1].to(dtype) * cdf[:, -1]).unsqueeze(1)
        idx = torch.searchsorted(cdf, target, right=True).squeeze(1)
        out[r0:r1] = idx.clamp_(max=V - 1).to(torch.int32)
    return out
