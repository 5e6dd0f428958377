"""Seeded generators for hidden states, LM-head weights and sampling uniforms.

The paper's measurements use real hidden states of Qwen3 models on RL math
data (Section 3.2, Section 4, Table 2); none of that is available here, so
every input is synthetic, with the shapes of those workloads:

* hidden states: fp32 N(0, 1) per element, normalised per row to unit RMS
  (x / sqrt(mean(x^2) + 1e-6)), then one round-to-nearest-even cast to bf16;
* LM-head weights W[V, d]: fp32 N(0, std^2), one RNE cast to bf16, with
  std = 0.02 (the usual initialiser range) or std = d^-1/2;
* response lengths: integers uniform in [lo, hi], packed back to back;
* sampling uniforms: one U[0, 1) draw per row, consumed by the token sampler.

Generators are ``torch.Generator`` objects seeded per tensor, on the device
the tensor is made on (mt19937 on the CPU, Philox on a GPU), so a seed names
a tensor on one kind of device. Each caller draws its inputs once and hands
the same tensors to both the oracle and the GPU path.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    """One synthetic workload: sizes, value distribution and batching."""

    name: str
    d: int
    V: int
    n_responses: int
    len_lo: int
    len_hi: int
    w_std: float          # std of W entries before the bf16 cast
    temperature: float
    seed: int
    micro_batch: int      # tokens per training-mode launch (0 = all)
    rollout_batch: int    # decode-step batch size used for the rollout pass (0 = none)
    oracle_rows: int      # rows the oracle checks (0 = all)

    def lengths(self) -> np.ndarray:
        return response_lengths(self.n_responses, self.len_lo, self.len_hi, self.seed)

    @property
    def tokens(self) -> int:
        return int(self.lengths().sum())


def response_lengths(n: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """n integer lengths, uniform in [lo, hi] (inclusive), seeded."""
    if lo == hi:
        return np.full(n, lo, dtype=np.int64)
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=n, dtype=np.int64)


def _generator(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def hidden_states(T: int, d: int, seed: int, device="cpu", chunk: int = 16384) -> torch.Tensor:
    """bf16 [T, d]: N(0,1) per element, RMS-normalised per row (eps 1e-6), RNE to bf16."""
    g = _generator(seed, device)
    out = torch.empty((T, d), dtype=torch.bfloat16, device=device)
    for r0 in range(0, T, chunk):
        r1 = min(T, r0 + chunk)
        x = torch.randn((r1 - r0, d), generator=g, dtype=torch.float32, device=device)
        x = x * torch.rsqrt(x.square().mean(dim=1, keepdim=True) + 1e-6)
        out[r0:r1] = x.to(torch.bfloat16)
    return out


def vocab_weights(V: int, d: int, std: float, seed: int, device="cpu", chunk: int = 16384) -> torch.Tensor:
    """bf16 [V, d] row-major (vocab-major, the nn.Linear layout): N(0, std^2), RNE to bf16."""
    g = _generator(seed, device)
    out = torch.empty((V, d), dtype=torch.bfloat16, device=device)
    for r0 in range(0, V, chunk):
        r1 = min(V, r0 + chunk)
        x = torch.randn((r1 - r0, d), generator=g, dtype=torch.float32, device=device)
        out[r0:r1] = (x * std).to(torch.bfloat16)
    return out


def uniforms(T: int, seed: int) -> np.ndarray:
    """fp64 [T] uniforms in [0, 1), one per row, for inverse-CDF token sampling."""
    return np.random.default_rng(seed).random(T)


def logprob_pairs(T: int, seed: int, tail: float = 0.01, scale: float = 1e-5):
    """Two fp32 log-probability streams of the same T tokens, as a trainer and a
    rollout engine would report them: b ~ -Exp(mean 2), and a = b plus mostly
    tiny discrepancies (std `scale`) with a heavy tail of std 0.3 on a fraction
    `tail` of the tokens (the shape of the mismatch the paper measures)."""
    rng = np.random.default_rng(seed)
    b = (-rng.exponential(2.0, T)).astype(np.float32)
    a = (b + rng.standard_normal(T) * np.where(rng.random(T) < tail, 0.3, scale)).astype(np.float32)
    return a, b


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a CPU or GPU tensor, as a host uint16 array."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


# Seeds: a configuration k draws hidden states from seed 1000 + k, weights from
# seed 2000 + k and uniforms from seed 3000 + k.
CONFIGS = {
    "tiny": WorkloadConfig("tiny", d=256, V=4096, n_responses=2, len_lo=32, len_hi=32,
                           w_std=1.0 / math.sqrt(256), temperature=1.0, seed=1,
                           micro_batch=0, rollout_batch=16, oracle_rows=0),
    "small": WorkloadConfig("small", d=2048, V=151936, n_responses=16, len_lo=128, len_hi=1024,
                            w_std=0.02, temperature=1.0, seed=2,
                            micro_batch=0, rollout_batch=0, oracle_rows=256),
    "mid": WorkloadConfig("mid", d=4096, V=151936, n_responses=64, len_lo=512, len_hi=4096,
                          w_std=0.02, temperature=1.0, seed=3,
                          micro_batch=16384, rollout_batch=0, oracle_rows=2048),
    "stress": WorkloadConfig("stress", d=4096, V=151936, n_responses=64, len_lo=512, len_hi=4096,
                             w_std=0.02, temperature=1.0, seed=3,
                             micro_batch=16384, rollout_batch=256, oracle_rows=256),
    "long": WorkloadConfig("long", d=5120, V=152064, n_responses=8, len_lo=16384, len_hi=16384,
                           w_std=0.02, temperature=0.7, seed=5,
                           micro_batch=32768, rollout_batch=64, oracle_rows=256),
}


def seeds(cfg: WorkloadConfig):
    """(hidden seed, weight seed, uniform seed) of a configuration."""
    return 1000 + cfg.seed, 2000 + cfg.seed, 3000 + cfg.seed
