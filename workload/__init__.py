"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This package draws random numbers and lays them out; it holds none of the
log-probability arithmetic. The only place it touches the model is the token
sampler in ``workload.sampler``, which plays the rollout engine's part (it
draws the token each row emits) and whose logits are never handed to either
side: both sides receive only the token ids it returns.
"""

from .gen import (  # noqa: F401
    WorkloadConfig,
    CONFIGS,
    response_lengths,
    hidden_states,
    vocab_weights,
    uniforms,
    logprob_pairs,
    bf16_bits,
)
