"""fp64 CPU oracle for the token log-probability path and its mismatch statistics.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or run
anything in this package; only the tests, the smoke check and the benchmark's
CPU-baseline leg use it. It shares no code with the HIP library: it reads the
raw bf16 bit patterns of the inputs, widens them exactly to fp64 and computes
each quantity straight from its definition.

Parity status (each function's own docstring names its pins):

* ``logprobs``      pinned (closed forms, brute force, library routines).
* ``mismatch``      pinned (Table 1 of the paper, closed forms, series).
* ``mismatch_seq``  pinned (closed forms, telescoping, brute force, boundaries).
* ``logit_grads``, ``logprob_grads``  pinned (finite differences of the pinned
  forward, float64 autograd, closed forms, the zero-sum identity).
* ``rmsnorm``, ``rmsnorm_grads``, ``round_bf16``  pinned (torch's bf16 cast and
  float64 rms_norm, ties, closed forms, finite differences, float64 autograd).
* ``ppo_loss``  pinned (float64 autograd through the textbook loss, closed
  forms, clip regions, response sums).
"""

from .logprobs import bf16_to_f64, logits, logprobs  # noqa: F401
from .grads import logit_grads, logprob_grads  # noqa: F401
from .mismatch import mismatch, mismatch_seq  # noqa: F401
from .ppo import ppo_loss  # noqa: F401
from .rmsnorm import f64_to_bf16_bits, rmsnorm, rmsnorm_grads, round_bf16  # noqa: F401
