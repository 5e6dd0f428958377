"""Batch invariance on the GPU: a row's logp / entropy / lse are bitwise the
same however rows are batched -- rollout decode batches of any size in any
order, training micro-batches of any size, a row alone -- at the headline
shape (d = 4096, V = 151936)."""

import numpy as np
import pytest
import torch

import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode
from tim_testutil import bits_equal, inputs, random_tokens, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


@pytest.fixture(scope="module")
def headline():
    T, d, V = 2048, 4096, 151936
    h, W = inputs(T, d, V, seed=31, w_std=0.02)
    tok = random_tokens(T, V, seed=31)
    ref = tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, micro_batch=0, lse=True)
    return h, W, tok, ref


def _same(out, ref, rows=None):
    for x, y in zip(out, ref):
        if rows is not None:
            y = y[rows]
        assert bits_equal(x, y)


@pytest.mark.parametrize("mb", [1, 100, 256, 1000, 2047])
def test_training_micro_batches(headline, mb):
    h, W, tok, ref = headline
    _same(tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, micro_batch=mb, lse=True), ref)


def test_rollout_random_groupings_shuffled(headline):
    h, W, tok, ref = headline
    T = h.shape[0]
    rng = np.random.default_rng(0)
    perm = rng.permutation(T)
    i = 0
    calls = 0
    while i < T:
        n = int(rng.integers(1, 257))
        rows = torch.as_tensor(perm[i:i + n], device="cuda")
        out = tim.logprobs(h[rows].contiguous(), W, tok[rows].contiguous(), 1.0, mode=Mode.ROLLOUT, lse=True)
        _same(out, ref, rows)
        i += n
        calls += 1
    print(f"[invariance] {calls} rollout calls of random size 1..256 all bitwise equal")


def test_single_rows_and_positions(headline):
    h, W, tok, ref = headline
    for r in [0, 1, 31, 32, 63, 64, 255, 256, 1023, 2047]:
        _same(tim.logprobs(h[r:r + 1], W, tok[r:r + 1], 1.0, mode=Mode.ROLLOUT, lse=True), ref, slice(r, r + 1))
    # the same row repeated at every position of a 256-row tile
    r = 777
    rep = h[r:r + 1].repeat(256, 1).contiguous()
    out = tim.logprobs(rep, W, tok[r:r + 1].repeat(256).contiguous(), 1.0, mode=Mode.TRAINING, lse=True)
    for x, y in zip(out, ref):
        assert bits_equal(x, y[r:r + 1].expand(256).contiguous())


def test_repeat_runs_identical(headline):
    h, W, tok, ref = headline
    for _ in range(3):
        _same(tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, micro_batch=512, lse=True), ref)


@pytest.mark.parametrize("d,mb", [(5120, 0), (5120, 20000), (4096, 40000)])
def test_training_launch_cap_splits_micro_batches(d, mb):
    """A training micro-batch longer than the planner's launch cap (8192 rows at d = 5120, 16384 at d = 4096) runs as
    consecutive launches: 8192 + 8192 + 300 rows for 16684 tokens at d = 5120 (one micro-batch, or 16684 / 20000),
    16384 + 300 at d = 4096. Bitwise the results of one rollout launch over all rows and of 256-row micro-batches."""
    T = 2 * 8192 + 300 if d == 5120 else 16384 + 300
    V = 4096
    h, W = inputs(T, d, V, seed=37)
    tok = random_tokens(T, V, seed=37)
    assert tim.rows_per_launch(T, d, Mode.TRAINING, mb) == (8192 if d == 5120 else 16384)
    assert tim.rows_per_launch(T, d, Mode.ROLLOUT, mb) == T
    ref = tim.logprobs(h, W, tok, 0.7, mode=Mode.ROLLOUT, lse=True)
    _same(tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, micro_batch=mb, lse=True), ref)
    _same(tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, micro_batch=256, lse=True), ref)
