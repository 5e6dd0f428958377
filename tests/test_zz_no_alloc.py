"""tim_logprobs_noalloc (the entry point that allocates nothing: partials in the library's per-GPU device array)
against tim_logprobs (partials in a caller workspace), through the C ABI: bitwise equal outputs on calls in a row
of decreasing size, in every launch shape (training micro-batches, a large rollout launch, a decode batch on half
tiles, the split-K4 engine), the largest launch the array holds, the host-side rejection of a larger one, and no
change in the device's free memory across calls."""

import pytest
import torch

import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode, Order
from tim_testutil import bits_equal, inputs, random_tokens, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _both(h, W, tok, tau, mode, mb, order=Order.INVARIANT):
    T = h.shape[0]
    ref = tim.logprobs(h, W, tok, tau, mode=mode, micro_batch=mb, order=order, lse=True)
    out = tuple(torch.full((T,), float("nan"), device="cuda") for _ in range(3))
    tim.logprobs_noalloc(h, W, tok, tau, mode=mode, micro_batch=mb, order=order, out=out)
    torch.cuda.synchronize()
    for name, x, y in zip(("logp", "entropy", "lse"), out, ref):
        assert bits_equal(x, y), f"{name} differs (T={T}, mode={mode}, mb={mb}, order={order})"


def test_noalloc_equals_workspace_calls_in_a_row():
    d, V = 4096, 151936
    h, W = inputs(5000, d, V, seed=41, w_std=0.02)
    tok = random_tokens(5000, V, 41)
    cases = [  # (rows, mode, micro_batch, order, tau): each call smaller than the one before
        (5000, Mode.TRAINING, 4096, Order.INVARIANT, 1.0),   # two micro-batches, persistent 256-row tiles
        (3001, Mode.ROLLOUT, 0, Order.INVARIANT, 0.7),       # one launch of 3001 rows
        (256, Mode.ROLLOUT, 0, Order.INVARIANT, 1.0),        # a full decode batch, 256-row tiles
        (200, Mode.TRAINING, 0, Order.SPLITK4, 1.3),         # the second engine's order
        (77, Mode.ROLLOUT, 0, Order.INVARIANT, 1.0),         # a ragged decode batch (half tiles)
        (1, Mode.ROLLOUT, 0, Order.INVARIANT, 1.0),
    ]
    for T, mode, mb, order, tau in cases:
        print(f"case T={T} mode={mode.name} mb={mb} order={order.name} tau={tau}", flush=True)
        _both(h[:T], W, tok[:T], tau, mode, mb, order)


def test_noalloc_largest_launch_and_rejection():
    d, V = 128, 151936  # 594 partials of 16 B per row: 7061 rows fill the 64 MiB array
    T = 7061
    h, W = inputs(T, d, V, seed=42)
    tok = random_tokens(T, V, 42)
    print(f"case largest T={T} d={d} V={V}", flush=True)
    _both(h, W, tok, 1.0, Mode.ROLLOUT, 0)
    _both(h[:1000], W, tok[:1000], 1.0, Mode.ROLLOUT, 0)  # then a smaller one
    h2, _ = inputs(T + 1, d, V, seed=43)
    tok2 = random_tokens(T + 1, V, 43)
    lp = torch.full((T + 1,), 5.0, device="cuda")
    with pytest.raises(RuntimeError, match="WORKSPACE"):
        tim.logprobs_noalloc(h2, W, tok2, 1.0, mode=Mode.ROLLOUT, out=(lp, None, None))
    torch.cuda.synchronize()
    assert (lp == 5.0).all(), "a rejected call wrote its output"


def test_noalloc_leaves_free_memory_unchanged():
    d, V = 256, 4096
    h, W = inputs(300, d, V, seed=44)
    tok = random_tokens(300, V, 44)
    out = tuple(torch.empty(300, device="cuda") for _ in range(3))
    tim.logprobs_noalloc(h, W, tok, 1.0, out=out)  # the device's first call may look the array up
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for T in (300, 129, 64, 5):
        tim.logprobs_noalloc(h[:T], W, tok[:T], 1.0, mode=Mode.ROLLOUT, out=tuple(o[:T] for o in out))
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0
