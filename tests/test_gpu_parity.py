"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle, element
by element, on seeded inputs that span several vocab and row tiles with ragged
tails, plus the degenerate cases of the method."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode, Order
from tim_testutil import (TOL_ENT, TOL_LOGP, bits_equal, check_close, inputs, oracle_rows, random_tokens,
                          require_gpu)
from workload import CONFIGS, bf16_bits, hidden_states, uniforms, vocab_weights
from workload.gen import seeds
from workload.sampler import sample_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_tiny_config_all_rows_both_modes():
    """d=256, V=4096, T=64 (2 responses of 32); tokens drawn from the fp64 softmax."""
    cfg = CONFIGS["tiny"]
    hs, ws, us = seeds(cfg)
    h = hidden_states(cfg.tokens, cfg.d, hs)
    W = vocab_weights(cfg.V, cfg.d, cfg.w_std, ws)
    tok = sample_tokens(h, W, cfg.temperature, uniforms(cfg.tokens, us))
    ref_lp, ref_H = oracle.logprobs(bf16_bits(h), bf16_bits(W), tok.numpy(), cfg.temperature)
    hg, Wg, tg = h.cuda(), W.cuda(), tok.cuda()
    outs = []
    for mode, mb in [(Mode.TRAINING, 0), (Mode.TRAINING, 16), (Mode.TRAINING, 5), (Mode.ROLLOUT, 0)]:
        lp, H, _ = tim.logprobs(hg, Wg, tg, cfg.temperature, mode=mode, micro_batch=mb)
        check_close(f"tiny logp {mode.name} mb={mb}", lp, ref_lp, TOL_LOGP)
        check_close(f"tiny entropy {mode.name} mb={mb}", H, ref_H, TOL_ENT)
        outs.append((lp, H))
    for lp, H in outs[1:]:
        assert bits_equal(lp, outs[0][0]) and bits_equal(H, outs[0][1])
    # the path against itself: every log-ratio is exactly 0
    lr, k3, w = tim.mismatch(outs[0][0], outs[3][0], 2.0)
    assert (lr == 0).all() and (k3 == 0).all() and (w == 1).all()


@pytest.mark.parametrize("T,d,V,tau,mode,mb", [
    (1, 128, 300, 1.0, Mode.ROLLOUT, 0),
    (37, 384, 4096 + 77, 0.7, Mode.ROLLOUT, 0),
    (130, 256, 1000, 1.3, Mode.ROLLOUT, 0),
    (300, 256, 2500, 1.0, Mode.TRAINING, 128),
    (513, 128, 777, 2.0, Mode.TRAINING, 0),
    (700, 640, 5000, 0.5, Mode.TRAINING, 256),
])
def test_ragged_shapes_all_rows(T, d, V, tau, mode, mb):
    print(f"case T={T} d={d} V={V} tau={tau} {mode.name} mb={mb}", flush=True)
    h, W = inputs(T, d, V, seed=T + V)
    tok = random_tokens(T, V, seed=T)
    lp, H, lse = tim.logprobs(h, W, tok, tau, mode=mode, micro_batch=mb, lse=True)
    ref_lp, ref_H = oracle_rows(h, W, tok, tau)
    check_close("logp", lp, ref_lp, TOL_LOGP)
    check_close("entropy", H, ref_H, TOL_ENT)
    z = oracle.logits(bf16_bits(h), bf16_bits(W), tau)
    m = z.max(axis=1, keepdims=True)
    ref_lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    check_close("lse", lse, ref_lse, TOL_LOGP)



@pytest.mark.parametrize("V", [2048 * 256, 2048 * 256 - 77])
def test_maximum_vocabulary_both_modes(V):
    """The largest vocabulary the boundary accepts (2048 tiles: the merge's widest tree, and 4096 or 4095 halves in
    a decode batch) and a ragged one just below it: every row against the oracle in both modes, the modes bitwise
    equal."""
    T, d = 9, 128
    print(f"case maximum vocabulary V={V}", flush=True)
    h, W = inputs(T, d, V, seed=V % 1009, w_std=0.1)
    tok = random_tokens(T, V, seed=V % 1009)
    tok[0] = V - 1          # the last entry of the last tile
    lp_r, H_r, _ = tim.logprobs(h, W, tok, 0.9, mode=Mode.ROLLOUT)
    lp_t, H_t, _ = tim.logprobs(h, W, tok, 0.9, mode=Mode.TRAINING)
    assert bits_equal(lp_r, lp_t) and bits_equal(H_r, H_t)
    ref_lp, ref_H = oracle_rows(h, W, tok, 0.9)
    check_close(f"max-vocab logp V={V}", lp_r, ref_lp, TOL_LOGP)
    check_close(f"max-vocab entropy V={V}", H_r, ref_H, TOL_ENT)


def test_eight_million_rows_one_call():
    """A call of 2^23 + 37 rows at d = 128: in rollout mode one launch of 32769 row tiles over the 2.15 GB hidden
    block, so row offsets pass 2^31 bytes; in training mode launches of 909312 rows (the planner's cap at d = 128).
    The modes bitwise equal, sampled rows (the first, the last, both sides of the 2^31-byte offset, seeded ones)
    against the oracle."""
    T, d, V = 2 ** 23 + 37, 128, 600
    assert tim.rows_per_launch(T, d, Mode.ROLLOUT) == T and tim.rows_per_launch(T, d, Mode.TRAINING) == 909312
    h, W = inputs(T, d, V, seed=23, w_std=0.1)
    tok = random_tokens(T, V, seed=23)
    lp_t, H_t, _ = tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING)
    lp_r, H_r, _ = tim.logprobs(h, W, tok, 1.0, mode=Mode.ROLLOUT)
    assert bits_equal(lp_r, lp_t) and bits_equal(H_r, H_t)
    rng = np.random.default_rng(23)
    edge = 2 ** 31 // (2 * d)  # the first row at byte offset 2^31
    rows = np.unique(np.concatenate([[0, 1, 255, 256, edge - 1, edge, T - 38, T - 1], rng.choice(T, 56, replace=False)]))
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0, rows=rows)
    check_close("8M-row logp", lp_t, ref_lp, TOL_LOGP, rows=rows)
    check_close("8M-row entropy", H_t, ref_H, TOL_ENT, rows=rows)

@pytest.mark.parametrize("V", [1, 2, 3, 255, 256, 257, 511, 513])
def test_small_and_ragged_vocab(V):
    T, d = 70, 256
    h, W = inputs(T, d, V, seed=V, w_std=0.2)
    tok = random_tokens(T, V, seed=V)
    lp, H, _ = tim.logprobs(h, W, tok, 1.0, mode=Mode.ROLLOUT)
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0)
    check_close(f"logp V={V}", lp, ref_lp, TOL_LOGP)
    check_close(f"entropy V={V}", H, ref_H, TOL_ENT)
    if V == 1:
        assert (lp == 0).all() and (H == 0).all()


def test_uniform_rows():
    """h = 0: every logit is 0, logp = -log V and H = log V."""
    T, d, V = 50, 256, 151936
    h = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    _, W = inputs(1, d, V, seed=3)
    tok = random_tokens(T, V, seed=3)
    lp, H, _ = tim.logprobs(h, W, tok, 1.0)
    check_close("uniform logp", lp, np.full(T, -math.log(V)), 2e-5)
    check_close("uniform entropy", H, np.full(T, math.log(V)), 2e-5)


def test_one_hot_dominant_row():
    """w_tok = c*h with every other row tiny: logp -> 0 and H -> 0."""
    T, d, V = 8, 256, 3000
    h, W = inputs(T, d, V, seed=4, w_std=1e-4)
    tok = torch.tensor([5, 255, 256, 1000, 2047, 2999, 1, 0], dtype=torch.int32, device="cuda")
    W[tok.long()] = (h.float() * 4.0).to(torch.bfloat16)  # z_tok = 4 * |h|^2 = 4 d
    lp, H, _ = tim.logprobs(h, W, tok, 1.0)
    assert (lp.abs() <= 1e-6).all(), lp
    assert ((H >= 0) & (H <= 1e-6)).all(), H


def test_out_of_range_tokens_give_nan_logp():
    T, d, V = 10, 256, 1000
    h, W = inputs(T, d, V, seed=5)
    tok = random_tokens(T, V, seed=5)
    bad = tok.clone()
    bad[[0, 3, 9]] = torch.tensor([-1, V, 2 ** 31 - 1], dtype=torch.int32, device="cuda")
    lp, H, lse = tim.logprobs(h, W, tok, 1.0, lse=True)
    lp2, H2, lse2 = tim.logprobs(h, W, bad, 1.0, lse=True)
    assert torch.isnan(lp2[[0, 3, 9]]).all()
    ok = [1, 2, 4, 5, 6, 7, 8]
    assert bits_equal(lp2[ok], lp[ok])
    assert bits_equal(H2, H) and bits_equal(lse2, lse)


def test_gather_is_bit_exact():
    """logp equals the fp32 logit of the token (as the kernel forms it) minus
    the log-normaliser, bit for bit; off-by-one gathers would differ by O(1)."""
    T, d, V = 300, 512, 2000
    h, W = inputs(T, d, V, seed=6)
    tok = random_tokens(T, V, seed=6)
    tok[:4] = torch.tensor([0, 255, 256, V - 1], dtype=torch.int32)
    lp, _, lse = tim.logprobs(h, W, tok, 0.8, lse=True)
    z = tim.logits(h, W, 0.8)
    ztok = z.gather(1, tok.long()[:, None])[:, 0]
    assert bits_equal(lp, ztok - lse)
    # the logits themselves against the oracle's fp64 contraction
    ref_z = oracle.logits(bf16_bits(h), bf16_bits(W), 0.8)
    check_close("logits", z.flatten(), ref_z.flatten(), 2e-5)


def test_temperature_power_of_two_is_exact():
    """(2h, tau = 2) and (h, tau = 1) give the same bits: both scalings are exact."""
    T, d, V = 200, 256, 3000
    h, W = inputs(T, d, V, seed=7)
    tok = random_tokens(T, V, seed=7)
    a = tim.logprobs(h, W, tok, 1.0, lse=True)
    b = tim.logprobs((h.float() * 2).to(torch.bfloat16), W, tok, 2.0, lse=True)
    for x, y in zip(a, b):
        assert bits_equal(x, y)


def test_splitk4_engine_matches_oracle_but_not_bits():
    T, d, V = 400, 1024, 6000
    h, W = inputs(T, d, V, seed=8, w_std=0.05)
    tok = random_tokens(T, V, seed=8)
    a = tim.logprobs(h, W, tok, 1.0)
    b = tim.logprobs(h, W, tok, 1.0, order=Order.SPLITK4)
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0)
    check_close("splitk4 logp", b[0], ref_lp, TOL_LOGP)
    check_close("splitk4 entropy", b[1], ref_H, TOL_ENT)
    differ = (a[0].view(torch.int32) != b[0].view(torch.int32)).float().mean().item()
    print(f"[splitk4] fraction of rows whose logp bits differ: {differ:.3f}")
    # the engine really reduces in another order: a sizeable share of rows change bits
    assert differ > 0.1
    zb = tim.logits(h, W, 1.0, order=Order.SPLITK4)
    za = tim.logits(h, W, 1.0)
    assert not torch.equal(za, zb)
    check_close("splitk4 logits", zb.flatten(), za.double().cpu().flatten(), 1e-4)


@pytest.mark.parametrize("V,mode", [(4096, Mode.TRAINING), (1000, Mode.TRAINING), (4096, Mode.ROLLOUT),
                                    (151936, Mode.ROLLOUT)])
def test_duplicated_vocabulary_shifts_by_log2(V, mode):
    """W -> [W; W] with every token in the first copy: each logit appears
    twice, so the normaliser doubles: logp drops by ln 2 and the entropy rises
    by ln 2 (with 2^k tiles per copy the two copies' subtrees are the same
    partials and the shift is exact up to the final log)."""
    T, d = 64, 256
    h, W = inputs(T, d, V, seed=V % 101, w_std=0.1)
    tok = random_tokens(T, V, seed=V % 101)
    W2 = torch.cat([W, W]).contiguous()
    lp, H, _ = tim.logprobs(h, W, tok, 1.0, mode=mode)
    lp2, H2, _ = tim.logprobs(h, W2, tok, 1.0, mode=mode)
    check_close(f"dup logp V={V}", lp2, (lp.double() - math.log(2)).cpu().numpy(), 5e-6)
    check_close(f"dup entropy V={V}", H2, (H.double() + math.log(2)).cpu().numpy(), 2e-5)


@pytest.mark.parametrize("mode", [Mode.TRAINING, Mode.ROLLOUT])
def test_non_finite_rows_stay_in_their_rows(mode):
    """A NaN or Inf in a row's hidden state gives that row non-finite outputs;
    every other row of the launch is bitwise what it is without them (no
    reduction crosses rows)."""
    T, d, V = 64, 256, 3000
    h, W = inputs(T, d, V, seed=48)
    tok = random_tokens(T, V, seed=48)
    clean = tim.logprobs(h, W, tok, 1.0, mode=mode, lse=True)
    bad = h.clone()
    bad[3, 17] = float("nan")
    bad[40, 0] = float("inf")
    bad[41, :] = float("nan")
    out = tim.logprobs(bad, W, tok, 1.0, mode=mode, lse=True)
    for r in (3, 40, 41):
        assert not torch.isfinite(out[0][r]) and not torch.isfinite(out[1][r])
    ok = [i for i in range(T) if i not in (3, 40, 41)]
    for x, y in zip(out, clean):
        assert bits_equal(x[ok], y[ok])


@pytest.mark.parametrize("T,d,V,tau,w_std,mode", [
    (40, 256, 5000, 0.02, 0.1, Mode.TRAINING),    # logits spread over hundreds of nats: most exps underflow
    (40, 256, 5000, 50.0, 0.1, Mode.ROLLOUT),     # near-uniform rows
    (70, 8192, 1000, 1.0, None, Mode.TRAINING),   # twice the headline's hidden size (128 stages per tile)
])
def test_extreme_temperatures_and_wide_rows(T, d, V, tau, w_std, mode):
    print(f"case T={T} d={d} V={V} tau={tau} {mode.name}", flush=True)
    h, W = inputs(T, d, V, seed=49 + d, w_std=w_std)
    tok = random_tokens(T, V, seed=49)
    lp, H, _ = tim.logprobs(h, W, tok, tau, mode=mode, lse=True)
    ref_lp, ref_H = oracle_rows(h, W, tok, tau)
    check_close(f"logp tau={tau} d={d}", lp, ref_lp, TOL_LOGP)
    check_close(f"entropy tau={tau} d={d}", H, ref_H, TOL_ENT)
    other = Mode.ROLLOUT if mode == Mode.TRAINING else Mode.TRAINING
    for x, y in zip(tim.logprobs(h, W, tok, tau, mode=other, lse=True), (lp, H)):
        assert bits_equal(x, y)
