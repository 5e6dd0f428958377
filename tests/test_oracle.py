"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each test fixes the oracle to something independent: exact rational
arithmetic, a closed form, a library routine (torch's bf16 widening, scipy's
log_softmax and entropy), an identity between two of its outputs that a
dropped term or a wrong index would break, or the values printed in Table 1.
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
from workload import bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(x):
    """fp32/fp64 array -> bf16 bit patterns (torch RNE cast)."""
    return bf16_bits(torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16))


def _rand_bits(shape, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return _bits(rng.standard_normal(shape) * scale)


# ---------------------------------------------------------------- bf16 widening

def test_bf16_widening_matches_torch():
    rng = np.random.default_rng(0)
    vals = np.concatenate([rng.standard_normal(1000) * 10.0 ** rng.integers(-40, 38, 1000),
                           [0.0, -0.0, np.inf, -np.inf, 1e-39, -1e-40, 3.0e38]]).astype(np.float32)
    t = torch.as_tensor(vals).to(torch.bfloat16)
    ref = t.to(torch.float64).numpy()
    got = oracle.bf16_to_f64(bf16_bits(t))
    np.testing.assert_array_equal(got, ref)
    nan_bits = np.array([0x7FC0, 0xFFC1], dtype=np.uint16)
    assert np.isnan(oracle.bf16_to_f64(nan_bits)).all()


# ---------------------------------------------------------------- logits

def test_logits_exact_rational():
    """z = (h . w) / tau against exact rational dot products."""
    T, d, V = 3, 16, 5
    hb = _rand_bits((T, d), 1)
    wb = _rand_bits((V, d), 2, 0.3)
    tau = 0.7
    z = oracle.logits(hb, wb, tau)
    hf = oracle.bf16_to_f64(hb)
    wf = oracle.bf16_to_f64(wb)
    for i in range(T):
        for v in range(V):
            exact = sum(Fraction(hf[i, k]) * Fraction(wf[v, k]) for k in range(d)) / Fraction(tau)
            assert abs(Fraction(z[i, v]) - exact) <= abs(exact) * Fraction(1, 2 ** 50) + Fraction(1, 2 ** 1000)


def test_logits_vocab_chunking_is_exact_split():
    hb = _rand_bits((4, 32), 3)
    wb = _rand_bits((50, 32), 4)
    a = oracle.logits(hb, wb, 1.0, vocab_chunk=7)
    b = oracle.logits(hb, wb, 1.0, vocab_chunk=50)
    np.testing.assert_allclose(a, b, rtol=1e-15, atol=1e-15)
    assert a.shape == (4, 50)


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("V", [1, 2, 7, 4096, 151936])
def test_uniform_row(V):
    """h = 0: every logit is 0, so logp = -log V and H = log V."""
    d = 32
    hb = _bits(np.zeros((2, d)))
    wb = _rand_bits((V, d), 5)
    tok = np.array([0, V - 1])
    lp, H = oracle.logprobs(hb, wb, tok, 1.0)
    np.testing.assert_allclose(lp, -math.log(V), rtol=0, atol=1e-12)
    np.testing.assert_allclose(H, math.log(V), rtol=0, atol=1e-12)


def test_identical_vocab_rows_uniform():
    """All w_v equal (h nonzero): uniform distribution again."""
    V, d = 300, 64
    row = _rand_bits((1, d), 6)
    wb = np.repeat(row, V, axis=0)
    hb = _rand_bits((3, d), 7)
    lp, H = oracle.logprobs(hb, wb, np.array([0, 17, 299]), 1.0)
    np.testing.assert_allclose(lp, -math.log(V), atol=1e-12)
    np.testing.assert_allclose(H, math.log(V), atol=1e-12)


def test_single_token_vocab():
    hb = _rand_bits((4, 32), 8)
    wb = _rand_bits((1, 32), 9)
    lp, H = oracle.logprobs(hb, wb, np.zeros(4, dtype=np.int64), 0.9)
    np.testing.assert_array_equal(lp, 0.0)
    np.testing.assert_allclose(H, 0.0, atol=1e-15)


def _planted(zrows, tau=1.0):
    """h = e_0, W[:, 0] = z values (exact in bf16): logits equal z / tau exactly."""
    zrows = np.asarray(zrows, dtype=np.float64)
    T, V = zrows.shape
    d = 32
    assert T == 1
    h = np.zeros((1, d)); h[0, 0] = 1.0
    w = np.zeros((V, d)); w[:, 0] = zrows[0]
    hb, wb = _bits(h), _bits(w)
    np.testing.assert_array_equal(oracle.bf16_to_f64(wb)[:, 0], zrows[0])  # exact in bf16
    return hb, wb


@pytest.mark.parametrize("z0,z1", [(0.0, 0.0), (1.5, -0.25), (-3.0, 5.0), (20.0, -20.0)])
def test_two_token_vocab_closed_form(z0, z1):
    hb, wb = _planted([[z0, z1]])
    for tok in (0, 1):
        lp, H = oracle.logprobs(hb, wb, np.array([tok]), 1.0)
        dz = (z0 - z1) if tok == 0 else (z1 - z0)
        exp_lp = -math.log1p(math.exp(-dz)) if dz > -700 else dz
        p = 1.0 / (1.0 + math.exp(-(z0 - z1)))
        exp_H = -sum(q * math.log(q) for q in (p, 1.0 - p) if q > 0)
        assert abs(lp[0] - exp_lp) <= 1e-13
        assert abs(H[0] - exp_H) <= 1e-13


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("tau", [1.0, 0.7, 3.0])
def test_planted_logits_vs_scipy(seed, tau):
    """Known logit vector: compare with scipy's log_softmax and entropy."""
    rng = np.random.default_rng(seed)
    V = 97
    z = oracle.bf16_to_f64(_bits(rng.standard_normal(V) * 4))
    hb, wb = _planted(z[None, :])
    ref_lsm = scipy.special.log_softmax(z / tau)
    ref_H = scipy.stats.entropy(scipy.special.softmax(z / tau))
    for tok in (0, 13, 96):
        lp, H = oracle.logprobs(hb, wb, np.array([tok]), tau)
        assert abs(lp[0] - ref_lsm[tok]) <= 1e-12
        assert abs(H[0] - ref_H) <= 1e-12


def test_one_hot_dominant_row():
    """The token's logit exceeds every other by >= 100: logp ~ 0 and H ~ 0."""
    V = 64
    z = np.full(V, -50.0); z[11] = 60.0
    hb, wb = _planted(z[None, :])
    lp, H = oracle.logprobs(hb, wb, np.array([11]), 1.0)
    assert -1e-40 <= lp[0] <= 0.0
    assert 0.0 <= H[0] <= 1e-40
    lp_other, _ = oracle.logprobs(hb, wb, np.array([3]), 1.0)
    assert abs(lp_other[0] - (-110.0)) <= 1e-12


# ---------------------------------------------------------------- identities

def _tiny(T=5, V=40, d=32, seed=11, scale=1.0):
    return _rand_bits((T, d), seed, scale), _rand_bits((V, d), seed + 1, 0.3)


@pytest.mark.parametrize("tau", [1.0, 0.5])
def test_probabilities_sum_to_one_and_entropy_identity(tau):
    """For each row: sum_v exp(logp(v)) = 1 and H = -sum_v p_v logp(v), where
    logp(v) is the oracle's own log-probability of token v."""
    T, V = 5, 40
    hb, wb = _tiny(T, V)
    rep = np.repeat(hb, V, axis=0)
    toks = np.tile(np.arange(V), T)
    lp, H = oracle.logprobs(rep, wb, toks, tau)
    lp = lp.reshape(T, V)
    p = np.exp(lp)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-13)
    np.testing.assert_allclose(-(p * lp).sum(axis=1), H.reshape(T, V)[:, 0], atol=1e-12)
    assert (np.ptp(H.reshape(T, V), axis=1) == 0).all()  # entropy does not depend on the token


def test_duplicated_vocabulary_shifts_by_log2():
    hb, wb = _tiny(6, 50)
    tok = np.array([0, 5, 10, 20, 30, 49])
    lp, H = oracle.logprobs(hb, wb, tok, 1.0)
    lp2, H2 = oracle.logprobs(hb, np.concatenate([wb, wb]), tok, 1.0)
    np.testing.assert_allclose(lp2, lp - math.log(2), atol=1e-12)
    np.testing.assert_allclose(H2, H + math.log(2), atol=1e-12)


def test_vocab_permutation_invariance():
    hb, wb = _tiny(6, 50)
    tok = np.array([0, 5, 10, 20, 30, 49])
    perm = np.random.default_rng(3).permutation(50)
    inv = np.argsort(perm)
    lp, H = oracle.logprobs(hb, wb, tok, 1.0)
    lp2, H2 = oracle.logprobs(hb, wb[perm], inv[tok], 1.0)
    np.testing.assert_allclose(lp2, lp, atol=1e-12)
    np.testing.assert_allclose(H2, H, atol=1e-12)


def test_temperature_divides_logits():
    """(2h, tau = 2) equals (h, tau = 1) exactly: doubling is exact in bf16 and fp64.
    (h, tau) equals the planted logits divided by tau, not multiplied."""
    hb, wb = _tiny(4, 30)
    h2 = _bits(oracle.bf16_to_f64(hb) * 2.0)
    tok = np.array([1, 2, 3, 4])
    a = oracle.logprobs(hb, wb, tok, 1.0)
    b = oracle.logprobs(h2, wb, tok, 2.0)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    c = oracle.logprobs(hb, wb, tok, 0.25)
    assert not np.allclose(a[1], c[1])
    # tau -> infinity flattens the distribution to uniform
    _, Hbig = oracle.logprobs(hb, wb, tok, 1e12)
    np.testing.assert_allclose(Hbig, math.log(30), atol=1e-9)


def test_rows_are_independent_and_blocking_is_invisible():
    hb, wb = _tiny(9, 33)
    tok = np.arange(9) * 3
    a = oracle.logprobs(hb, wb, tok, 1.0, row_block=256)
    b = oracle.logprobs(hb, wb, tok, 1.0, row_block=2)
    for i in range(9):
        c = oracle.logprobs(hb[i:i + 1], wb, tok[i:i + 1], 1.0)
        assert abs(c[0][0] - a[0][i]) <= 1e-14 and abs(c[1][0] - a[1][i]) <= 1e-14
    np.testing.assert_allclose(a[0], b[0], atol=1e-14)
    np.testing.assert_allclose(a[1], b[1], atol=1e-14)


def test_ranges_on_random_rows():
    hb, wb = _tiny(20, 500, d=64, scale=3.0)
    tok = np.random.default_rng(1).integers(0, 500, 20)
    lp, H = oracle.logprobs(hb, wb, tok, 1.0)
    assert (lp <= 0).all()
    assert (H >= 0).all() and (H <= math.log(500) + 1e-12).all()


def test_out_of_range_token_gives_nan_logp():
    hb, wb = _tiny(3, 20)
    lp, H = oracle.logprobs(hb, wb, np.array([-1, 5, 20]), 1.0)
    assert np.isnan(lp[0]) and np.isnan(lp[2]) and np.isfinite(lp[1])
    assert np.isfinite(H).all()


# ---------------------------------------------------------------- mismatch

def _table1():
    rows = np.loadtxt(os.path.join(GOLDEN, "table1_token_logprobs.txt"), comments="#")
    return rows[:, 1], rows[:, 2], rows[:, 3]


def test_mismatch_table1_sign_and_values():
    """Table 1: delta = log pi_train - log pi_rollout. Each printed value is
    rounded to 3 decimals, so the recomputed delta is within 1.5e-3."""
    rollout, train, printed = _table1()
    delta, k3, w = oracle.mismatch(train, rollout, 2.0)
    assert np.max(np.abs(delta - printed)) <= 1.5e-3
    # position 4 is the argmax flip: -0.827 - (-0.694) = -0.133
    assert abs(delta[3] - (-0.133)) < 1e-12
    assert abs(k3[3] - 0.0084651) < 5e-7
    assert abs(w[3] - 0.8754650) < 5e-7
    # the opposite convention would flip the sign of the large entry
    d_swapped, _, _ = oracle.mismatch(rollout, train, 2.0)
    assert abs(d_swapped[3] - printed[3]) > 0.2


@pytest.mark.parametrize("C", [0.5, 1.0, 2.0])
def test_mismatch_identical_inputs(C):
    x = np.random.default_rng(0).standard_normal(100).astype(np.float32) - 3
    delta, k3, w = oracle.mismatch(x, x, C)
    assert (delta == 0).all() and (k3 == 0).all()
    assert (w == min(1.0, C)).all()


def test_k3_literal_form_at_moderate_delta():
    d = np.array([-3.0, -1.0, -0.5, -0.1, 0.1, 0.5, 1.0, 3.0])
    _, k3, _ = oracle.mismatch(d, np.zeros_like(d), 2.0)
    r = np.exp(d)
    np.testing.assert_allclose(k3, (r - 1) - np.log(r), rtol=1e-12)


def test_k3_taylor_series_at_small_delta():
    d = np.array([-1e-3, -1e-5, -1e-7, 1e-7, 1e-5, 1e-3, 0.001])
    _, k3, _ = oracle.mismatch(d, np.zeros_like(d), 2.0)
    series = d ** 2 / 2 + d ** 3 / 6 + d ** 4 / 24 + d ** 5 / 120
    np.testing.assert_allclose(k3, series, rtol=1e-8)
    assert abs(k3[-1] - 5.0016670834e-7) < 1e-16
    assert (oracle.mismatch(np.random.default_rng(1).standard_normal(1000), np.zeros(1000), 2.0)[1] >= 0).all()


def test_truncated_weight():
    d = np.array([math.log(2.0), 0.0, -0.133, 5.0, -50.0])
    _, _, w = oracle.mismatch(d, np.zeros_like(d), 2.0)
    assert abs(w[0] - 2.0) < 1e-15
    assert w[1] == 1.0
    assert abs(w[2] - math.exp(-0.133)) < 1e-15
    assert w[3] == 2.0
    assert 0 < w[4] < 1e-21
    _, _, wc = oracle.mismatch(np.array([0.0, math.log(0.5) + 1e-9]), np.zeros(2), 0.5)
    assert wc[0] == 0.5 and wc[1] == 0.5


# ---------------------------------------------------------------- sequence level (Section 4.2, appendix)

def _random_stream(seed, n_resp, max_len, scale=1e-2):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, max_len + 1, size=n_resp)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T = int(cu[-1])
    b = (rng.standard_normal(T) - 2.0).astype(np.float32)
    a = (b + scale * rng.standard_normal(T)).astype(np.float32)
    return a, b, cu


@pytest.mark.parametrize("est", ["k1", "k3"])
def test_seq_constant_delta_closed_form(est):
    """A response of L tokens with the same delta scores L * K(delta) (exactly,
    as math.fsum of equal terms is the correctly rounded product)."""
    for delta, L in [(-0.133, 7), (0.01, 1000), (1e-4, 16384), (0.5, 3)]:
        a = np.full(L, delta, dtype=np.float64)
        score, _, _ = oracle.mismatch_seq(a, np.zeros(L), [0, L], est, 2.0, 1e-3)
        K = -delta if est == "k1" else math.expm1(delta) - delta
        assert score[0] == L * K, (est, delta, L)


def test_seq_k1_telescopes():
    """K1 = -log r_corr = logp_b - logp_a, so a response's K1 score is
    sum(logp_b) - sum(logp_a) over it."""
    a, b, cu = _random_stream(3, 20, 300)
    score, _, _ = oracle.mismatch_seq(a, b, cu, "k1", 2.0, 1e-3)
    for j in range(len(cu) - 1):
        s0, s1 = cu[j], cu[j + 1]
        ref = math.fsum(b[s0:s1].astype(np.float64)) - math.fsum(a[s0:s1].astype(np.float64))
        assert abs(score[j] - ref) <= 1e-12 * (1 + abs(ref))


@pytest.mark.parametrize("C,tau", [(2.0, 1e-3), (0.5, 0.0), (2.0, -1.0)])
def test_seq_identical_inputs(C, tau):
    x = (np.random.default_rng(4).standard_normal(50) - 3).astype(np.float32)
    cu = np.array([0, 10, 10, 50], dtype=np.int64)
    for est in ("k1", "k3"):
        score, keep, w = oracle.mismatch_seq(x, x, cu, est, C, tau)
        assert (score == 0).all()
        assert (keep == (0.0 <= tau)).all()
        assert (w == (min(1.0, C) if 0.0 <= tau else 0.0)).all()


def test_seq_empty_responses_and_keep_boundary():
    a = np.array([0.1, -0.2, 0.05], dtype=np.float64)
    b = np.zeros(3)
    cu = np.array([0, 0, 3, 3], dtype=np.int64)
    score, keep, w = oracle.mismatch_seq(a, b, cu, "k3", 2.0, 1e-3)
    assert score[0] == 0 and score[2] == 0 and keep[0] and keep[2]
    s = score[1]
    assert s > 0
    # keep is score <= tau: the score itself is kept, the next float below rejects
    _, keep_eq, w_eq = oracle.mismatch_seq(a, b, cu, "k3", 2.0, s)
    _, keep_lt, w_lt = oracle.mismatch_seq(a, b, cu, "k3", 2.0, np.nextafter(s, -np.inf))
    assert keep_eq[1] and not keep_lt[1]
    np.testing.assert_allclose(w_eq, np.minimum(np.exp(a - b), 2.0), rtol=1e-15)
    assert (w_lt == 0).all()


@pytest.mark.parametrize("est", ["k1", "k3"])
def test_seq_brute_force(est):
    """Token-by-token accumulation in plain Python (each token looks up its
    response by scanning the offsets) on small random streams."""
    a, b, cu = _random_stream(11, 13, 40, scale=0.05)
    C, tau = 1.5, 2e-3
    score, keep, w = oracle.mismatch_seq(a, b, cu, est, C, tau)
    n = len(cu) - 1
    acc = [0.0] * n
    for t in range(len(a)):
        j = next(j for j in range(n) if cu[j] <= t < cu[j + 1])
        d = float(a[t]) - float(b[t])
        acc[j] += (-d) if est == "k1" else (math.exp(d) - 1.0 - d)
    for j in range(n):
        assert abs(score[j] - acc[j]) <= 1e-12 + 1e-9 * abs(acc[j])
        assert keep[j] == (score[j] <= tau)
        for t in range(cu[j], cu[j + 1]):
            d = float(a[t]) - float(b[t])
            ref = min(math.exp(d), C) if keep[j] else 0.0
            assert abs(w[t] - ref) <= 4e-16 * ref
    if est == "k3":
        assert (score >= 0).all()
    assert 0 < keep.sum() < n  # the draw exercises both outcomes


def test_seq_response_order_is_irrelevant():
    a, b, cu = _random_stream(5, 9, 60)
    score, keep, w = oracle.mismatch_seq(a, b, cu, "k3", 2.0, 1e-3)
    perm = np.random.default_rng(6).permutation(len(cu) - 1)
    pieces = [(a[cu[j]:cu[j + 1]], b[cu[j]:cu[j + 1]]) for j in perm]
    a2 = np.concatenate([p[0] for p in pieces])
    b2 = np.concatenate([p[1] for p in pieces])
    cu2 = np.concatenate([[0], np.cumsum([len(p[0]) for p in pieces])])
    score2, keep2, _ = oracle.mismatch_seq(a2, b2, cu2, "k3", 2.0, 1e-3)
    assert (score2 == score[perm]).all() and (keep2 == keep[perm]).all()


# ---------------------------------------------------------------- gradients

def _loss(hb, wb, tok, tau, g, e):
    lp, H = oracle.logprobs(hb, wb, tok, tau)
    lp = np.where(np.isnan(lp), 0.0, lp)
    return float((g * lp).sum() + (e * H).sum())


def _grid_bits(shape, seed):
    """bf16 values k / 256 with 64 <= |k| <= 248: every value +-1/256 and +-2/256
    is again exact in bf16, so finite differences perturb exactly."""
    rng = np.random.default_rng(seed)
    k = rng.integers(64, 249, size=shape) * rng.choice([-1, 1], size=shape)
    return _bits(k / 256.0)


def _fd(f, x_bits, idx, step=1.0 / 256):
    """Richardson-extrapolated central difference of f at x_bits[idx] (O(step^4))."""
    x = oracle.bf16_to_f64(x_bits)

    def at(delta):
        y = x.copy()
        y[idx] += delta
        yb = _bits(y)
        assert oracle.bf16_to_f64(yb)[idx] == y[idx]  # the perturbed value is exact
        return f(yb)
    d1 = at(step) - at(-step)
    d2 = at(2 * step) - at(-2 * step)
    return (8 * d1 - d2) / (12 * step)


@pytest.mark.parametrize("tau", [1.0, 0.7])
def test_grads_match_finite_differences(tau):
    """Derivative by definition: perturb every input of a tiny case in the pinned forward."""
    T, d, V = 3, 8, 6
    hb, wb = _grid_bits((T, d), 40), _grid_bits((V, d), 41)
    tok = np.array([0, 3, 5])
    rng = np.random.default_rng(42)
    g, e = rng.standard_normal(T), rng.standard_normal(T)
    dh, dw = oracle.logprob_grads(hb, wb, tok, tau, g, e)
    for i in range(T):
        for k in range(d):
            fd = _fd(lambda xb: _loss(xb, wb, tok, tau, g, e), hb, (i, k))
            assert abs(fd - dh[i, k]) <= 1e-6 * (1 + abs(fd)), (i, k, fd, dh[i, k])
    for v in range(V):
        for k in range(d):
            fd = _fd(lambda xb: _loss(hb, xb, tok, tau, g, e), wb, (v, k))
            assert abs(fd - dw[v, k]) <= 1e-6 * (1 + abs(fd)), (v, k, fd, dw[v, k])


@pytest.mark.parametrize("tau", [1.0, 0.6])
def test_grads_match_torch_autograd(tau):
    """torch autograd in float64 through the textbook forward (log_softmax,
    gather, entropy) -- a library differentiation, independent of the oracle's
    closed-form Jacobian."""
    T, d, V = 7, 48, 37
    hb, wb = _tiny(T, V, d=d, scale=2.0)
    tok = np.array([0, 36, 5, -1, 12, 37, 20])  # two out-of-range ids: no logp term
    rng = np.random.default_rng(5)
    g, e = rng.standard_normal(T), rng.standard_normal(T)
    h = torch.tensor(oracle.bf16_to_f64(hb), requires_grad=True)
    w = torch.tensor(oracle.bf16_to_f64(wb), requires_grad=True)
    logq = torch.log_softmax((h @ w.T) / tau, dim=1)
    H = -(logq.exp() * logq).sum(dim=1)
    ok = torch.tensor((tok >= 0) & (tok < V))
    lp = logq[torch.arange(T), torch.tensor(np.clip(tok, 0, V - 1))]
    L = (torch.tensor(g) * torch.where(ok, lp, torch.zeros_like(lp))).sum() + (torch.tensor(e) * H).sum()
    L.backward()
    dh, dw = oracle.logprob_grads(hb, wb, tok, tau, g, e)
    np.testing.assert_allclose(dh, h.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dw, w.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_grads_sum_to_zero_over_vocab():
    """sum_v dz_v = 0 (softmax gradients): dW's columns sum to zero, and dh does
    not change when every w_v is shifted by the same vector."""
    T, d, V = 5, 32, 40
    hb, wb = _tiny(T, V, d=d)
    tok = np.array([1, 2, 39, 0, 17])
    rng = np.random.default_rng(6)
    g, e = rng.standard_normal(T), rng.standard_normal(T)
    dacc = oracle.logit_grads(hb, wb, tok, 1.0, g, e)
    np.testing.assert_allclose(dacc.sum(axis=1), 0.0, atol=1e-14)
    dh, dw = oracle.logprob_grads(hb, wb, tok, 1.0, g, e)
    np.testing.assert_allclose(dw.sum(axis=0), 0.0, atol=1e-12)
    # a common shift of every w_v by a vector c (exact on the k / 256 grid)
    wg = _grid_bits((V, d), 8)
    c = np.random.default_rng(9).integers(-4, 5, size=d) / 256.0
    w2 = oracle.bf16_to_f64(wg) + c
    wg2 = _bits(w2)
    np.testing.assert_array_equal(oracle.bf16_to_f64(wg2), w2)
    dh1, _ = oracle.logprob_grads(hb, wg, tok, 1.0, g, e)
    dh2, _ = oracle.logprob_grads(hb, wg2, tok, 1.0, g, e)
    np.testing.assert_allclose(dh2, dh1, atol=1e-12)


def test_grads_uniform_row_closed_form():
    """h = 0: every logit is 0, p = 1/V, H = log V, q + H = 0. Then
    dh = g (w_a - mean_v w_v) / tau, the entropy gradient vanishes, dW = 0."""
    T, d, V = 3, 16, 11
    hb = _bits(np.zeros((T, d)))
    wb = _rand_bits((V, d), 7)
    tok = np.array([0, 4, 10])
    g = np.array([1.0, -2.0, 0.5])
    e = np.array([3.0, 1.0, -1.0])
    tau = 0.8
    dh, dw = oracle.logprob_grads(hb, wb, tok, tau, g, e)
    w = oracle.bf16_to_f64(wb)
    exp_dh = g[:, None] * (w[tok] - w.mean(axis=0)) / tau
    np.testing.assert_allclose(dh, exp_dh, atol=1e-14)
    np.testing.assert_array_equal(dw, 0.0)


@pytest.mark.parametrize("z0,z1", [(0.0, 0.0), (1.5, -0.25), (-3.0, 5.0)])
def test_grads_two_token_closed_form(z0, z1):
    """V = 2 is the logistic model: with s = sigmoid(z0 - z1) and token 0,
    dlogp/dz0 = 1 - s, dlogp/dz1 = s - 1; dH/dz0 = -s (1 - s) (z0 - z1) = -dH/dz1."""
    hb, wb = _planted([[z0, z1]])
    s = 1.0 / (1.0 + math.exp(-(z0 - z1)))
    dacc = oracle.logit_grads(hb, wb, np.array([0]), 1.0, np.array([1.0]), np.array([0.0]))
    np.testing.assert_allclose(dacc[0], [1 - s, s - 1], atol=1e-15)
    dacc = oracle.logit_grads(hb, wb, np.array([0]), 1.0, np.array([0.0]), np.array([1.0]))
    dH0 = -s * (1 - s) * (z0 - z1)
    np.testing.assert_allclose(dacc[0], [dH0, -dH0], atol=1e-15)


def test_grads_linear_in_upstream():
    T, d, V = 4, 32, 25
    hb, wb = _tiny(T, V, d=d)
    tok = np.array([3, 1, 4, 1])
    rng = np.random.default_rng(9)
    g1, e1, g2, e2 = (rng.standard_normal(T) for _ in range(4))
    a = oracle.logit_grads(hb, wb, tok, 1.3, g1, e1)
    b = oracle.logit_grads(hb, wb, tok, 1.3, g2, e2)
    c = oracle.logit_grads(hb, wb, tok, 1.3, 2 * g1 - g2, 2 * e1 - e2)
    np.testing.assert_allclose(c, 2 * a - b, atol=1e-14)
    z = oracle.logit_grads(hb, wb, tok, 1.3, np.zeros(T), np.zeros(T))
    np.testing.assert_array_equal(z, 0.0)


# ---------------------------------------------------------------- final RMS norm

def test_round_bf16_matches_torch_cast_of_fp32_values():
    rng = np.random.default_rng(20)
    v = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    got = oracle.round_bf16(v.astype(np.float64))
    ref = torch.as_tensor(v).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_ties_to_even_and_off_tie():
    u = 2.0 ** -7  # bf16 spacing in [1, 2)
    cases = [(1 + u / 2, 1.0), (1 + 3 * u / 2, 1 + 2 * u), (-(1 + u / 2), -1.0), (1 + u / 2 + 2.0 ** -40, 1 + u),
             (1 + u / 2 - 2.0 ** -40, 1.0), (0.0, 0.0), (2 - u / 4, 2.0), (2 - 3 * u / 4, 2 - u), (2 - u / 2, 2.0),
             (3 * 2.0 ** -130, None)]
    for v, want in cases:
        got = float(oracle.round_bf16(np.array([v]))[0])
        if want is None:  # below bf16's normal range: still a multiple of its own 8-bit spacing
            m, e = math.frexp(got)
            assert m * 256 == int(m * 256)
        else:
            assert got == want, (v, got, want)


def test_rmsnorm_constant_row_closed_form():
    T, d = 3, 64
    c = np.array([0.5, -3.0, 0.0078125])
    x = np.repeat(c[:, None], d, axis=1)
    for eps in (0.0, 1e-6):
        hb, r, n = oracle.rmsnorm(_bits(x), None, eps)
        for t in range(T):
            assert r[t] == 1.0 / math.sqrt(c[t] * c[t] + eps)
            np.testing.assert_array_equal(n[t], c[t] * r[t])
        np.testing.assert_array_equal(oracle.bf16_to_f64(hb), oracle.round_bf16(n))


@pytest.mark.parametrize("eps", [1e-6, 1e-2])
def test_rmsnorm_matches_torch_rms_norm_float64(eps):
    T, d = 9, 384
    xb = _rand_bits((T, d), 21, 3.0)
    gb = _rand_bits((d,), 22, 1.0)
    x = torch.tensor(oracle.bf16_to_f64(xb))
    g = torch.tensor(oracle.bf16_to_f64(gb))
    _, r, n = oracle.rmsnorm(xb, gb, eps)
    ref = torch.nn.functional.rms_norm(x, (d,), weight=None, eps=eps).numpy()
    np.testing.assert_allclose(n, ref, rtol=1e-14, atol=0)
    ref_g = torch.nn.functional.rms_norm(x, (d,), weight=g, eps=eps).numpy()
    np.testing.assert_allclose(n * g.numpy()[None, :], ref_g, rtol=1e-14, atol=0)


def test_rmsnorm_roundings_match_bf16_model_arithmetic():
    """The model's own arithmetic, in torch on the CPU: fp32 variance and scale,
    a cast to bf16, then bf16 * bf16 with the weight. It rounds from fp32 where
    the oracle rounds from fp64, so the two agree except on rare straddles."""
    T, d, eps = 64, 256, 1e-6
    xb = _rand_bits((T, d), 23, 2.0)
    gb = _rand_bits((d,), 24, 1.0)
    hb, _, _ = oracle.rmsnorm(xb, gb, eps)
    x32 = torch.tensor(oracle.bf16_to_f64(xb), dtype=torch.float32)
    var = x32.pow(2).mean(-1, keepdim=True)
    hs = (x32 * torch.rsqrt(var + eps)).to(torch.bfloat16)
    g16 = torch.tensor(oracle.bf16_to_f64(gb), dtype=torch.float32).to(torch.bfloat16)
    ref = bf16_bits(g16 * hs)
    same = (hb == ref).mean()
    assert same >= 0.999, same
    # without a weight: the single rounding of the normalised row, and a weight of ones changes nothing
    hb1, _, _ = oracle.rmsnorm(xb, None, eps)
    hbo, _, _ = oracle.rmsnorm(xb, _bits(np.ones(d)), eps)
    np.testing.assert_array_equal(hb1, hbo)
    assert (hb1 == bf16_bits(hs)).mean() >= 0.999


def test_rmsnorm_grads_match_finite_differences():
    T, d, eps = 2, 8, 1e-3
    xb, gb = _grid_bits((T, d), 25), _grid_bits((d,), 26)
    G = np.random.default_rng(27).standard_normal((T, d))
    dx, dg = oracle.rmsnorm_grads(xb, gb, eps, G)

    def L_x(xbits):
        return float((G * oracle.bf16_to_f64(gb)[None, :] * oracle.rmsnorm(xbits, gb, eps)[2]).sum())

    def L_g(gbits):
        return float((G * oracle.bf16_to_f64(gbits)[None, :] * oracle.rmsnorm(xb, gbits, eps)[2]).sum())
    for t in range(T):
        for k in range(d):
            fd = _fd(L_x, xb, (t, k))
            assert abs(fd - dx[t, k]) <= 1e-6 * (1 + abs(fd)), (t, k, fd, dx[t, k])
    for k in range(d):
        fd = _fd(L_g, gb, (k,))
        assert abs(fd - dg[k]) <= 1e-9 * (1 + abs(fd)), (k, fd, dg[k])


def test_rmsnorm_grads_match_torch_autograd_and_scale_identity():
    T, d = 6, 96
    xb = _rand_bits((T, d), 28, 2.0)
    gb = _rand_bits((d,), 29, 1.0)
    G = np.random.default_rng(30).standard_normal((T, d))
    for eps in (1e-6, 0.0):
        x = torch.tensor(oracle.bf16_to_f64(xb), requires_grad=True)
        g = torch.tensor(oracle.bf16_to_f64(gb), requires_grad=True)
        (torch.nn.functional.rms_norm(x, (d,), weight=g, eps=eps) * torch.tensor(G)).sum().backward()
        dx, dg = oracle.rmsnorm_grads(xb, gb, eps, G)
        np.testing.assert_allclose(dx, x.grad.numpy(), rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(dg, g.grad.numpy(), rtol=1e-11, atol=1e-13)
    # eps = 0: the normalised row does not change with the row's scale, so x . dL/dx = 0 per row
    dx0, _ = oracle.rmsnorm_grads(xb, gb, 0.0, G)
    x0 = oracle.bf16_to_f64(xb)
    np.testing.assert_allclose((x0 * dx0).sum(axis=1), 0.0, atol=1e-12)
    # without a weight: the same as a weight of ones
    a = oracle.rmsnorm_grads(xb, None, 1e-6, G)
    b = oracle.rmsnorm_grads(xb, _bits(np.ones(d)), 1e-6, G)
    np.testing.assert_array_equal(a[0], b[0])


# ---------------------------------------------------------------- PPO / GRPO token loss

def _ppo_case(seed, T=40, n_seq=5):
    rng = np.random.default_rng(seed)
    lens = rng.multinomial(T - n_seq, np.ones(n_seq) / n_seq) + 1
    cu = np.concatenate([[0], np.cumsum(lens)])
    lo = -rng.exponential(2.0, T)
    lp = lo + rng.normal(0, 0.3, T)
    A = rng.normal(0, 1, T)
    w = rng.uniform(0, 2, T)
    return lp, lo, A, w, cu


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.2), (0.2, 0.28)])
def test_ppo_matches_torch_autograd(eps_low, eps_high):
    lp, lo, A, w, cu = _ppo_case(31)
    n = len(cu) - 1
    out = oracle.ppo_loss(lp, lo, A, cu, eps_low, eps_high, w)
    x = torch.tensor(lp, requires_grad=True)
    r = torch.exp(x - torch.tensor(lo))
    At = torch.tensor(A)
    tok = -torch.minimum(r * At, torch.clamp(r, 1 - eps_low, 1 + eps_high) * At) * torch.tensor(w)
    seq = torch.stack([tok[cu[j]:cu[j + 1]].sum() for j in range(n)])
    L = seq.mean()
    L.backward()
    np.testing.assert_allclose(out["token_loss"], tok.detach().numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(out["seq_loss"], seq.detach().numpy(), rtol=1e-13, atol=1e-14)
    assert abs(out["batch_loss"] - L.item()) <= 1e-13
    np.testing.assert_allclose(out["grad"], x.grad.numpy(), rtol=1e-13, atol=1e-15)
    # C has the gradient of -r A and vanishes at r = 1
    x2 = torch.tensor(lp, requires_grad=True)
    r2 = torch.exp(x2 - torch.tensor(lo))
    (-(r2 - 1) * At).sum().backward()
    np.testing.assert_allclose(x2.grad.numpy(), (-At * r2).detach().numpy(), rtol=1e-14)
    np.testing.assert_allclose(out["contribution"], (-(r2 - 1) * At).detach().numpy(), rtol=1e-14, atol=1e-15)


def test_ppo_closed_forms_and_clip_regions():
    lp, lo, A, w, cu = _ppo_case(32)
    n = len(cu) - 1
    same = oracle.ppo_loss(lo, lo, A, cu, 0.2, 0.3, w)      # r = 1
    np.testing.assert_array_equal(same["token_loss"], -A * w)
    np.testing.assert_allclose(same["grad"], -A * w / n, rtol=1e-15)
    np.testing.assert_array_equal(same["contribution"], 0.0)
    assert not same["clipped"].any()
    zero = oracle.ppo_loss(lp, lo, np.zeros_like(A), cu, 0.2, 0.3, w)
    assert not zero["token_loss"].any() and not zero["grad"].any() and zero["batch_loss"] == 0.0
    # one token per case: (delta, A) -> (loss, grad factor, clipped)
    el, eh = 0.2, 0.3
    cases = [(math.log(1.5), 2.0, -2.0 * (1 + eh), 0.0, True),      # A > 0, above 1 + eps_high: clipped
             (math.log(0.5), 2.0, -2.0 * 0.5, -2.0 * 0.5, False),   # A > 0, below 1 - eps_low: unclipped
             (math.log(0.5), -2.0, 2.0 * (1 - el), 0.0, True),      # A < 0, below 1 - eps_low: clipped
             (math.log(1.5), -2.0, 2.0 * 1.5, 2.0 * 1.5, False),    # A < 0, above 1 + eps_high: unclipped
             (math.log(1.1), 2.0, -2.0 * 1.1, -2.0 * 1.1, False)]   # inside: unclipped
    for dlt, a, loss, grad, clipped in cases:
        o = oracle.ppo_loss(np.array([dlt - 1.0]), np.array([-1.0]), np.array([a]), [0, 1], el, eh)
        assert abs(o["token_loss"][0] - loss) <= 1e-12, (dlt, a, o["token_loss"][0], loss)
        assert abs(o["grad"][0] - grad) <= 1e-12, (dlt, a, o["grad"][0], grad)
        assert bool(o["clipped"][0]) == clipped
        assert o["batch_loss"] == o["seq_loss"][0] == o["token_loss"][0]


def test_ppo_batch_is_mean_of_response_sums_and_order_free():
    lp, lo, A, w, cu = _ppo_case(33, T=60, n_seq=6)
    out = oracle.ppo_loss(lp, lo, A, cu, 0.2, 0.2, w)
    assert abs(out["batch_loss"] - out["seq_loss"].mean()) <= 1e-14
    for j in range(len(cu) - 1):
        assert abs(out["seq_loss"][j] - out["token_loss"][cu[j]:cu[j + 1]].sum()) <= 1e-13
    # responses in another order: the same response sums, permuted
    order = [3, 0, 5, 1, 4, 2]
    segs = [(cu[j], cu[j + 1]) for j in order]
    idx = np.concatenate([np.arange(a, b) for a, b in segs])
    cu2 = np.concatenate([[0], np.cumsum([b - a for a, b in segs])])
    out2 = oracle.ppo_loss(lp[idx], lo[idx], A[idx], cu2, 0.2, 0.2, w[idx])
    np.testing.assert_array_equal(out2["seq_loss"], out["seq_loss"][order])
    assert abs(out2["batch_loss"] - out["batch_loss"]) <= 1e-15
