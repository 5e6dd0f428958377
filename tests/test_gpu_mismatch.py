"""tim_mismatch on the GPU against the fp64 oracle and the paper's Table 1."""

import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from tim_testutil import TOL_W_REL, bits_equal, require_gpu

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _run(a, b, C):
    ag = torch.as_tensor(np.asarray(a, dtype=np.float32)).cuda()
    bg = torch.as_tensor(np.asarray(b, dtype=np.float32)).cuda()
    return [x.cpu().double().numpy() for x in tim.mismatch(ag, bg, C)]


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1000, 1 << 20, (1 << 20) + 3])
def test_mismatch_vs_oracle(n):
    rng = np.random.default_rng(n)
    b = (-rng.exponential(2.0, n)).astype(np.float32)
    # mostly tiny discrepancies, some large, like the paper's heavy tail
    a = (b + rng.standard_normal(n) * np.where(rng.random(n) < 0.05, 0.5, 1e-4)).astype(np.float32)
    lr, k3, w = _run(a, b, 2.0)
    rlr, rk3, rw = oracle.mismatch(a, b, 2.0)
    # delta: one fp32 rounding of the exact difference
    assert np.all(np.abs(lr - rlr) <= 2.0 ** -24 * np.abs(rlr) + 1e-45)
    # k3: the kernel rounds an fp64 value within 2^-46 of K3 once to fp32
    # (2^-24 relative, 2^-23 with room for a value next to a rounding
    # midpoint); the oracle's fp64 expm1(d) - d carries expm1's own rounding,
    # up to 2^-52 |expm1(d)| absolute, which for |d| ~ 1e-10 (tiny log-probs a
    # few ulp apart) is the larger term
    k3_tol = 2.0 ** -23 * rk3 + 2.0 ** -52 * np.abs(np.expm1(rlr)) + 2.0 ** -149
    assert np.all(np.abs(k3 - rk3) <= k3_tol)
    assert np.all(np.abs(w - rw) <= TOL_W_REL * rw)
    assert (k3 >= 0).all()
    print(f"[mismatch n={n}] max rel err w = {np.max(np.abs(w - rw) / rw):.2e}")


def test_table1_vector():
    rows = np.loadtxt(os.path.join(GOLDEN, "table1_token_logprobs.txt"), comments="#")
    rollout, train, printed = rows[:, 1], rows[:, 2], rows[:, 3]
    lr, k3, w = _run(train, rollout, 2.0)
    assert np.max(np.abs(lr - printed)) <= 1.5e-3
    assert abs(lr[3] - (-0.133)) < 1e-6
    assert abs(k3[3] - 0.0084651) < 1e-6
    assert abs(w[3] - 0.8754650) < 1e-6


def test_identical_inputs_exact_zero():
    x = (-np.random.default_rng(1).exponential(3.0, 4099)).astype(np.float32)
    for C in (0.5, 1.0, 2.0):
        lr, k3, w = _run(x, x, C)
        assert (lr == 0).all() and (k3 == 0).all() and (w == min(1.0, C)).all()


def test_truncation_boundary_and_nan():
    b = np.zeros(6, dtype=np.float32)
    a = np.array([math.log(2.0), 1.0, -0.5, 20.0, np.nan, -np.inf], dtype=np.float32)
    lr, k3, w = _run(a, b, 2.0)
    assert abs(w[0] - 2.0) <= 2e-7 * 2 and w[1] == 2.0 and w[3] == 2.0
    assert abs(w[2] - math.exp(-0.5)) <= 1e-7
    assert np.isnan(lr[4]) and np.isnan(k3[4]) and np.isnan(w[4])
    assert w[5] == 0.0


def test_null_outputs_skipped():
    a = torch.randn(100, device="cuda")
    b = torch.randn(100, device="cuda")
    lr = torch.full((100,), 7.0, device="cuda")
    k3 = torch.full((100,), 7.0, device="cuda")
    lib = tim.load_library()
    st = lib.tim_mismatch(a.data_ptr(), b.data_ptr(), 100, 2.0, lr.data_ptr(), None, None,
                          torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert torch.equal(lr, a - b) and (k3 == 7.0).all()


def _k3_exact(a32, b32):
    """K3 = e^d - 1 - d of the exact difference of two fp32 values, as a
    rational: the power series to d^16 (the remainder is below 1e-60 of the
    sum for |d| < 1e-2)."""
    d = Fraction(float(a32)) - Fraction(float(b32))
    term, total = d, Fraction(0)
    for n in range(2, 17):
        term = term * d / n
        total += term
    return total


def _tiny_delta_pairs():
    """Log-prob pairs whose difference is a few ulp (near -1 and -2) or a
    fixed small delta (+-2^-23, 1e-7, 1e-6, 1e-5)."""
    a, b = [], []
    for base in (-1.0, -2.0, -0.75, -1.5):
        b0 = np.float32(base)
        for k in range(1, 5):
            up, dn = b0, b0
            for _ in range(k):
                up = np.nextafter(up, np.float32(np.inf))
                dn = np.nextafter(dn, np.float32(-np.inf))
            a += [up, dn]
            b += [b0, b0]
    for base in (-1.0, -2.0, -3.7, -0.02):
        for d in (2.0 ** -23, -(2.0 ** -23), 1e-7, -1e-7, 1e-6, -1e-6, 1e-5, -1e-5):
            if np.float32(base + d) != np.float32(base):  # a delta below half an ulp of base rounds away
                b += [np.float32(base)]
                a += [np.float32(base + d)]
    return np.array(a, dtype=np.float32), np.array(b, dtype=np.float32)


def test_k3_relative_at_tiny_delta():
    """K3 where e^d - 1 - d cancels in fp32 (|d| down to one ulp of a
    log-prob near -1): the GPU value is the exact K3 (rational power series
    of the exact fp32 difference) rounded once, to within 2^-24 relative."""
    a, b = _tiny_delta_pairs()
    lr, k3, w = _run(a, b, 2.0)
    worst = 0.0
    for i in range(len(a)):
        ex = _k3_exact(a[i], b[i])
        assert ex > 0
        err = abs(Fraction(float(k3[i])) - ex) / ex
        worst = max(worst, float(err))
        assert err <= Fraction(2) ** -24 * (1 + Fraction(2) ** -20), (i, float(a[i]), float(b[i]), float(err))
        # and the ratio's weight from the exact difference
        assert abs(w[i] - math.exp(float(Fraction(float(a[i])) - Fraction(float(b[i]))))) <= 2.0 ** -23
    print(f"[k3 tiny delta] n={len(a)} max rel err vs exact = {worst:.3e} (one fp32 rounding = {2.0 ** -24:.3e})")


def test_k3_agrees_with_sequence_score():
    """A one-token response's K3 score (fp64) rounds to the token-level K3."""
    rng = np.random.default_rng(77)
    b = (-rng.exponential(2.0, 4096)).astype(np.float32)
    a = (b + rng.standard_normal(4096) * np.where(rng.random(4096) < 0.05, 0.3, 1e-6)).astype(np.float32)
    ag, bg = torch.as_tensor(a).cuda(), torch.as_tensor(b).cuda()
    _, k3, w = tim.mismatch(ag, bg, 2.0)
    cu = torch.arange(0, 4097, dtype=torch.int64, device="cuda")
    sc, keep, wt = tim.mismatch_seq(ag, bg, cu, C=2.0, tau_seq=1e30)
    assert bits_equal(sc.float(), k3)
    assert bits_equal(wt, w)
