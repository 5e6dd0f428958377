"""tim_mismatch_seq on the GPU: sequence scores, keep mask and token weights
against the fp64 oracle; fixed-order (position-invariant) scores; edge cases."""

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Estimator
from tim_testutil import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _stream(seed, lens, scale=1e-3, tail=0.02):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T = int(cu[-1])
    b = (-rng.exponential(2.0, T)).astype(np.float32)
    # mostly tiny discrepancies, a few large ones (the paper's heavy tail)
    a = (b + rng.standard_normal(T) * np.where(rng.random(T) < tail, 0.3, scale)).astype(np.float32)
    return a, b, cu


def _gpu_run(a, b, cu, est, C, tau):
    ag = torch.as_tensor(a).cuda()
    bg = torch.as_tensor(b).cuda()
    cg = torch.as_tensor(cu).cuda()
    s, k, w = tim.mismatch_seq(ag, bg, cg, C=C, tau_seq=tau, estimator=est)
    return s.cpu().numpy(), k.cpu().numpy().astype(bool), w.cpu().double().numpy()


def _check(a, b, cu, est, C, tau):
    name = "k1" if est == Estimator.K1 else "k3"
    s, k, w = _gpu_run(a, b, cu, est, C, tau)
    rs, rk, rw = oracle.mismatch_seq(a, b, cu, name, C, tau)
    d = a.astype(np.float64) - b.astype(np.float64)
    per = np.abs(-d if name == "k1" else np.expm1(d) - d)
    mag = np.array([per[cu[j]:cu[j + 1]].sum() for j in range(len(cu) - 1)])
    # fp64 terms (a few ulp each) summed in another order: ~1e-16 * length * magnitude; for K3 also the
    # oracle's own fp64 expm1(d) - d, off by up to 2^-52 |expm1(d)| per term (the kernel's K3 terms are
    # accurate to ~2^-50 relative however small d is)
    oerr = np.zeros(len(cu) - 1)
    if name == "k3":
        te = 2.0 ** -52 * np.abs(np.expm1(d))
        oerr = np.array([te[cu[j]:cu[j + 1]].sum() for j in range(len(cu) - 1)])
    tol = 1e-13 * mag * np.maximum(1, np.diff(cu)) + oerr + 1e-300
    assert np.all(np.abs(s - rs) <= tol), np.max(np.abs(s - rs) / np.maximum(tol, 1e-300))
    # keep: the same decision wherever the score is not within the tolerance of tau
    clear = np.abs(rs - tau) > tol
    assert (k[clear] == rk[clear]).all()
    # weights: fp32 min(exp(delta), C), zero in rejected responses
    seg = np.repeat(np.arange(len(cu) - 1), np.diff(cu))
    kept = k[seg]
    assert (w[~kept] == 0).all()
    wr = np.minimum(np.exp(d), C)
    assert np.all(np.abs(w[kept] - wr[kept]) <= 1e-6 * wr[kept])
    return s, k, w, rs, rk


@pytest.mark.parametrize("est", [Estimator.K1, Estimator.K3])
@pytest.mark.parametrize("lens", [[5], [0, 1, 255, 256, 257, 0, 1000], [16384, 3, 4096], list(range(0, 600, 37))])
def test_vs_oracle(est, lens):
    a, b, cu = _stream(len(lens) * 7 + int(est), lens)
    for tau in (1e-3, 1e-2, 0.0):
        _check(a, b, cu, est, 2.0, tau)
    _check(a, b, cu, est, 0.7, 1e-3)


def test_position_invariance_bitwise():
    """A response's score and weights do not depend on where it sits in the
    stream or what else is in the launch."""
    rng = np.random.default_rng(5)
    lens = rng.integers(0, 3000, size=40)
    a, b, cu = _stream(9, lens)
    s, k, w = _gpu_run(a, b, cu, Estimator.K3, 2.0, 1e-3)
    for j in [0, 7, 23, 39]:
        s0, s1 = cu[j], cu[j + 1]
        # alone
        sj, kj, wj = _gpu_run(a[s0:s1].copy(), b[s0:s1].copy(), np.array([0, s1 - s0]), Estimator.K3, 2.0, 1e-3)
        assert sj[0] == s[j] and kj[0] == k[j] and (wj == w[s0:s1]).all()
        # behind a ragged prefix of other tokens
        pre = int(rng.integers(1, 999))
        a2 = np.concatenate([a[:pre], a[s0:s1]])
        b2 = np.concatenate([b[:pre], b[s0:s1]])
        s2, _, w2 = _gpu_run(a2, b2, np.array([0, pre, pre + s1 - s0]), Estimator.K3, 2.0, 1e-3)
        assert s2[1] == s[j] and (w2[pre:] == w[s0:s1]).all()


def test_identical_inputs_and_nan():
    x = (-np.random.default_rng(1).exponential(3.0, 5000)).astype(np.float32)
    cu = np.array([0, 0, 1, 4096, 5000], dtype=np.int64)
    for est in (Estimator.K1, Estimator.K3):
        s, k, w = _gpu_run(x, x, cu, est, 2.0, 1e-3)
        assert (s == 0).all() and k.all() and (w == 1.0).all()
    y = x.copy()
    y[4500] = np.nan
    s, k, w = _gpu_run(y, x, cu, Estimator.K3, 2.0, 1e-3)
    assert np.isnan(s[3]) and not k[3] and (w[4096:] == 0).all()
    assert k[:3].all() and (w[:4096] == 1.0).all()


def test_malformed_offsets_are_clamped():
    """Offsets past T or decreasing give empty responses; nothing outside the
    arrays is touched (the sentinel weights stay put)."""
    a, b, _ = _stream(2, [100])
    ag, bg = torch.as_tensor(a).cuda(), torch.as_tensor(b).cuda()
    cu = torch.tensor([0, 60, 40, 100, 250, -5], dtype=torch.int64, device="cuda")
    score = torch.full((5,), 7.0, dtype=torch.float64, device="cuda")
    keep = torch.full((5,), 9, dtype=torch.uint8, device="cuda")
    w = torch.full((100,), -1.0, dtype=torch.float32, device="cuda")
    tim.mismatch_seq(ag, bg, cu, out=(score, keep, w))
    s = score.cpu().numpy()
    rs, _, _ = oracle.mismatch_seq(a, b, [0, 60], "k3", 2.0, 1e-3)
    assert abs(s[0] - rs[0]) <= 1e-12 * abs(rs[0]) + 1e-300
    # [60, 40) reversed -> empty; [40, 100) valid; [100, 250) clamped to empty; [250, -5) empty
    assert s[1] == 0 and s[3] == 0 and s[4] == 0
    rs2, _, _ = oracle.mismatch_seq(a, b, [40, 100], "k3", 2.0, 1e-3)
    assert abs(s[2] - rs2[0]) <= 1e-12 * abs(rs2[0]) + 1e-300
    assert (keep.cpu().numpy() <= 1).all()


def test_no_responses_is_noop():
    a = torch.zeros(4, dtype=torch.float32, device="cuda")
    cu = torch.zeros(1, dtype=torch.int64, device="cuda")
    s, k, w = tim.mismatch_seq(a, a, cu)
    assert s.numel() == 0 and k.numel() == 0 and (w == 0).all()
