"""GPU parity of the final RMS norm (tim_rmsnorm, tim_rmsnorm_backward) against
the fp64 oracle, its batch invariance, and the norm feeding the LM head.

Rounding decisions. The kernel rounds the normalised row (and its product with
the weight) to bf16 from fp32 values; the oracle rounds the same quantities
from fp64. The two agree except where the fp32 and fp64 values straddle a bf16
rounding boundary; there the codes differ by one unit in the last place. The
tests require every code to match or be such a neighbour, and nearly all to
match.

Tolerances (fp32 arithmetic, unit roundoff u = 2^-24): the sum of squares runs
as d/64 chained terms per lane and a 6-level tree, so rstd is within
((d/64 + 8)/2 + 2) u relative; the backward row sum likewise, giving
|d grad_x| <= (d/64 + 64) u (r |g G| + r^3 |x| sum|G g x| / d); grad_gamma sums
256-row blocks in order and then the blocks: (256 + T/256 + 32) u sum_t |G x r|."""

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from tim_testutil import TOL_ENT, TOL_LOGP, bits_equal, check_close, inputs, random_tokens, require_gpu
from workload import bf16_bits

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _x(T, d, seed, scale=2.0):
    g = torch.Generator(device="cpu").manual_seed(9000 + seed)
    return (torch.randn(T, d, generator=g) * scale).to(torch.bfloat16).cuda()


def _gamma(d, seed):
    g = torch.Generator(device="cpu").manual_seed(9500 + seed)
    return (1.0 + 0.3 * torch.randn(d, generator=g)).to(torch.bfloat16).cuda()


def _check_codes(name, got_bits, ref_bits, n=None, gamma_bits=None):
    """Every code equals the oracle's, or comes from the other rounding of a
    normalised value that straddles a boundary: without a weight that is the
    neighbouring code; with one, the weight times either neighbour of the
    oracle's inner code, rounded (which can land two codes away)."""
    got = got_bits.astype(np.int32)
    ref = ref_bits.astype(np.int32)
    diff = got != ref
    if gamma_bits is None:
        ok = (((got ^ ref) & 0x8000) == 0) & (np.abs((got & 0x7FFF) - (ref & 0x7FFF)) == 1)
        valid = ok[diff]
    else:
        rows, cols = np.nonzero(diff)
        inner = oracle.f64_to_bf16_bits(oracle.round_bf16(n[rows, cols])).astype(np.int32)
        sign, mag = inner & 0x8000, inner & 0x7FFF
        gw = oracle.bf16_to_f64(gamma_bits)[cols]
        cands = []
        for m2 in (mag - 1, mag + 1):
            v = oracle.bf16_to_f64((sign | np.clip(m2, 0, 0x7F7F)).astype(np.uint16))
            cands.append(oracle.f64_to_bf16_bits(oracle.round_bf16(gw * v)).astype(np.int32))
        g = got[rows, cols]
        valid = (g == cands[0]) | (g == cands[1])
    frac = diff.mean()
    print(f"[parity] {name}: {diff.sum()} of {diff.size} bf16 codes differ from the oracle's, all from the other "
          f"rounding of a straddling value: {bool(valid.all())}")
    assert valid.all(), f"{name}: a code is neither the oracle's nor the other valid rounding"
    assert frac <= 1e-3, f"{name}: {frac:.2e} of the codes differ"


@pytest.mark.parametrize("T,d,with_gamma,eps", [(300, 640, True, 1e-6), (77, 200, False, 1e-5),
                                                (4096, 4096, True, 1e-6), (1, 8, True, 0.0),
                                                (257, 2048, False, 1e-6), (129, 5120, True, 1e-6),
                                                (33, 8192, True, 1e-6)])
def test_rmsnorm_vs_oracle(T, d, with_gamma, eps):
    print(f"case T={T} d={d} gamma={with_gamma} eps={eps}", flush=True)
    x = _x(T, d, T + d)
    g = _gamma(d, d) if with_gamma else None
    h, rstd = tim.rmsnorm(x, g, eps)
    torch.cuda.synchronize()
    gb = None if g is None else bf16_bits(g)
    ref_h, ref_r, ref_n = oracle.rmsnorm(bf16_bits(x), gb, eps)
    _check_codes(f"h T={T} d={d}", bf16_bits(h), ref_h, ref_n, gb)
    rel = np.abs(rstd.double().cpu().numpy() - ref_r) / ref_r
    bound = ((d / 64 + 8) / 2 + 2) * U
    print(f"[parity] rstd: max rel err {rel.max():.2e} bound {bound:.2e}")
    assert (rel <= bound).all()


def test_rmsnorm_batch_invariance_and_unit_weight():
    T, d = 1000, 1024
    x = _x(T, d, 1)
    g = _gamma(d, 1)
    h, r = tim.rmsnorm(x, g)
    for a, b in [(0, 1), (17, 18), (300, 777), (999, 1000)]:
        hs, rs = tim.rmsnorm(x[a:b].contiguous(), g)
        assert torch.equal(hs.view(torch.int16), h[a:b].view(torch.int16))
        assert bits_equal(rs, r[a:b].contiguous())
    h1, _ = tim.rmsnorm(x, None)
    ho, _ = tim.rmsnorm(x, torch.ones(d, dtype=torch.bfloat16, device="cuda"))
    assert torch.equal(h1.view(torch.int16), ho.view(torch.int16))


def test_norm_feeds_the_lm_head():
    """logp / entropy of the normalised rows against the oracle's norm and log-probs."""
    T, d, V, tau = 260, 256, 3000, 0.9
    x = _x(T, d, 5, scale=1.5)
    g = _gamma(d, 5)
    _, W = inputs(1, d, V, seed=5)
    tok = random_tokens(T, V, 5)
    lp, ent, lse, h, rstd = tim.logprobs_from_residual(x, g, W, tok, eps=1e-6, temperature=tau, entropy=True)
    ref_h, _, _ = oracle.rmsnorm(bf16_bits(x), bf16_bits(g), 1e-6)
    ref_lp, ref_H = oracle.logprobs(ref_h, bf16_bits(W), tok.cpu().numpy(), tau)
    check_close("logp after the norm", lp, ref_lp, TOL_LOGP)
    check_close("entropy after the norm", ent, ref_H, TOL_ENT)


# 2048, 4096 and 5120 keep the row in registers between the passes; the others reread it
@pytest.mark.parametrize("T,d,with_gamma", [(300, 640, True), (513, 256, False), (1, 8, True), (257, 2048, True),
                                            (130, 4096, False), (66, 5120, True), (40, 8192, True)])
def test_rmsnorm_backward_vs_oracle(T, d, with_gamma):
    print(f"case T={T} d={d} gamma={with_gamma}", flush=True)
    x = _x(T, d, 3 * T + d)
    g = _gamma(d, 2 * d) if with_gamma else None
    eps = 1e-6
    _, rstd = tim.rmsnorm(x, g, eps)
    G = torch.randn(T, d, generator=torch.Generator(device="cpu").manual_seed(T)).cuda()
    gx, gg = tim.rmsnorm_backward(x, g, rstd, G)
    torch.cuda.synchronize()
    gb = None if g is None else bf16_bits(g)
    Gn = G.double().cpu().numpy()
    dx, dg = oracle.rmsnorm_grads(bf16_bits(x), gb, eps, Gn)
    xf = oracle.bf16_to_f64(bf16_bits(x))
    gf = np.ones(d) if g is None else oracle.bf16_to_f64(gb)
    r = 1.0 / np.sqrt((xf * xf).mean(axis=1) + eps)
    s_abs = np.abs(Gn * gf[None, :] * xf).sum(axis=1)
    mag_x = r[:, None] * np.abs(gf[None, :] * Gn) + (r ** 3 * s_abs / d)[:, None] * np.abs(xf)
    err_x = np.abs(gx.double().cpu().numpy() - dx)
    rx = (err_x / ((d / 64 + 64) * U * mag_x + 1e-30)).max()
    mag_g = np.abs(Gn * xf * r[:, None]).sum(axis=0)
    err_g = np.abs(gg.double().cpu().numpy() - dg)
    rg = (err_g / ((256 + T / 256 + 32) * U * mag_g + 1e-30)).max()
    print(f"[parity] rmsnorm backward T={T} d={d}: grad_x max err/bound {rx:.3f}, grad_gamma max err/bound {rg:.3f}")
    assert rx <= 1.0 and rg <= 1.0
    # rows alone give the same grad_x bits; grad_gamma accumulates onto its buffer
    gx1, _ = tim.rmsnorm_backward(x[:1].contiguous(), g, rstd[:1].contiguous(), G[:1].contiguous(), want_gamma=False)
    assert bits_equal(gx1, gx[:1].contiguous())
    buf = gg.clone()
    tim.rmsnorm_backward(x, g, rstd, G, want_x=False, grad_gamma=buf, accumulate=True)
    torch.cuda.synchronize()
    assert torch.allclose(buf, 2 * gg, rtol=1e-6, atol=0)


def test_rmsnorm_degenerate_calls():
    d = 64
    buf = torch.full((d,), 5.0, device="cuda")
    e = torch.empty(0, d, dtype=torch.bfloat16, device="cuda")
    tim.rmsnorm_backward(e, None, torch.empty(0, device="cuda"), torch.empty(0, d, device="cuda"), want_x=False,
                         grad_gamma=buf)
    assert (buf == 0).all()
    buf.fill_(5.0)
    tim.rmsnorm_backward(e, None, torch.empty(0, device="cuda"), torch.empty(0, d, device="cuda"), want_x=False,
                         grad_gamma=buf, accumulate=True)
    assert (buf == 5.0).all()
    h, r = tim.rmsnorm(e)
    assert h.shape == (0, d) and r.shape == (0,)


@pytest.mark.parametrize("d,with_gamma,T", [(2048, True, 65536 + 77), (4096, False, 65536 + 77),
                                            (4096, True, 131072 + 77), (2048, False, 262144 + 77)])
def test_rmsnorm_backward_large_call_vs_oracle(d, with_gamma, T):
    """Calls of at least 65536 rows at d = 2048 / 4096 form grad_gamma's block
    sums in the grad_x pass (each wave's rows in order, then (q0 + q1) + (q2 +
    q3) per block; above 131072 rows at d = 4096, 262144 at d = 2048, a wave
    takes more than 64 rows): grad_gamma against the oracle within its bound, grad_x bitwise equal
    to the same rows evaluated alone (the smaller call's path) and to the
    oracle on sampled rows, and grad_gamma without grad_x the same bits."""
    print(f"case large T={T} d={d} gamma={with_gamma}", flush=True)
    x = _x(T, d, d + 7)
    g = _gamma(d, d + 8) if with_gamma else None
    eps = 1e-6
    _, rstd = tim.rmsnorm(x, g, eps)
    G = torch.randn(T, d, generator=torch.Generator(device="cuda").manual_seed(d), device="cuda")
    gx, gg = tim.rmsnorm_backward(x, g, rstd, G)
    _, gg_only = tim.rmsnorm_backward(x, g, rstd, G, want_x=False)
    torch.cuda.synchronize()
    assert bits_equal(gg_only, gg)
    rows = [0, 1, 255, 256, 4097, 65535, T - 1]
    for r in rows:
        gx1, _ = tim.rmsnorm_backward(x[r:r + 1].contiguous(), g, rstd[r:r + 1].contiguous(), G[r:r + 1].contiguous(),
                                      want_gamma=False)
        assert bits_equal(gx1, gx[r:r + 1].contiguous())
    gb = None if g is None else bf16_bits(g)
    # the oracle over row chunks: grad_x rows are independent and grad_gamma is
    # the sum of the chunks' column sums
    dg = np.zeros(d)
    mag_g = np.zeros(d)
    err_x = 0.0
    dx_max = 0.0
    for c0 in range(0, T, 16384):
        c1 = min(T, c0 + 16384)
        xb = bf16_bits(x[c0:c1])
        Gn = G[c0:c1].double().cpu().numpy()
        dx_c, dg_c = oracle.rmsnorm_grads(xb, gb, eps, Gn)
        dg += dg_c
        xf = oracle.bf16_to_f64(xb)
        r_ = 1.0 / np.sqrt((xf * xf).mean(axis=1) + eps)
        mag_g += np.abs(Gn * xf * r_[:, None]).sum(axis=0)
        sel = [r - c0 for r in rows if c0 <= r < c1]
        if sel:
            got = gx[c0:c1].double().cpu().numpy()[sel]
            err_x = max(err_x, float(np.abs(got - dx_c[sel]).max()))
            dx_max = max(dx_max, float(np.abs(dx_c[sel]).max()))
    err_g = np.abs(gg.double().cpu().numpy() - dg)
    rg = (err_g / ((256 + T / 256 + 32) * U * mag_g + 1e-30)).max()
    err_x /= dx_max
    print(f"[parity] large rmsnorm backward T={T} d={d}: grad_gamma max err/bound {rg:.2e}, "
          f"grad_x max rel err {err_x:.2e}")
    assert rg <= 1.0 and err_x <= 1e-5
