"""GPU parity of the backward (tim_logprobs_backward, tim_logit_grads) against
the fp64 oracle, element by element, with the tolerance derived from the
arithmetic, plus its invariances: grad_hidden bitwise independent of the
batching, grad_w bitwise independent of the micro-batch size and continued
exactly by accumulation.

Tolerance. The GPU rounds each logit gradient once to bf16 (8 significant
bits, round to nearest even: relative error at most u = 2^-8) around an fp32
value that is itself within ~1e-6 relative of the exact one (recomputed logits
and lse), then accumulates bf16 x bf16 products in fp32 over K terms in 32-term
MFMA steps. Per output element c = sum_i x_i y_i the error is then at most
(2^-8 + (K / 32 + 32) 2^-24) * sum_i |x_i y_i| plus the fp32 gradient error;
the tests take 2^-8 + (K / 32 + 64) 2^-24 of the fp64 sum_i |x_i y_i| plus 1e-5
of its largest value. The bound is reached when one term dominates a sum (the
sampled token's gradient in a column of grad_w), so observed errors come close
to it; they cannot pass it."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from tim_testutil import bits_equal, inputs, random_tokens, require_gpu
from workload import bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _upstream(T, seed, entropy=True, device="cuda"):
    g = torch.Generator(device="cpu").manual_seed(7000 + seed)
    gl = torch.randn(T, generator=g, dtype=torch.float32)
    ge = torch.randn(T, generator=g, dtype=torch.float32) if entropy else None
    return gl.to(device), (ge.to(device) if ge is not None else None)


def _case(T, d, V, tau, seed, entropy=True, bad_tokens=False):
    h, W = inputs(T, d, V, seed=seed)
    tok = random_tokens(T, V, seed)
    if bad_tokens and T > 3:
        tok[1] = -1
        tok[3] = V
    lp, H, lse = tim.logprobs(h, W, tok, tau, lse=True)
    gl, ge = _upstream(T, seed, entropy)
    return h, W, tok, H, lse, gl, ge


def _oracle_dacc(h, W, tok, tau, gl, ge):
    return oracle.logit_grads(bf16_bits(h), bf16_bits(W), tok.cpu().numpy(), tau, gl.cpu().double().numpy(),
                              None if ge is None else ge.cpu().double().numpy())


def _bound_check(name, got, ref, mag, K):
    """|got - ref| <= (2^-8 + (K/32 + 64) 2^-24) mag + 1e-5 max(mag) elementwise."""
    got = got.double().cpu().numpy()
    c = 2.0 ** -8 + (K / 32 + 64) * 2.0 ** -24
    tol = c * mag + 1e-5 * mag.max()
    err = np.abs(got - ref)
    ratio = float((err / tol).max())
    rel = err / np.maximum(mag, 1e-30)
    print(f"[parity] {name}: n={got.size} max|err|={err.max():.3e} max err/tol={ratio:.3f} "
          f"median err/mag={np.median(rel):.2e}")
    assert np.isfinite(got).all(), f"{name}: non-finite output"
    assert ratio <= 1.0, f"{name}: error exceeds the derived bound ({ratio:.3f})"


@pytest.mark.parametrize("T,d,V,tau,entropy", [
    (300, 256, 4173, 1.0, True),
    (77, 128, 1000, 0.7, False),
    (513, 384, 2500, 1.3, True),
])
def test_logit_grads_vs_oracle(T, d, V, tau, entropy):
    print(f"case T={T} d={d} V={V} tau={tau} entropy={entropy}", flush=True)
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=T + V, entropy=entropy, bad_tokens=True)
    got = tim.logit_grads(h, W, tok, lse, gl, tau, entropy=H if entropy else None, grad_entropy=ge)
    torch.cuda.synchronize()
    v_pad = got.shape[1]
    assert v_pad % 256 == 0 and v_pad >= V
    assert (got[:, V:] == 0).all(), "entries past V must be zero"
    ref = _oracle_dacc(h, W, tok, tau, gl, ge)
    g = got[:, :V].double().cpu().numpy()
    # per-element scale of the terms that form it, from the oracle's own p, q, H
    from oracle.logprobs import logits as _z  # the oracle's fp64 logits (same inputs)
    z = _z(bf16_bits(h), bf16_bits(W), tau)
    m = z.max(axis=1, keepdims=True)
    q = z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))
    p = np.exp(q)
    Hr = -(p * q).sum(axis=1, keepdims=True)
    gabs = np.abs(gl.cpu().double().numpy())[:, None]
    eabs = np.zeros_like(gabs) if ge is None else np.abs(ge.cpu().double().numpy())[:, None]
    tk = tok.cpu().numpy().astype(np.int64)
    onehot = np.zeros_like(p)
    ok = (tk >= 0) & (tk < V)
    onehot[np.arange(T)[ok], tk[ok]] = 1.0
    scale = (gabs * (onehot + p) + eabs * p * (np.abs(q) + Hr)) / tau
    err = np.abs(g - ref)
    tol = 2.0 ** -8 * np.abs(ref) + 2e-5 * scale
    print(f"[parity] dlogits T={T} V={V}: max|err|={err.max():.3e} max err/tol={(err / tol).max():.3f}")
    assert (err <= tol).all()


@pytest.mark.parametrize("T,d,V,tau,mb,entropy", [
    (300, 256, 4173, 1.0, 128, True),
    (700, 640, 5000, 0.5, 256, True),
    (130, 128, 777, 2.0, 0, False),
    (1, 128, 300, 1.0, 0, True),
    (200, 8192, 1000, 0.3, 128, True),   # a long hidden chain, a sharp distribution
])
def test_backward_vs_oracle(T, d, V, tau, mb, entropy):
    print(f"case T={T} d={d} V={V} tau={tau} mb={mb} entropy={entropy}", flush=True)
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=3 * T + V, entropy=entropy, bad_tokens=True)
    gh, gw = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H if entropy else None, grad_entropy=ge,
                                   micro_batch=mb)
    # grad_w alone (the logit-gradient pass then writes only the weight pass's operand) gives the same bits
    _, gw_only = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H if entropy else None, grad_entropy=ge,
                                       micro_batch=mb, want_hidden=False)
    assert bits_equal(gw_only, gw)
    torch.cuda.synchronize()
    dacc = _oracle_dacc(h, W, tok, tau, gl, ge)
    hf = oracle.bf16_to_f64(bf16_bits(h))
    wf = oracle.bf16_to_f64(bf16_bits(W))
    v_pad = (V + 255) // 256 * 256
    t_all = (T + 127) // 128 * 128  # the weight-gradient chain runs over every token
    _bound_check(f"grad_hidden T={T} V={V}", gh, dacc @ wf, np.abs(dacc) @ np.abs(wf), v_pad)
    _bound_check(f"grad_w T={T} V={V}", gw, dacc.T @ hf, np.abs(dacc).T @ np.abs(hf), t_all)



@pytest.mark.parametrize("T,d,V,mb", [(1, 384, 1, 0), (129, 384, 255, 128), (300, 384, 257, 128),
                                      (513, 640, 129, 256)])
def test_backward_ragged_shapes_vs_oracle(T, d, V, mb):
    """The products read whole 256-row tiles of packed operands: hidden sizes that leave padding rows in the last
    tile (384, 640), vocabularies of one entry and around a tile edge, micro-batches that end inside a tile. Both
    gradients against the oracle within the derived bound."""
    print(f"case ragged T={T} d={d} V={V} mb={mb}", flush=True)
    h, W, tok, H, lse, gl, ge = _case(T, d, V, 0.9, seed=5 * T + V + d, bad_tokens=True)
    gh, gw = tim.logprobs_backward(h, W, tok, lse, gl, 0.9, entropy=H, grad_entropy=ge, micro_batch=mb)
    torch.cuda.synchronize()
    if V == 1:  # one entry: p = 1, q = 0, H = 0, so every logit gradient is exactly zero
        assert (gh == 0).all() and (gw == 0).all()
        return
    dacc = _oracle_dacc(h, W, tok, 0.9, gl, ge)
    hf = oracle.bf16_to_f64(bf16_bits(h))
    wf = oracle.bf16_to_f64(bf16_bits(W))
    v_pad = (V + 255) // 256 * 256
    step = mb if 0 < mb < T else T
    t_all = sum(-(-min(step, T - t0) // 128) * 128 for t0 in range(0, T, step))
    _bound_check(f"grad_hidden ragged T={T} d={d} V={V}", gh, dacc @ wf, np.abs(dacc) @ np.abs(wf), v_pad)
    _bound_check(f"grad_w ragged T={T} d={d} V={V}", gw, dacc.T @ hf, np.abs(dacc).T @ np.abs(hf), t_all)



def test_backward_maximum_vocabulary():
    """The largest vocabulary the boundary accepts (V = 2048 * 256: 2048 vocabulary tiles, the widest packed A
    operand of grad_hidden and B operand of grad_w): grad_hidden on every row and grad_w on 64 seeded vocabulary rows
    plus every token's row against the oracle, within the derived bound."""
    T, d, V, tau = 9, 128, 2048 * 256, 1.1
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=17)
    gh, gw = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge)
    torch.cuda.synchronize()
    dacc = _oracle_dacc(h, W, tok, tau, gl, ge)
    wf = oracle.bf16_to_f64(bf16_bits(W))
    hf = oracle.bf16_to_f64(bf16_bits(h))
    _bound_check("grad_hidden max-vocab", gh, dacc @ wf, np.abs(dacc) @ np.abs(wf), V)
    rng = np.random.default_rng(17)
    vrows = np.unique(np.concatenate([tok.cpu().numpy().astype(np.int64), rng.choice(V, 61, replace=False),
                                      [0, V - 1, V - 256]]))
    da = np.ascontiguousarray(dacc[:, vrows])
    _bound_check("grad_w max-vocab rows", torch.as_tensor(gw.double().cpu().numpy()[vrows]), da.T @ hf,
                 np.abs(da).T @ np.abs(hf), 128)


def test_backward_largest_pass():
    """A pass of 2^22 - 100 tokens, padded to 2^22 (the largest pass the boundary accepts, and the weight gradient's
    longest chain: its stage offsets reach 2^31 - 16 KB), gives bitwise the gradients of two passes of 2^21 tokens;
    grad_hidden on sampled rows against the oracle within the derived bound."""
    T, d, V, tau = 2 ** 22 - 100, 128, 256, 1.0
    h, W = inputs(T, d, V, seed=19, w_std=0.1)
    tok = random_tokens(T, V, 19)
    lp, H, lse = tim.logprobs(h, W, tok, tau, lse=True)
    gl, ge = _upstream(T, 19)
    gh0, gw0 = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=0)
    gh1, gw1 = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=2 ** 21)
    assert bits_equal(gh0, gh1) and bits_equal(gw0, gw1)
    assert torch.isfinite(gw0).all()
    rng = np.random.default_rng(19)
    rows = np.unique(np.concatenate([[0, 2 ** 21 - 1, 2 ** 21, T - 1], rng.choice(T, 60, replace=False)]))
    idx = torch.as_tensor(rows, device="cuda")
    hs, ts = h.index_select(0, idx), tok.index_select(0, idx)
    dacc = oracle.logit_grads(bf16_bits(hs), bf16_bits(W), ts.cpu().numpy(), tau,
                              gl.index_select(0, idx).cpu().double().numpy(), ge.index_select(0, idx).cpu().double().numpy())
    wf = oracle.bf16_to_f64(bf16_bits(W))
    _bound_check("grad_hidden largest pass", gh0.index_select(0, idx), dacc @ wf, np.abs(dacc) @ np.abs(wf), V)

@pytest.mark.parametrize("mb", [128, 256, 0])
def test_backward_ignores_stale_workspace(mb):
    """A workspace left full of NaN (bf16 0xFFFF) by earlier work gives bitwise the gradients of a zeroed one: the
    padding along K is written as zeros by the transposes and the logit-gradient pass, and the padding rows of the
    last packed tiles (here d = 384 of 512, and micro-batches ending inside a tile) reach only outputs that are
    never written. Micro-batches of 128 take the transpose of the logit gradients; one pass of 300 (padded to 384)
    has the logit-gradient pass write them transposed itself, token rows 300..383 as zeros; 256 + 44 takes one
    of each."""
    T, d, V = 300, 384, 1000
    h, W, tok, H, lse, gl, ge = _case(T, d, V, 1.0, seed=15)
    n = tim.backward_workspace_size(T, d, V, mb)
    got = []
    for fill in (255, 0):
        ws = torch.full((n,), fill, dtype=torch.uint8, device="cuda")
        got.append(tim.logprobs_backward(h, W, tok, lse, gl, 1.0, entropy=H, grad_entropy=ge, micro_batch=mb,
                                         workspace=ws))
    (gh_nan, gw_nan), (gh_zero, gw_zero) = got
    assert torch.isfinite(gh_nan).all() and torch.isfinite(gw_nan).all()
    assert bits_equal(gh_nan, gh_zero) and bits_equal(gw_nan, gw_zero)

def test_grad_hidden_is_batch_invariant_and_grad_w_micro_batch_invariant():
    T, d, V, tau = 700, 256, 4173, 0.8
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=11)
    ref_h, ref_w = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge)
    for mb in (128, 256, 384, 640):
        gh, gw = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=mb)
        assert bits_equal(gh, ref_h), f"grad_hidden changed with micro_batch={mb}"
        assert bits_equal(gw, ref_w), f"grad_w changed with micro_batch={mb}"
    # rows alone and at other offsets
    for a, b in [(0, 1), (5, 6), (250, 513), (699, 700)]:
        gh, _ = tim.logprobs_backward(h[a:b].contiguous(), W, tok[a:b].contiguous(), lse[a:b].contiguous(),
                                      gl[a:b].contiguous(), tau, entropy=H[a:b].contiguous(),
                                      grad_entropy=ge[a:b].contiguous(), want_w=False)
        assert bits_equal(gh, ref_h[a:b].contiguous()), f"grad_hidden rows [{a},{b}) changed"
    print("[invariance] backward: grad_hidden bitwise across micro-batches and row subsets; "
          "grad_w bitwise across micro-batches 0/128/256/384/640")


def test_grad_w_accumulation_continues_the_chain():
    """dW(first 256 rows) then += dW(next 444 rows) is bitwise dW(all 700 rows)."""
    T, d, V, tau = 700, 128, 2000, 1.0
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=12)
    _, ref_w = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, want_hidden=False)
    part = lambda a, b: dict(hidden=h[a:b].contiguous(), tokens=tok[a:b].contiguous(), lse=lse[a:b].contiguous(),
                             grad_logp=gl[a:b].contiguous(), entropy=H[a:b].contiguous(),
                             grad_entropy=ge[a:b].contiguous())
    buf = torch.full((V, d), float("nan"), dtype=torch.float32, device="cuda")
    p1 = part(0, 256)
    tim.logprobs_backward(p1["hidden"], W, p1["tokens"], p1["lse"], p1["grad_logp"], tau, entropy=p1["entropy"],
                          grad_entropy=p1["grad_entropy"], want_hidden=False, grad_w=buf)
    p2 = part(256, 700)
    tim.logprobs_backward(p2["hidden"], W, p2["tokens"], p2["lse"], p2["grad_logp"], tau, entropy=p2["entropy"],
                          grad_entropy=p2["grad_entropy"], want_hidden=False, grad_w=buf, accumulate=True)
    assert bits_equal(buf, ref_w)


def test_softmax_gradient_sums_to_zero():
    """sum_v dlogits = 0 per row, so sum_v grad_w[v, :] = 0 up to the rounding bound."""
    T, d, V, tau = 512, 256, 3000, 1.0
    h, W, tok, H, lse, gl, ge = _case(T, d, V, tau, seed=13)
    _, gw = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, want_hidden=False)
    dacc = _oracle_dacc(h, W, tok, tau, gl, ge)
    hf = oracle.bf16_to_f64(bf16_bits(h))
    mag = (np.abs(dacc).T @ np.abs(hf)).sum(axis=0)
    s = np.abs(gw.double().sum(dim=0).cpu().numpy())
    print(f"[invariant] max |sum_v grad_w| / sum_v |terms| = {(s / mag).max():.2e}")
    assert (s <= 2.0 ** -8 * mag).all()


def test_degenerate_calls():
    T, d, V = 64, 128, 500
    h, W, tok, H, lse, gl, ge = _case(T, d, V, 1.0, seed=14)
    # no upstream gradient: all zero
    z = torch.zeros_like(gl)
    gh, gw = tim.logprobs_backward(h, W, tok, lse, z, 1.0, entropy=H, grad_entropy=z)
    assert (gh == 0).all() and (gw == 0).all()
    # T == 0: grad_w is cleared unless accumulating
    buf = torch.full((V, d), 3.0, dtype=torch.float32, device="cuda")
    e = lambda *s, dt=torch.float32: torch.empty(*s, dtype=dt, device="cuda")
    tim.logprobs_backward(e(0, d, dt=torch.bfloat16), W, e(0, dt=torch.int32), e(0), e(0), 1.0, grad_w=buf,
                          want_hidden=False)
    assert (buf == 0).all()
    buf.fill_(3.0)
    tim.logprobs_backward(e(0, d, dt=torch.bfloat16), W, e(0, dt=torch.int32), e(0), e(0), 1.0, grad_w=buf,
                          want_hidden=False, accumulate=True)
    assert (buf == 3.0).all()
    # h = 0 rows: uniform softmax; grad_hidden = g (w_a - mean w) / tau, grad_w = 0
    h0 = torch.zeros_like(h)
    lp0, H0, lse0 = tim.logprobs(h0, W, tok, 1.0, lse=True)
    gh, gw = tim.logprobs_backward(h0, W, tok, lse0, gl, 1.0, entropy=H0, grad_entropy=ge)
    wf = W.double()
    exp = gl.double()[:, None] * (wf[tok.long()] - wf.mean(dim=0))
    err = (gh.double() - exp).abs().max().item()
    print(f"[parity] uniform rows: max|grad_hidden - g (w_a - mean w)| = {err:.2e}")
    assert err <= 2.0 ** -8 * 2 * wf.abs().max().item() * gl.abs().max().item()
    assert (gw == 0).all()


def test_persistent_backward_full_vocab():
    """The backward at the headline shape (d = 4096, V = 151936) with micro-batches of 4352 tokens and a ragged
    second one (T = 4613): every pass runs on the persistent grid (logit gradients: 594 x 17 tiles; grad_hidden:
    16 x 17 tiles; grad_w: 16 x 594 tiles, a workgroup walking ~37 of them), and the second micro-batch's grad_w
    pass resumes each tile from the value the first stored. Checked element by element against the oracle:
    grad_w on the row of every sampled token plus 64 seeded vocabulary rows (the first, the last, the tail tile),
    grad_hidden on 256 seeded rows (both micro-batches' edges included), each within the derived bound."""
    T, d, V, tau, mb = 4613, 4096, 151936, 1.0, 4352
    print(f"case T={T} d={d} V={V} mb={mb}", flush=True)
    h, W = inputs(T, d, V, seed=31, w_std=0.02)
    tok = random_tokens(T, V, 31)
    lp, H, lse = tim.logprobs(h, W, tok, tau, lse=True)
    gl, ge = _upstream(T, 31)
    gh, gw = tim.logprobs_backward(h, W, tok, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=mb)
    torch.cuda.synchronize()
    gh_n, gw_n = gh.double().cpu().numpy(), gw.double().cpu().numpy()
    del gh, gw
    print("[persistent backward] GPU done; oracle logit gradients of every row", flush=True)
    dacc = oracle.logit_grads(bf16_bits(h), bf16_bits(W), tok.cpu().numpy(), tau, gl.cpu().double().numpy(),
                              ge.cpu().double().numpy(), row_block=1024)
    rng = np.random.default_rng(31)
    vrows = np.unique(np.concatenate([tok.cpu().numpy().astype(np.int64), rng.choice(V, 61, replace=False),
                                      [0, V - 1, V - 100]]))
    hf = oracle.bf16_to_f64(bf16_bits(h))
    da_v = np.ascontiguousarray(dacc[:, vrows])
    t_all = (mb + 127) // 128 * 128 + (T - mb + 127) // 128 * 128  # the chain over both micro-batches' padded tokens
    _bound_check(f"grad_w on {len(vrows)} vocabulary rows (persistent, resumed)", torch.as_tensor(gw_n[vrows]),
                 da_v.T @ hf, np.abs(da_v).T @ np.abs(hf), t_all)
    trows = np.unique(np.concatenate([rng.choice(T, 250, replace=False), [0, mb - 1, mb, T - 1, 255, 256]]))
    wf = oracle.bf16_to_f64(bf16_bits(W))
    da_t = dacc[trows]
    del dacc
    v_pad = (V + 255) // 256 * 256
    _bound_check(f"grad_hidden on {len(trows)} rows (persistent)", torch.as_tensor(gh_n[trows]), da_t @ wf,
                 np.abs(da_t) @ np.abs(wf), v_pad)
