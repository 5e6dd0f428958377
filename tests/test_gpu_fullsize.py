"""Full-size workloads on the GPU, in the launch configurations the benchmark
uses, checked against the fp64 oracle on seeded row samples, plus bitwise
batch invariance across every batching the workloads name and the
controlled-mismatch report between the invariant path and the split-K4 engine.

Shapes (synthetic, seeded; see workload.gen):
  small  d=2048, V=151936, 16 responses U[128,1024] packed, one training call
  mid    d=4096, V=151936, 64 responses U[512,4096] packed, micro-batches of 16384
  stress the mid stream evaluated in rollout groupings of random size 1..256
         (shuffled) and training micro-batches 4096 / 16384 / 65536; split-K4
         engine supplies the second log-probs for the mismatch statistics
  long   d=5120, V=152064, 8 x 16384 tokens, tau = 0.7, micro-batches of 32768
         and rollout decode batches of 64
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode, Order
from tim_testutil import TOL_ENT, TOL_LOGP, TOL_W_REL, bits_equal, check_close, require_gpu
from workload import CONFIGS, bf16_bits, hidden_states, logprob_pairs, uniforms, vocab_weights
from workload.gen import seeds
from workload.sampler import sample_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


_cache = {}


def workload(name):
    """Inputs of a named configuration, drawn once per test session on the GPU."""
    if name in _cache:
        return _cache[name]
    _cache.clear()
    torch.cuda.empty_cache()
    cfg = CONFIGS[name]
    hs, ws, us = seeds(cfg)
    T = cfg.tokens
    print(f"[fullsize] drawing {name}: T={T} d={cfg.d} V={cfg.V} tau={cfg.temperature}", flush=True)
    h = hidden_states(T, cfg.d, hs, device="cuda")
    W = vocab_weights(cfg.V, cfg.d, cfg.w_std, ws, device="cuda")
    tok = sample_tokens(h, W, cfg.temperature, uniforms(T, us), dtype=torch.float32)
    torch.cuda.synchronize()
    _cache[name] = (cfg, h, W, tok)
    return _cache[name]


def oracle_sample(cfg, h, W, tok, lp, H, seed=7):
    """The oracle on the configuration's seeded row sample (cfg.oracle_rows: 2048 rows of the mid
    workload, 256 of the others)."""
    T = h.shape[0]
    rows = np.sort(np.random.default_rng(seed).choice(T, size=min(cfg.oracle_rows, T), replace=False))
    idx = torch.as_tensor(rows, device="cuda")
    print(f"[fullsize] {cfg.name}: oracle on {len(rows)} sampled rows", flush=True)
    ref_lp, ref_H = oracle.logprobs(bf16_bits(h.index_select(0, idx)), bf16_bits(W),
                                    tok.index_select(0, idx).cpu().numpy(), cfg.temperature, row_block=1024)
    check_close(f"{cfg.name} logp ({len(rows)} sampled rows)", lp, ref_lp, TOL_LOGP, rows)
    check_close(f"{cfg.name} entropy ({len(rows)} sampled rows)", H, ref_H, TOL_ENT, rows)
    # statistical pins of the sampled workload: E[logp(sampled)] = -E[H]
    lpn, Hn = lp.double().cpu().numpy(), H.double().cpu().numpy()
    assert abs(lpn.mean() + Hn.mean()) < 6 * lpn.std() / math.sqrt(T)
    assert (Hn >= 0).all() and (Hn <= math.log(cfg.V) + 1e-4).all() and (lpn <= 1e-6).all()
    return ref_lp, ref_H


def test_small_one_packed_call():
    cfg, h, W, tok = workload("small")
    lp, H, _ = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=0)
    oracle_sample(cfg, h, W, tok, lp, H)


def test_mid_micro_batches():
    cfg, h, W, tok = workload("mid")
    lp, H, _ = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=cfg.micro_batch)
    oracle_sample(cfg, h, W, tok, lp, H)
    # mean entropy of this synthetic workload: ln V - sigma_z^2 / 2, sigma_z = 0.02 sqrt(d)
    sig2 = (0.02 ** 2) * cfg.d
    assert abs(H.double().mean().item() - (math.log(cfg.V) - sig2 / 2)) < 0.05


def test_mid_backward():
    """The backward at the mid shape (d=4096, V=151936) on the first 20000 tokens
    (a full 16384-token micro-batch and a ragged one): sampled grad_hidden rows
    against the oracle within the derived bound, grad_hidden and grad_w bitwise
    across micro-batch sizes, and sum_v grad_w[v, :] = 0 within its bound."""
    cfg, h, W, tok = workload("mid")
    T, d, V, tau = 20000, cfg.d, cfg.V, cfg.temperature
    hs, ts = h[:T].contiguous(), tok[:T].contiguous()
    _, H, lse = tim.logprobs(hs, W, ts, tau, micro_batch=16384, lse=True)
    g = torch.Generator(device="cpu").manual_seed(99)
    gl = torch.randn(T, generator=g).cuda()
    ge = (0.1 * torch.randn(T, generator=g)).cuda()
    gh, gw = tim.logprobs_backward(hs, W, ts, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=16384)
    gh2, gw2 = tim.logprobs_backward(hs, W, ts, lse, gl, tau, entropy=H, grad_entropy=ge, micro_batch=4096)
    assert bits_equal(gh, gh2) and bits_equal(gw, gw2)
    torch.cuda.synchronize()
    wf = oracle.bf16_to_f64(bf16_bits(W))
    v_pad = (V + 255) // 256 * 256
    c = 2.0 ** -8 + (v_pad / 32 + 64) * 2.0 ** -24
    rows = np.sort(np.random.default_rng(3).choice(T, size=4, replace=False))
    worst = 0.0
    for r in rows:
        dacc = oracle.logit_grads(bf16_bits(hs[r:r + 1]), bf16_bits(W), ts[r:r + 1].cpu().numpy(), tau,
                                  gl[r:r + 1].double().cpu().numpy(), ge[r:r + 1].double().cpu().numpy())
        ref = (dacc @ wf)[0]
        mag = (np.abs(dacc) @ np.abs(wf))[0]
        err = np.abs(gh[r].double().cpu().numpy() - ref)
        worst = max(worst, float((err / (c * mag + 1e-5 * mag.max())).max()))
    print(f"[parity] mid grad_hidden on {len(rows)} sampled rows: max err/bound = {worst:.3f}")
    assert worst <= 1.0
    # sum_v dlogits = 0 per row: |sum_v grad_w[v, k]| <= c_w sum_t sum_v |dlogits| |h_tk|, and
    # sum_v |dlogits_tv| <= (2 |g_t| + 2 |e_t| log V) / tau (sum_v p |q + H| <= 2 H <= 2 log V)
    cw = 2.0 ** -8 + ((T + 127) // 128 * 128 / 32 + 64) * 2.0 ** -24
    row_l1 = (2 * gl.double().abs() + 2 * ge.double().abs() * math.log(V)) / tau
    bound = cw * (row_l1[:, None] * hs.double().abs()).sum(dim=0)
    colsum = gw.double().sum(dim=0).abs()
    print(f"[invariant] mid: max |sum_v grad_w| / bound = {(colsum / bound).max().item():.2e}")
    assert (colsum <= bound).all()
    assert torch.isfinite(gw).all()


def test_stress_invariance_and_mismatch_report():
    cfg, h, W, tok = workload("stress")
    T = h.shape[0]
    ref = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=16384, lse=True)
    for mb in (4096, 65536):
        out = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=mb, lse=True)
        for x, y in zip(out, ref):
            assert bits_equal(x, y), f"micro-batch {mb} differs"
    # training micro-batches above 16384 rows run as 16384-row launches at d = 4096; launches of other sizes:
    # rollout mode's one launch over the whole stream, and a two-stage launch of the first 65536 rows
    out = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.ROLLOUT, lse=True)
    for x, y in zip(out, ref):
        assert bits_equal(x, y), "one launch over the stream differs"
    n = 65536
    ws = torch.empty(tim.workspace_size(n, h.shape[1], W.shape[0], Mode.ROLLOUT), dtype=torch.uint8, device="cuda")
    tim.logprobs_partials(h[:n], W, tok[:n], ws, cfg.temperature, mode=Mode.TRAINING)
    part = tuple(torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(3))
    tim.logprobs_merge(ws, tok[:n], W.shape[0], out=part)
    for x, y in zip(part, ref):
        assert bits_equal(x, y[:n].contiguous()), "a 65536-row launch differs"
    del ws
    # rollout: every row once, in shuffled decode batches of random size 1..256
    rng = np.random.default_rng(44)
    perm = torch.as_tensor(rng.permutation(T), device="cuda")
    got = [torch.empty_like(ref[i]) for i in range(3)]
    i = calls = 0
    while i < T:
        n = int(rng.integers(1, 257))
        rows = perm[i:i + n]
        out = tim.logprobs(h.index_select(0, rows), W, tok.index_select(0, rows), cfg.temperature,
                           mode=Mode.ROLLOUT, lse=True)
        for g, o in zip(got, out):
            g[rows] = o
        i += n
        calls += 1
    for x, y in zip(got, ref):
        assert bits_equal(x, y), "rollout groupings differ from training"
    oracle_sample(cfg, h, W, tok, ref[0], ref[1], seed=9)
    print(f"[stress] {calls} rollout calls + micro-batches 4096/16384/65536 + launches of {T} and 65536 rows: "
          f"all {T} rows bitwise equal")
    # second engine: split-K4 reduction order
    eng = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=16384, order=Order.SPLITK4)
    oracle_sample(cfg, h, W, tok, eng[0], eng[1], seed=8)
    lr, k3, w = tim.mismatch(ref[0], eng[0], 2.0)
    d = lr.abs().double()
    q = torch.quantile(d[: 1 << 24].float(), torch.tensor([0.5, 0.99], device="cuda")).tolist()
    print(f"[stress] |dlogp| p50={q[0]:.3e} p99={q[1]:.3e} max={d.max().item():.3e}; mean k3="
          f"{k3.double().mean().item():.3e}; IS weight (C=2) mean={w.double().mean().item():.9f} "
          f"min={w.min().item():.7f} max={w.max().item():.7f}; rows differing in bits: "
          f"{(lr != 0).double().mean().item():.3f}")
    # mean K3 two ways on the path: the token-level fp32 values averaged, and the fp64 sequence score of the
    # whole stream as one response over T; each token's value is that term rounded once, so they agree to ~2^-24
    whole = torch.tensor([0, T], dtype=torch.int64, device="cuda")
    sc_all, _, _ = tim.mismatch_seq(ref[0], eng[0], whole, C=2.0, tau_seq=1e30)
    m_tok, m_seq = k3.double().mean().item(), sc_all.item() / T
    print(f"[stress] mean k3: token-level {m_tok:.9e}, sequence-level fp64 {m_seq:.9e}")
    assert abs(m_tok - m_seq) <= 1e-6 * m_seq
    # the engines agree within the oracle tolerance, so every weight is within 2e-3 of 1
    assert d.max().item() < 2 * TOL_LOGP
    assert ((w - 1).abs() <= 2 * TOL_W_REL).all()
    # the statistics of the two engines' log-probs follow from their difference
    assert torch.equal(lr, ref[0] - eng[0])
    assert ((w.double() - torch.clamp(torch.exp(lr.double()), max=2.0)).abs() <= TOL_W_REL * w.double()).all()
    # the mismatch stages at this size against the oracle, on seeded streams of the same length with the
    # paper's heavy-tailed discrepancies (inputs drawn by the workload module, not by the path)
    a_np, b_np = logprob_pairs(T, seed=1003)
    a_g, b_g = torch.as_tensor(a_np).cuda(), torch.as_tensor(b_np).cuda()
    lr2, k3_2, w2 = tim.mismatch(a_g, b_g, 2.0)
    r_lr, r_k3, r_w = oracle.mismatch(a_np, b_np, 2.0)
    assert np.all(np.abs(lr2.double().cpu().numpy() - r_lr) <= 2.0 ** -24 * np.abs(r_lr) + 1e-45)
    # K3 to one fp32 rounding, beside the oracle's own fp64 rounding of expm1 (see test_gpu_mismatch)
    k3_tol = 2.0 ** -23 * r_k3 + 2.0 ** -52 * np.abs(np.expm1(r_lr)) + 2.0 ** -149
    assert np.all(np.abs(k3_2.double().cpu().numpy() - r_k3) <= k3_tol)
    assert np.all(np.abs(w2.double().cpu().numpy() - r_w) <= TOL_W_REL * r_w)
    # sequence level over the packed responses (Section 4.2): K1/K3 scores, the
    # rejection mask at tau_seq = 0.001 and the truncated-and-rejected weights
    lens = cfg.lengths()
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    for est, name in ((tim.Estimator.K1, "k1"), (tim.Estimator.K3, "k3")):
        sc, kp, wt = tim.mismatch_seq(a_g, b_g, torch.as_tensor(cu, device="cuda"), C=2.0, tau_seq=1e-3,
                                      estimator=est)
        r_sc, r_kp, r_wt = oracle.mismatch_seq(a_np, b_np, cu, name, 2.0, 1e-3)
        sc = sc.cpu().numpy()
        mag = np.abs(r_sc) + 1e-30
        # + the oracle's own fp64 rounding of expm1 in each K3 term (see test_gpu_seqstats)
        te = 2.0 ** -52 * np.abs(np.expm1(r_lr)) if name == "k3" else np.zeros(T)
        oerr = np.array([te[cu[j]:cu[j + 1]].sum() for j in range(len(cu) - 1)])
        assert np.all(np.abs(sc - r_sc) <= 1e-9 * np.maximum(mag, np.abs(sc)) + oerr + 1e-15), \
            np.max(np.abs(sc - r_sc))
        clear = np.abs(r_sc - 1e-3) > 1e-12
        assert (kp.cpu().numpy().astype(bool)[clear] == r_kp[clear]).all()
        assert np.all(np.abs(wt.double().cpu().numpy() - r_wt) <= TOL_W_REL * r_wt)
        print(f"[stress] sequence {name}: {len(lens)} responses, score min/median/max = {sc.min():.3e}/"
              f"{np.median(sc):.3e}/{sc.max():.3e}; rejected at tau_seq=1e-3: {int((~r_kp).sum())}")


def test_long_training_vs_decode_batches():
    cfg, h, W, tok = workload("long")
    T = h.shape[0]
    lp, H, lse = tim.logprobs(h, W, tok, cfg.temperature, mode=Mode.TRAINING, micro_batch=cfg.micro_batch,
                              lse=True)
    oracle_sample(cfg, h, W, tok, lp, H)
    # rollout pass: decode batches of 64 rows
    B = cfg.rollout_batch
    ws = torch.empty(tim.workspace_size(B, cfg.d, cfg.V, Mode.ROLLOUT), dtype=torch.uint8, device="cuda")
    got = [torch.empty_like(lp), torch.empty_like(H), torch.empty_like(lse)]
    for t0 in range(0, T, B):
        sl = slice(t0, min(T, t0 + B))
        tim.logprobs(h[sl], W, tok[sl], cfg.temperature, mode=Mode.ROLLOUT, lse=True, workspace=ws,
                     out=(got[0][sl], got[1][sl], got[2][sl]))
    assert bits_equal(got[0], lp) and bits_equal(got[1], H) and bits_equal(got[2], lse)
    print(f"[long] {T // B} decode batches of {B} rows bitwise equal to micro-batches of {cfg.micro_batch}")
