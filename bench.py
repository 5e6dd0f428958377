"""Benchmark of the fused LM-head token log-prob + entropy path on one MI355X.

Workload (synthetic, seeded): d = 4096, V = 151936, 64 packed responses with
lengths uniform in [512, 4096] (about 147k tokens), hidden states RMS-normalised
N(0, 1) in bf16, W ~ N(0, 0.02^2) in bf16, tokens drawn from the model's own
softmax at temperature 1. Training mode, micro-batches of 16384 rows.

One step = the whole path over the whole token stream, with every input
resident in HBM: per micro-batch the partials kernel (LM-head GEMM on MFMA +
temperature + per-tile softmax partials + token gather) and the merge kernel
(fixed-order tree -> logp, entropy), then the mismatch-statistics kernel over
the stream against a second engine's log-probs (computed once, untimed, by the
split-K4 reduction order).

Reported beside the step (not part of `value`): rollout decode batches of 1,
16, 64, 128, 192 and 256 rows (achieved GB/s against the 8 TB/s HBM peak), the
sequence-level statistics, the backward of the fused log-prob over the same
stream (logit gradients, grad_hidden, grad_w), and the small (d = 2048, one
packed call) and long (d = 5120, tau = 0.7, micro-batches of 32768, plus its
rollout pass in decode batches of 64, checked bit for bit against training)
workloads' own rates, and the vendor GEMM (hipBLASLt) alone on the shapes of
the head's three contractions as a practical ceiling measured in the same run.
The oracle's parity on its sample is asserted (1e-3).

Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--config mid]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (256 CUs x 2.4 GHz)


def launch_slices(T: int, mb: int, lr: int):
    """Row ranges of the training launches: micro-batches of mb rows, each in launches of at most lr rows (the
    library's planner, tim_logprobs_rows_per_launch), exactly as tim_logprobs runs them."""
    out = []
    for m0 in range(0, T, mb):
        m1 = min(T, m0 + mb)
        out += [(a, min(m1, a + lr)) for a in range(m0, m1, lr)]
    return out
PEAK_HBM_GBS = 8000.0
METRIC = "tokens/s fused LM-head logp+entropy (d=4096,V=151936); % bf16 MFMA peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the sources of the LM-head forward kernel (its tile pass and epilogue)."""
    h = hashlib.sha256()
    for f in ("tilepass.h", "lmhead.hip"):
        h.update(open(os.path.join(ROOT, "paper_2605_14220_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def load_traffic(name: str):
    """HBM bytes per launch of the partials kernel from the committed rocprofv3
    PMC summary, if it was taken on the current kernel source; else None."""
    p = os.path.join(ROOT, "profiles", f"traffic_{name}.txt")
    if not os.path.exists(p):
        return None
    kv = {}
    for line in open(p):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(h, W, tok, tau, rows: int, seed: int = 7, threads: int | None = None):
    """Time the fp64 oracle on a seeded sample of rows on the host cores (all
    of them, or `threads`)."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    import oracle
    from workload import bf16_bits

    T = h.shape[0]
    idx = np.sort(np.random.default_rng(seed).choice(T, size=rows, replace=False))
    it = torch.as_tensor(idx, device=h.device)
    hb = bf16_bits(h.index_select(0, it))
    tb = tok.index_select(0, it).cpu().numpy()
    wb = bf16_bits(W)
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=threads):
        t0 = time.perf_counter()
        lp, ent = oracle.logprobs(hb, wb, tb, tau)
        dt = time.perf_counter() - t0
        used = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return idx, lp, ent, dt, used


def host_info():
    """The host the oracle baseline runs on: logical CPUs and CPU model."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"host_cpus": os.cpu_count(), "cpu_model": model}


def _threads():
    from threadpoolctl import threadpool_info
    return int(max([p.get("num_threads", 1) for p in threadpool_info()] or [1]))


def oracle_beside(dev, T, tau, cu, adv, norm_sample, bwd_sample, W):
    """The oracle timed beside the other rows of the path, each on inputs that
    are seeded and synthetic (never the path's outputs), with the largest
    GPU - oracle difference on the same inputs:
    * mismatch, sequence statistics and PPO loss over the whole packed stream
      of seeded log-prob pairs (trainer / rollout) of the workload's shape;
    * the final RMS norm and its gradients on sampled rows of the hidden states;
    * grad_hidden of the backward on sampled rows (each depends on its row only)."""
    import numpy as np
    import torch

    import oracle
    import paper_2605_14220_amd as tim
    from oracle.logprobs import bf16_to_f64
    from workload import bf16_bits, logprob_pairs

    thr = _threads()
    res = {}

    def timed(fn):
        t0 = time.perf_counter()
        r = fn()
        return r, time.perf_counter() - t0

    a_np, b_np = logprob_pairs(T, seed=71)
    a_t, b_t = torch.from_numpy(a_np).to(dev), torch.from_numpy(b_np).to(dev)
    cu_np = cu.cpu().numpy()
    sample = f"the whole {T}-token packed stream of seeded log-prob pairs (workload.logprob_pairs, seed 71)"

    (lr_r, k3_r, w_r), dt = timed(lambda: oracle.mismatch(a_np, b_np, 2.0))
    lr_g, k3_g, w_g = (x.double().cpu().numpy() for x in tim.mismatch(a_t, b_t, 2.0))
    res["mismatch"] = {
        "cpu_oracle": {"value": T / dt, "unit": "tokens/s", "cores": thr, "kind": "oracle", "sample": sample},
        "oracle_parity": {"max_abs_dlog_ratio": float(np.abs(lr_g - lr_r).max()),
                          "max_abs_dk3": float(np.abs(k3_g - k3_r).max()),
                          "max_rel_dis_weight": float((np.abs(w_g - w_r) / w_r).max())}}

    (sc_r, keep_r, ws_r), dt = timed(lambda: oracle.mismatch_seq(a_np, b_np, cu_np, "k3", 2.0, 1e-3))
    sc_g, keep_g, ws_g = tim.mismatch_seq(a_t, b_t, cu, C=2.0, tau_seq=1e-3)
    res["seq"] = {
        "cpu_oracle": {"value": T / dt, "unit": "tokens/s", "cores": thr, "kind": "oracle", "sample": sample},
        "oracle_parity": {"max_rel_dscore": float(np.abs(sc_g.cpu().numpy() - sc_r).max() / np.abs(sc_r).max()),
                          "keep_masks_equal": bool(np.array_equal(keep_g.cpu().numpy().astype(bool), keep_r)),
                          "max_abs_dweight": float(np.abs(ws_g.double().cpu().numpy() - ws_r).max())}}

    w32 = w_r.astype(np.float32)  # the oracle's own truncated token weights
    adv_np = adv.cpu().numpy()
    pr, dt = timed(lambda: oracle.ppo_loss(a_np, b_np, adv_np, cu_np, 0.2, 0.28, weight=w32))
    pg = tim.ppo_loss(a_t, b_t, adv, cu, 0.2, 0.28, torch.from_numpy(w32).to(dev))
    res["ppo"] = {
        "cpu_oracle": {"value": T / dt, "unit": "tokens/s", "cores": thr, "kind": "oracle",
                       "sample": sample + ", seeded advantages, the oracle's own truncated IS weights"},
        "oracle_parity": {"rel_dbatch_loss": float(abs(float(pg["batch_loss"].item()) - pr["batch_loss"])
                                                   / max(abs(pr["batch_loss"]), 1e-300)),
                          "max_abs_dgrad": float(np.abs(pg["grad"].double().cpu().numpy() - pr["grad"]).max()),
                          "clipped_equal": bool(np.array_equal(pg["clipped"].cpu().numpy().astype(bool),
                                                               pr["clipped"]))}}

    if norm_sample is not None:
        idx, x_bits, g_bits, G, h_gpu, gx_gpu = norm_sample
        (hb_r, _, _), dt_f = timed(lambda: oracle.rmsnorm(x_bits, g_bits, 1e-6))
        (dx_r, _), dt_b = timed(lambda: oracle.rmsnorm_grads(x_bits, g_bits, 1e-6, G))
        code_diff = np.abs(h_gpu.astype(np.int32) - hb_r.astype(np.int32))
        res["rmsnorm"] = {
            "cpu_oracle": {"value": len(idx) / (dt_f + dt_b), "unit": "rows/s (forward + backward)", "cores": thr,
                           "kind": "oracle", "sample": f"{len(idx)} seeded rows (seed 72) of the hidden states"},
            "oracle_parity": {"codes_equal_frac": float((code_diff == 0).mean()),
                              "max_code_diff": int(code_diff.max()),
                              "max_rel_dgrad_x": float(np.abs(gx_gpu - dx_r).max() / np.abs(dx_r).max())}}

    if bwd_sample is not None:
        idx, h_bits, tok_np, g_lp, g_h, gh_gpu = bwd_sample
        w_bits = bf16_bits(W)

        def grad_hidden():
            dacc = oracle.logit_grads(h_bits, w_bits, tok_np, tau, g_lp, g_h)
            dh = np.zeros((len(idx), w_bits.shape[1]))
            for v0 in range(0, w_bits.shape[0], 8192):  # dacc . W over vocabulary chunks (bounded memory)
                dh += dacc[:, v0:v0 + 8192] @ bf16_to_f64(w_bits[v0:v0 + 8192])
            return dh
        dh_r, dt = timed(grad_hidden)
        res["backward"] = {
            "cpu_oracle": {"value": len(idx) / dt, "unit": "tokens/s (grad_hidden rows)", "cores": thr,
                           "kind": "oracle", "sample": f"grad_hidden of {len(idx)} seeded rows (seed 73)"},
            "oracle_parity": {"max_rel_dgrad_hidden": float(np.abs(gh_gpu - dh_r).max() / np.abs(dh_r).max())}}
    return res


def decode_sweep(tim, h, W, tok, tau, sizes, n_calls=40):
    """Rollout-mode decode calls of B rows (one launch each): each call streams
    all of W once, so the algorithmic bytes are W + the rows' hidden states,
    tokens, partials (written and read) and outputs; HBM-bound."""
    import torch
    from paper_2605_14220_amd import Mode

    T, d = h.shape
    V = W.shape[0]
    dev = h.device
    stream = torch.cuda.current_stream(dev)
    res = []
    for B in sizes:
        rws = torch.empty(tim.workspace_size(B, d, V, Mode.ROLLOUT), dtype=torch.uint8, device=dev)
        r_out = tuple(torch.empty(B, dtype=torch.float32, device=dev) for _ in range(3))
        for i in range(3):
            tim.logprobs(h[i * B:(i + 1) * B], W, tok[i * B:(i + 1) * B], tau, mode=Mode.ROLLOUT, lse=True,
                         workspace=rws, out=r_out)
        r0 = torch.cuda.Event(enable_timing=True)
        r1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        r0.record(stream)
        for i in range(n_calls):
            a0 = (i * B) % (T - B)
            tim.logprobs(h[a0:a0 + B], W, tok[a0:a0 + B], tau, mode=Mode.ROLLOUT, lse=True, workspace=rws, out=r_out)
        r1.record(stream)
        torch.cuda.synchronize()
        r_ms = r0.elapsed_time(r1) / n_calls
        per_row = rws.numel() // (16 * B)  # partials per row of this call's shape
        r_bytes = 2.0 * V * d + 2.0 * B * d + 4 * B + 16.0 * B * per_row * 2 + 12 * B
        gbs = r_bytes / (r_ms / 1e3) / 1e9
        res.append({"rows_per_call": B, "ms_per_call": r_ms, "tokens_per_s": B / (r_ms / 1e3), "bound": "hbm",
                    "achieved_GBps": gbs, "peak_GBps": PEAK_HBM_GBS, "frac": gbs / PEAK_HBM_GBS,
                    "bytes_per_call": r_bytes})
        log(f"[bench] rollout decode batch of {B}: {r_ms:.3f} ms/call (partials + merge), {gbs:.0f} GB/s "
            f"algorithmic = {gbs / PEAK_HBM_GBS:.1%} of 8 TB/s")
        del rws
    return res


def other_workload(name, steps, decode_rows=0):
    """Timed rate of another configuration's packed stream in training
    mode (its micro-batches, partials + merge per micro-batch), with the
    partials kernel's own time per full launch, and for the long workload the
    rollout pass in decode batches of its rollout size over the whole stream."""
    import numpy as np
    import torch

    import paper_2605_14220_amd as tim
    from paper_2605_14220_amd import Mode
    from workload import CONFIGS, hidden_states, uniforms, vocab_weights
    from workload.gen import seeds
    from workload.sampler import sample_tokens

    cfg = CONFIGS[name]
    dev = torch.device("cuda:0")
    T, d, V, tau = cfg.tokens, cfg.d, cfg.V, cfg.temperature
    mb = cfg.micro_batch or T
    hs, ws, us = seeds(cfg)
    h = hidden_states(T, d, hs, device=dev)
    W = vocab_weights(V, d, cfg.w_std, ws, device=dev)
    tok = sample_tokens(h, W, tau, uniforms(T, us), dtype=torch.float32)
    ws_buf = torch.empty(tim.workspace_size(T, d, V, Mode.TRAINING, mb), dtype=torch.uint8, device=dev)
    out = tuple(torch.empty(T, dtype=torch.float32, device=dev) for _ in range(3))
    lr = tim.rows_per_launch(T, d, Mode.TRAINING, mb)
    slices = launch_slices(T, mb, lr)
    stream = torch.cuda.current_stream(dev)

    def step(evs):
        for i, (a, b) in enumerate(slices):
            if evs is not None:
                evs[i][0].record(stream)
            tim.logprobs_partials(h[a:b], W, tok[a:b], ws_buf, tau, mode=Mode.TRAINING)
            if evs is not None:
                evs[i][1].record(stream)
            tim.logprobs_merge(ws_buf, tok[a:b], V, out=(out[0][a:b], out[1][a:b], out[2][a:b]))

    step(None)
    torch.cuda.synchronize()
    allev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in slices]
             for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for k in range(steps):
        step(allev[k])
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    full = [e0.elapsed_time(e1) for evs in allev for (a, b), (e0, e1) in zip(slices, evs) if b - a == lr]
    k_ms = float(np.mean(full))
    k_frac = 2.0 * d * V * lr / (k_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS
    r = {"workload": f"{name}: d={d} V={V} {cfg.n_responses} responses U[{cfg.len_lo},{cfg.len_hi}] packed = {T} "
                     f"tokens, training mode, micro-batch {mb}, tau={tau}",
         "tokens": T, "steps": steps, "ms_per_step": ms, "tokens_per_s": T / (ms / 1e3),
         "mfma_peak_frac": 2.0 * d * V * T / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
         "partials_launch_ms": k_ms, "partials_rows_per_launch": lr, "partials_frac": k_frac}
    log(f"[bench] {name}: {ms:.3f} ms/step, {r['tokens_per_s']:,.0f} tokens/s = {r['mfma_peak_frac']:.1%} of bf16 "
        f"peak; partials kernel {k_ms:.3f} ms per {lr}-row launch = {k_frac:.1%}")
    if decode_rows:
        B = decode_rows
        rws = torch.empty(tim.workspace_size(B, d, V, Mode.ROLLOUT), dtype=torch.uint8, device=dev)
        dec = tuple(torch.empty(T, dtype=torch.float32, device=dev) for _ in range(3))
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for a in range(0, T, B):
            b = min(T, a + B)
            tim.logprobs(h[a:b], W, tok[a:b], tau, mode=Mode.ROLLOUT, lse=True, workspace=rws,
                         out=(dec[0][a:b], dec[1][a:b], dec[2][a:b]))
        e1.record(stream)
        torch.cuda.synchronize()
        d_ms = e0.elapsed_time(e1)
        calls = (T + B - 1) // B
        same = all(torch.equal(x.view(torch.int32), y.view(torch.int32)) for x, y in zip(dec, out))
        r["rollout_pass"] = {"rows_per_call": B, "calls": calls, "ms": d_ms, "ms_per_call": d_ms / calls,
                             "achieved_GBps": 2.0 * V * d / (d_ms / calls / 1e3) / 1e9,
                             "bitwise_equal_to_training": same}
        log(f"[bench] {name}: rollout pass in {calls} decode batches of {B}: {d_ms:.1f} ms "
            f"({d_ms / calls:.3f} ms/call), bitwise equal to training: {same}")
        if not same:
            raise SystemExit(f"bench: {name} rollout pass differs from training mode")
    del h, W, tok, ws_buf
    torch.cuda.empty_cache()
    return r


def vendor_gemm_reference(dev, d, V, rows, reps=5):
    """The vendor GEMM (hipBLASLt through torch.mm, bf16 in, bf16 out) alone on the shapes of the head's
    contractions at one micro-batch: the forward's logits h @ W^T (K = d; the fused kernel does the softmax on
    top), and the backward's grad_hidden = dlogits @ W (K = V padded to 256) and grad_w = dlogits^T @ h (K =
    rows, dlogits^T contiguous, as the backward stages it). A practical ceiling measured on the same box in the
    same run, not part of the path; median of `reps` timed calls after one untimed."""
    import torch
    import numpy as np
    vp = -(-V // 256) * 256
    g = torch.Generator(device=dev).manual_seed(5)
    h = torch.empty(rows, d, device=dev, dtype=torch.bfloat16).normal_(generator=g)
    W = torch.empty(vp, d, device=dev, dtype=torch.bfloat16).normal_(0.0, 0.02, generator=g)
    out = {}

    def timed(name, fn, flop):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        tf = flop / (ms / 1e3) / 1e12
        out[name] = {"ms": ms, "achieved": tf, "frac": tf / PEAK_BF16_TFLOPS}
        log(f"[bench] vendor GEMM {name}: {ms:.3f} ms, {tf:.1f} TFLOP/s = {tf / PEAK_BF16_TFLOPS:.1%} of bf16 peak")

    logits = torch.empty(rows, V, device=dev, dtype=torch.bfloat16)
    timed("forward_logits", lambda: torch.mm(h, W[:V].t(), out=logits), 2.0 * rows * V * d)
    del logits
    dl = torch.empty(rows, vp, device=dev, dtype=torch.bfloat16).normal_(0.0, 0.01, generator=g)
    gh = torch.empty(rows, d, device=dev, dtype=torch.bfloat16)
    timed("grad_hidden", lambda: torch.mm(dl, W, out=gh), 2.0 * rows * vp * d)
    dlt = dl.t().contiguous()
    del dl, gh
    gw = torch.empty(vp, d, device=dev, dtype=torch.bfloat16)
    timed("grad_w", lambda: torch.mm(dlt, h, out=gw), 2.0 * rows * vp * d)
    del dlt, gw, h, W
    torch.cuda.empty_cache()
    out["note"] = ("hipBLASLt via torch.mm on the same shapes (micro-batch rows), plain GEMM without the fused "
                   "softmax / gradient epilogues: the practical MFMA ceiling of these contractions on this box")
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="mid")
    ap.add_argument("--cpu-rows", type=int, default=4096, help="rows of the oracle CPU baseline (0 = skip)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after timing, run a plain copy kernel of known size (torch.neg over 2^28 fp32: "
                         "1 GiB read + 1 GiB written) so a counter profile can scale HBM byte counters")
    ap.add_argument("--no-backward", dest="backward", action="store_false",
                    help="skip the backward measurement")
    ap.add_argument("--no-others", dest="others", action="store_false",
                    help="skip the small and long workloads")
    ap.add_argument("--no-vendor", dest="vendor", action="store_false",
                    help="skip the vendor GEMM reference on the same shapes")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: this path runs on a single GPU "
              f"(token- or vocabulary-parallel sharding is a design note only, not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2605_14220_amd as tim
    from paper_2605_14220_amd import Mode, Order
    from workload import CONFIGS, hidden_states, uniforms, vocab_weights
    from workload.gen import seeds
    from workload.sampler import sample_tokens

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    tim.load_library()
    dev = torch.device("cuda:0")
    cfg = CONFIGS[args.config]
    T = cfg.tokens
    d, V, tau = cfg.d, cfg.V, cfg.temperature
    mb = cfg.micro_batch or T
    hs, ws, us = seeds(cfg)

    t_gen = time.perf_counter()
    h = hidden_states(T, d, hs, device=dev)
    W = vocab_weights(V, d, cfg.w_std, ws, device=dev)
    tok = sample_tokens(h, W, tau, uniforms(T, us), dtype=torch.float32)
    torch.cuda.synchronize()
    log(f"[bench] {cfg.name}: T={T} d={d} V={V} tau={tau} micro_batch={mb}; inputs ready in "
        f"{time.perf_counter() - t_gen:.1f}s")

    ws_buf = torch.empty(tim.workspace_size(T, d, V, Mode.TRAINING, mb), dtype=torch.uint8, device=dev)
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    ent = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    stats = tuple(torch.empty(T, dtype=torch.float32, device=dev) for _ in range(3))
    # the second engine's log-probs (split-K4 reduction order), untimed
    logp_b, _, _ = tim.logprobs(h, W, tok, tau, mode=Mode.TRAINING, micro_batch=mb, order=Order.SPLITK4,
                                workspace=ws_buf)
    lr = tim.rows_per_launch(T, d, Mode.TRAINING, mb)  # the planner's launches within each micro-batch
    slices = launch_slices(T, mb, lr)
    stream = torch.cuda.current_stream(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in slices]

    def step(record: bool):
        for i, (a, b) in enumerate(slices):
            if record:
                ev[i][0].record(stream)
            tim.logprobs_partials(h[a:b], W, tok[a:b], ws_buf, tau, mode=Mode.TRAINING)
            if record:
                ev[i][1].record(stream)
            tim.logprobs_merge(ws_buf, tok[a:b], V, out=(logp[a:b], ent[a:b], lse[a:b]))
        tim.mismatch(logp, logp_b, 2.0, out=stats)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    # the composed step is exactly tim_logprobs: check it bit for bit once
    ref = tim.logprobs(h, W, tok, tau, mode=Mode.TRAINING, micro_batch=mb, lse=True, workspace=ws_buf)
    step(False)
    torch.cuda.synchronize()
    assert torch.equal(ref[0], logp) and torch.equal(ref[1], ent) and torch.equal(ref[2], lse)

    kern_ms = []
    step_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for k in range(args.steps):
        step_ev[k][0].record(stream)
        step(True)
        step_ev[k][1].record(stream)
        # the events of this step are read after the timed region; keep them per step
        kern_ms.append([(e0, e1) for e0, e1 in ev])
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in slices]
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps
    tok_per_s = T / (ms_per_step / 1e3)
    ms_median = float(np.median([e0.elapsed_time(e1) for e0, e1 in step_ev]))

    # dominant kernel: lmhead_partials over full micro-batches
    durs = []
    for stepev in kern_ms:
        for (a, b), (e0, e1) in zip(slices, stepev):
            if b - a == lr:
                durs.append(e0.elapsed_time(e1))
    avg_ms = float(np.mean(durs))
    flop_per_launch = 2.0 * d * V * lr
    achieved_tflops = flop_per_launch / (avg_ms / 1e3) / 1e12
    path_tflops = 2.0 * d * V * tok_per_s / 1e12
    traffic = load_traffic(f"lmhead_partials_{cfg.name}")
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step ({wall / args.steps * 1e3:.3f} wall), "
        f"{tok_per_s:,.0f} tokens/s, path {path_tflops:.1f} TFLOP/s = {path_tflops / PEAK_BF16_TFLOPS:.1%} of "
        f"bf16 peak; partials kernel {avg_ms:.3f} ms/launch = {achieved_tflops:.1f} TFLOP/s")

    # rollout mode (decode steps): each call streams all of W once; HBM-bound
    sweep = decode_sweep(tim, h, W, tok, tau, (1, 16, 64, 128, 192, 256))
    rollout = next(r for r in sweep if r["rows_per_call"] == 64)

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("[bench] calibration copy: 3 x torch.neg over 2^28 fp32 (1 GiB in, 1 GiB out)")

    # sequence level (Section 4.2): K3 scores of the packed responses, the
    # rejection mask at tau_seq = 0.001 and the truncated-and-rejected weights
    lens = cfg.lengths()
    cu = torch.as_tensor(np.concatenate([[0], np.cumsum(lens)]).astype(np.int64), device=dev)
    seq_out = (torch.empty(len(lens), dtype=torch.float64, device=dev),
               torch.empty(len(lens), dtype=torch.uint8, device=dev), torch.empty(T, dtype=torch.float32, device=dev))
    for _ in range(3):
        tim.mismatch_seq(logp, logp_b, cu, C=2.0, tau_seq=1e-3, out=seq_out)
    q0 = torch.cuda.Event(enable_timing=True)
    q1 = torch.cuda.Event(enable_timing=True)
    n_seq_calls = 50
    torch.cuda.synchronize()
    q0.record(stream)
    for _ in range(n_seq_calls):
        tim.mismatch_seq(logp, logp_b, cu, C=2.0, tau_seq=1e-3, out=seq_out)
    q1.record(stream)
    torch.cuda.synchronize()
    seq_ms = q0.elapsed_time(q1) / n_seq_calls
    seq_bytes = 12.0 * T + 9.0 * len(lens)
    seq = {"responses": len(lens), "tokens": T, "ms_per_call": seq_ms, "tokens_per_s": T / (seq_ms / 1e3),
           "achieved_GBps": seq_bytes / (seq_ms / 1e3) / 1e9, "bytes_per_call": seq_bytes,
           "rejected_at_tau_1e-3": int((seq_out[1] == 0).sum().item()),
           "max_k3_score": float(seq_out[0].max().item())}
    log(f"[bench] sequence-level K3 scores / mask / weights over {len(lens)} responses: {seq_ms * 1e3:.1f} us/call")

    # clipped PPO/GRPO loss over the stream (logp_b stands in for the old log-probs), weighted by the
    # sequence-level TIS + RS weights, with its gradient
    adv = torch.repeat_interleave(torch.randn(len(lens), generator=torch.Generator(device="cpu").manual_seed(96)),
                                  torch.as_tensor(lens)).float().to(dev)
    pl = tim.ppo_loss(logp, logp_b, adv, cu, 0.2, 0.28, seq_out[2])
    for _ in range(3):
        tim.ppo_loss(logp, logp_b, adv, cu, 0.2, 0.28, seq_out[2], out=pl)
    q0.record(stream)
    for _ in range(n_seq_calls):
        tim.ppo_loss(logp, logp_b, adv, cu, 0.2, 0.28, seq_out[2], out=pl)
    q1.record(stream)
    torch.cuda.synchronize()
    ppo_ms = q0.elapsed_time(q1) / n_seq_calls
    ppo = {"responses": len(lens), "tokens": T, "ms_per_call": ppo_ms, "tokens_per_s": T / (ppo_ms / 1e3),
           "bytes_per_call": 16.0 * T + 13.0 * T + 24.0 * len(lens),
           "batch_loss": float(pl["batch_loss"].item()), "clipped_tokens": int(pl["clipped"].sum().item())}
    log(f"[bench] PPO/GRPO loss + gradient over {len(lens)} responses: {ppo_ms * 1e3:.1f} us/call")

    # the final RMS norm in front of the head over the whole stream (HBM-bound), and its backward
    gam = (1.0 + 0.1 * torch.randn(d, generator=torch.Generator(device="cpu").manual_seed(98))).to(torch.bfloat16).to(dev)
    h_n = torch.empty_like(h)
    for _ in range(2):
        tim.rmsnorm(h, gam, 1e-6, out=h_n)
    n0 = torch.cuda.Event(enable_timing=True)
    n1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    n0.record(stream)
    for _ in range(10):
        _, rstd_n = tim.rmsnorm(h, gam, 1e-6, out=h_n)
    n1.record(stream)
    torch.cuda.synchronize()
    nf_ms = n0.elapsed_time(n1) / 10
    G_n = torch.randn(T, d, generator=torch.Generator(device=dev).manual_seed(97), device=dev)
    gg_n = torch.empty(d, dtype=torch.float32, device=dev)
    gx_n, _ = tim.rmsnorm_backward(h, gam, rstd_n, G_n, grad_gamma=gg_n)
    torch.cuda.synchronize()
    n0.record(stream)
    for _ in range(5):
        tim.rmsnorm_backward(h, gam, rstd_n, G_n, grad_gamma=gg_n)
    n1.record(stream)
    torch.cuda.synchronize()
    nb_ms = n0.elapsed_time(n1) / 5
    norm_sample = None
    if args.cpu_rows > 0:
        from workload import bf16_bits
        idx_n = np.sort(np.random.default_rng(72).choice(T, size=min(2048, T), replace=False))
        it_n = torch.as_tensor(idx_n, device=dev)
        norm_sample = (idx_n, bf16_bits(h.index_select(0, it_n)), bf16_bits(gam), G_n.index_select(0, it_n).double().cpu().numpy(),
                       bf16_bits(h_n.index_select(0, it_n)), gx_n.index_select(0, it_n).double().cpu().numpy())
    nf_bytes = 4.0 * T * d + 4.0 * T
    nb_bytes = 10.0 * T * d + 4.0 * T  # x (2 B) and G (4 B) read, grad_x (4 B) written per element; rstd
    norm = {"forward_ms": nf_ms, "forward_GBps": nf_bytes / (nf_ms / 1e3) / 1e9,
            "forward_frac": nf_bytes / (nf_ms / 1e3) / 1e9 / PEAK_HBM_GBS, "forward_bytes": nf_bytes,
            "backward_ms": nb_ms, "backward_GBps": nb_bytes / (nb_ms / 1e3) / 1e9,
            "backward_frac": nb_bytes / (nb_ms / 1e3) / 1e9 / PEAK_HBM_GBS, "backward_bytes": nb_bytes,
            "bound": "hbm", "peak_GBps": PEAK_HBM_GBS}
    log(f"[bench] final RMS norm over {T} rows: forward {nf_ms:.3f} ms ({norm['forward_GBps']:.0f} GB/s = "
        f"{norm['forward_frac']:.1%} of 8 TB/s), backward {nb_ms:.3f} ms ({norm['backward_GBps']:.0f} GB/s algorithmic)")
    del G_n, gx_n, h_n
    torch.cuda.empty_cache()

    # backward of the fused log-prob over the whole stream (the trainer's gradients)
    bwd = None
    bwd_sample = None
    if args.backward:
        g = torch.Generator(device="cpu").manual_seed(99)
        g_lp = torch.randn(T, generator=g).to(dev)
        g_h = (0.1 * torch.randn(T, generator=g)).to(dev)
        bws = torch.empty(tim.backward_workspace_size(T, d, V, mb), dtype=torch.uint8, device=dev)
        gw = torch.empty((V, d), dtype=torch.float32, device=dev)

        def bstep():
            return tim.logprobs_backward(h, W, tok, lse, g_lp, tau, entropy=ent, grad_entropy=g_h, micro_batch=mb,
                                         grad_w=gw, workspace=bws)
        gh, _ = bstep()
        torch.cuda.synchronize()
        b0 = torch.cuda.Event(enable_timing=True)
        b1 = torch.cuda.Event(enable_timing=True)
        n_b = 2
        b0.record(stream)
        for _ in range(n_b):
            gh, _ = bstep()
        b1.record(stream)
        torch.cuda.synchronize()
        b_ms = b0.elapsed_time(b1) / n_b
        b_flop = 3 * 2.0 * d * V * T
        bwd = {"ms_per_call": b_ms, "tokens_per_s": T / (b_ms / 1e3), "bound": "mfma",
               "achieved": b_flop / (b_ms / 1e3) / 1e12, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
               "frac": b_flop / (b_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, "flop_per_call": b_flop,
               "micro_batch": mb, "workspace_GB": bws.numel() / 1e9,
               "finite": bool(torch.isfinite(gh).all().item() and torch.isfinite(gw).all().item())}
        log(f"[bench] backward over {T} tokens (micro-batch {mb}): {b_ms:.1f} ms/call, {bwd['tokens_per_s']:,.0f} "
            f"tokens/s, {bwd['achieved']:.1f} TFLOP/s = {bwd['frac']:.1%} of bf16 peak (3 contractions)")
        if args.cpu_rows > 0:
            from workload import bf16_bits
            idx_b = np.sort(np.random.default_rng(73).choice(T, size=4, replace=False))
            it_b = torch.as_tensor(idx_b, device=dev)
            bwd_sample = (idx_b, bf16_bits(h.index_select(0, it_b)), tok.index_select(0, it_b).cpu().numpy(),
                          g_lp.index_select(0, it_b).double().cpu().numpy(),
                          g_h.index_select(0, it_b).double().cpu().numpy(),
                          gh.index_select(0, it_b).double().cpu().numpy())
        del bws, gw, gh
        torch.cuda.empty_cache()

    # mismatch report between the two engines (context)
    dl = stats[0].abs()
    q = torch.quantile(dl.float(), torch.tensor([0.5, 0.99], device=dev)).tolist()
    # mean K3 also from the fp64 sequence score of the whole stream as one response (the token values are
    # those terms rounded once to fp32, so the two agree to ~2^-24)
    whole = torch.tensor([0, T], dtype=torch.int64, device=dev)
    sc_all, _, _ = tim.mismatch_seq(logp, logp_b, whole, C=2.0, tau_seq=1e30)
    mis = {"abs_dlogp_p50": q[0], "abs_dlogp_p99": q[1], "abs_dlogp_max": float(dl.max()),
           "mean_k3": float(stats[1].double().mean()), "mean_k3_fp64_sequence_sum": float(sc_all.item()) / T,
           "mean_is_weight": float(stats[2].double().mean()), "C": 2.0}

    cpu = None
    cpu_single = None
    parity = None
    mstats = None
    if args.cpu_rows > 0:
        log(f"[bench] oracle CPU baseline on {args.cpu_rows} sampled rows ...")
        idx, lp_ref, ent_ref, dt, threads = cpu_baseline(h, W, tok, tau, args.cpu_rows)
        cpu = {"value": args.cpu_rows / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
               "sample": f"{args.cpu_rows} seeded rows (seed 7) of the {T}-token stream, fp64 numpy oracle, "
                         f"{dt:.1f} s", **host_info()}
        it = torch.as_tensor(idx, device=dev)
        e_lp = float(np.max(np.abs(logp.index_select(0, it).double().cpu().numpy() - lp_ref)))
        e_h = float(np.max(np.abs(ent.index_select(0, it).double().cpu().numpy() - ent_ref)))
        parity = {"rows": int(args.cpu_rows), "max_abs_dlogp": e_lp, "max_abs_dentropy": e_h, "tol": 1e-3}
        if not (e_lp <= 1e-3 and e_h <= 1e-3):
            raise SystemExit(f"bench: oracle parity failed on the sample: max|dlogp|={e_lp} max|dH|={e_h} > 1e-3")
        log(f"[bench] oracle: {cpu['value']:.1f} tokens/s on {threads} threads; parity on sample: "
            f"max|dlogp|={e_lp:.2e} max|dH|={e_h:.2e}")
        n1 = max(1, args.cpu_rows // 16)
        _, _, _, dt1, thr1 = cpu_baseline(h, W, tok, tau, n1, seed=8, threads=1)
        cpu_single = {"value": n1 / dt1, "unit": "tokens/s", "cores": int(thr1), "kind": "oracle",
                      "sample": f"{n1} seeded rows (seed 8) of the {T}-token stream, one thread, {dt1:.1f} s",
                      **host_info()}
        log(f"[bench] oracle on one thread: {cpu_single['value']:.1f} tokens/s ({n1} rows)")
        log("[bench] oracle beside the other rows ...")
        beside = oracle_beside(dev, T, tau, cu, adv, norm_sample, bwd_sample, W)
        for key, obj in (("mismatch", None), ("seq", seq), ("ppo", ppo), ("rmsnorm", norm), ("backward", bwd)):
            if key in beside and obj is not None:
                obj.update(beside[key])
        mstats = beside.get("mismatch")
        log("[bench] oracle beside: " + "; ".join(
            f"{k} {v['cpu_oracle']['value']:.3g} {v['cpu_oracle']['unit']} parity {v['oracle_parity']}"
            for k, v in beside.items()))

    others = None
    if args.others and args.config == "mid":
        del ws_buf
        torch.cuda.empty_cache()
        others = {"small": other_workload("small", steps=5),
                  "long": other_workload("long", steps=3, decode_rows=CONFIGS["long"].rollout_batch)}

    vendor = None
    if args.vendor:
        torch.cuda.empty_cache()
        vendor = vendor_gemm_reference(dev, d, V, mb)

    out = {
        "metric": METRIC,
        "value": tok_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_median": ms_median,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: d={d} V={V} {cfg.n_responses} responses U[{cfg.len_lo},{cfg.len_hi}] "
                               f"packed = {T} tokens, training mode, micro-batch {mb}, tau={tau}",
                   "tokens": T, "d": d, "V": V, "micro_batch": mb, "temperature": tau},
        "mfma_peak_frac": path_tflops / PEAK_BF16_TFLOPS,
        "roofline": {"bound": "mfma", "achieved": achieved_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved_tflops / PEAK_BF16_TFLOPS,
                     "traffic": traffic,
                     "kernel": "lmhead_partials", "launch_ms": avg_ms, "flop_per_launch": flop_per_launch,
                     "rows_per_launch": lr},
        "cpu_baseline": cpu,
        "cpu_baseline_single_thread": cpu_single,
        "parity_sample": parity,
        "mismatch_vs_splitk4": mis,
        "mismatch_stats": mstats,
        "rollout_decode": rollout,
        "rollout_decode_sweep": sweep,
        "other_workloads": others,
        "sequence_mismatch": seq,
        "backward": bwd,
        "rmsnorm": norm,
        "ppo_loss": ppo,
        "vendor_gemm_reference": vendor,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
