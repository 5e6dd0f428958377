"""The C-ABI library on the host: it loads, exports every entry point that
include/tim.h declares, sizes workspaces by the documented formula and rejects
every bad argument with the documented status before touching the GPU.

No call here reaches a kernel launch: each passes an argument that the host
checks reject (or T == 0), so these tests run without a GPU.
"""

import ctypes
import math
import os
import re
import subprocess

import pytest

import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode, Order, Status

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tim.h")

FAKE = 0x10000        # 16-byte aligned, never dereferenced (rejected before any launch)
FAKE_MIS = 0x10008    # misaligned


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(tim_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return tim.load_library()


def test_header_declares_the_boundary():
    names = declared_functions()
    assert names == ["tim_logit_grads", "tim_logits", "tim_logprobs", "tim_logprobs_backward",
                     "tim_logprobs_backward_workspace_size", "tim_logprobs_merge", "tim_logprobs_noalloc",
                     "tim_logprobs_partials", "tim_logprobs_rows_per_launch",
                     "tim_logprobs_workspace_size", "tim_mismatch", "tim_mismatch_seq", "tim_ppo_loss", "tim_rmsnorm",
                     "tim_rmsnorm_backward", "tim_rmsnorm_backward_workspace_size", "tim_status_string"]


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", tim.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT\s+(\w+)$", out, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for s in Status:
        text = lib.tim_status_string(int(s)).decode()
        assert text.startswith("TIM_OK" if s == 0 else "TIM_ERR_")
    assert lib.tim_status_string(99).decode() == "unknown tim_status"


def _launch_cap(d):
    # the largest multiple of 8192 rows whose bf16 hidden block plus 16384 d bytes of weight tiles fits 224 MiB
    return max(8192, (224 * 2 ** 20 // (2 * d) - 8192) // 8192 * 8192)


@pytest.mark.parametrize("d,cap", [(4096, 16384), (5120, 8192), (2048, 49152), (8192, 8192), (128, 909312)])
def test_training_launch_cap(lib, d, cap):
    assert _launch_cap(d) == cap
    assert tim.rows_per_launch(10 ** 6, d, Mode.TRAINING, 0) == cap
    assert tim.rows_per_launch(10 ** 6, d, Mode.TRAINING, 4 * cap) == cap
    assert tim.rows_per_launch(10 ** 6, d, Mode.TRAINING, cap - 128) == cap - 128
    assert tim.rows_per_launch(cap - 1, d, Mode.TRAINING, 0) == cap - 1
    assert tim.rows_per_launch(10 ** 6, d, Mode.ROLLOUT, 4096) == 10 ** 6  # rollout: one launch over all T rows


@pytest.mark.parametrize("args", [(0, 4096, 1, 0), (-5, 4096, 1, 0), (10, 100, 1, 0), (10, 0, 1, 0), (10, 4096, 7, 0),
                                  (10, 4096, 1, -1)])
def test_rows_per_launch_zero_when_invalid(lib, args):
    assert lib.tim_logprobs_rows_per_launch(*args) == 0


@pytest.mark.parametrize("T,d,V,mode,mb", [
    (64, 256, 4096, Mode.TRAINING, 0),
    (147000, 4096, 151936, Mode.TRAINING, 16384),
    (147000, 4096, 151936, Mode.TRAINING, 200000),
    (200, 4096, 151936, Mode.ROLLOUT, 16384),
    (129, 4096, 151936, Mode.ROLLOUT, 0),
    (128, 4096, 151936, Mode.ROLLOUT, 0),
    (64, 4096, 151936, Mode.ROLLOUT, 0),
    (5, 128, 1, Mode.ROLLOUT, 0),
    (7, 128, 4096 + 129, Mode.ROLLOUT, 0),
    (131072, 5120, 152064, Mode.TRAINING, 32768),
    (131072, 5120, 152064, Mode.TRAINING, 0),
    (138564, 4096, 151936, Mode.TRAINING, 65536),
])
def test_workspace_size_formula(lib, T, d, V, mode, mb):
    rows = T if (mode == Mode.ROLLOUT or mb == 0 or mb >= T) else mb
    if mode == Mode.TRAINING:  # training launches of at most the cache-fitting row count
        rows = min(rows, _launch_cap(d))
    # decode batches (rollout, at most 128 rows) keep one partial per half tile
    width = 128 if (mode == Mode.ROLLOUT and rows <= 128) else 256
    assert tim.workspace_size(T, d, V, mode, mb) == rows * math.ceil(V / width) * 16


@pytest.mark.parametrize("args", [(0, 256, 4096, 1, 0), (-1, 256, 4096, 1, 0), (10, 100, 4096, 1, 0),
                                  (10, 256, 0, 1, 0), (10, 256, 4096, 7, 0), (10, 256, 4096, 1, -1),
                                  (10, 256, 2048 * 256 + 1, 1, 0)])
def test_workspace_size_zero_when_invalid(lib, args):
    assert lib.tim_logprobs_workspace_size(*args) == 0


def _lp(lib, hidden=FAKE, w=FAKE, tokens=FAKE, T=8, d=256, V=4096, tau=1.0, mode=1, mb=0, order=0,
        logp=FAKE, ent=None, lse=None, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = 1 << 40
    return lib.tim_logprobs(hidden, w, tokens, T, d, V, tau, mode, mb, order, logp, ent, lse, ws, ws_bytes, None)


def test_logprobs_T_zero_is_noop_even_with_null_pointers(lib):
    assert _lp(lib, hidden=None, w=None, tokens=None, logp=None, ws=None, T=0) == Status.OK


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(hidden=None), Status.ERR_NULL),
    (dict(w=None), Status.ERR_NULL),
    (dict(tokens=None), Status.ERR_NULL),
    (dict(logp=None), Status.ERR_NULL),
    (dict(d=0), Status.ERR_SHAPE),
    (dict(d=-128), Status.ERR_SHAPE),
    (dict(d=64), Status.ERR_SHAPE),
    (dict(d=200), Status.ERR_SHAPE),
    (dict(d=384, order=1), Status.ERR_SHAPE),
    (dict(V=0), Status.ERR_SHAPE),
    (dict(V=-5), Status.ERR_SHAPE),
    (dict(V=2048 * 256 + 1), Status.ERR_SHAPE),
    (dict(tau=0.0), Status.ERR_VALUE),
    (dict(tau=-1.0), Status.ERR_VALUE),
    (dict(tau=float("nan")), Status.ERR_VALUE),
    (dict(tau=float("inf")), Status.ERR_VALUE),
    (dict(mode=2), Status.ERR_VALUE),
    (dict(mode=-1), Status.ERR_VALUE),
    (dict(order=2), Status.ERR_VALUE),
    (dict(mb=-1), Status.ERR_VALUE),
    (dict(hidden=FAKE_MIS), Status.ERR_VALUE),
    (dict(w=FAKE_MIS), Status.ERR_VALUE),
    (dict(ws=None), Status.ERR_WORKSPACE),
    (dict(ws=FAKE_MIS), Status.ERR_WORKSPACE),
    (dict(ws_bytes=8 * 16 * 16 - 1), Status.ERR_WORKSPACE),
    (dict(ws_bytes=0), Status.ERR_WORKSPACE),
    (dict(T=100, mb=10, ws_bytes=10 * 16 * 16 - 16), Status.ERR_WORKSPACE),
    (dict(mode=0, ws_bytes=8 * 32 * 16 - 1), Status.ERR_WORKSPACE),
])
def test_logprobs_rejects(lib, kw, expect):
    assert _lp(lib, **kw) == expect


def _lp_noalloc(lib, hidden=FAKE, w=FAKE, tokens=FAKE, T=8, d=256, V=4096, tau=1.0, mode=1, mb=0, order=0,
                logp=FAKE):
    return lib.tim_logprobs_noalloc(hidden, w, tokens, T, d, V, tau, mode, mb, order, logp, None, None, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=0, hidden=None, w=None, tokens=None, logp=None), Status.OK),
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(hidden=None), Status.ERR_NULL),
    (dict(logp=None), Status.ERR_NULL),
    (dict(d=200), Status.ERR_SHAPE),
    (dict(tau=0.0), Status.ERR_VALUE),
    (dict(mode=3), Status.ERR_VALUE),
    (dict(w=FAKE_MIS), Status.ERR_VALUE),
    # partials beyond the 64 MiB device array: at V = 151936 (594 tiles of 16 B per row) 7061 rows fit, 7062 not
    (dict(T=7062, d=4096, V=151936, mode=0), Status.ERR_WORKSPACE),
    (dict(T=20000, d=4096, V=151936, mode=1, mb=7062), Status.ERR_WORKSPACE),
    (dict(T=20000, d=4096, V=151936, mode=1, mb=0), Status.ERR_WORKSPACE),
    (dict(T=1, d=128, V=2048 * 256, mode=1), Status.ERR_HIP),
])
def test_logprobs_noalloc_rejects_on_the_host(lib, kw, expect):
    """Every argument check of tim_logprobs_noalloc, including its scratch limit, runs on the host before any
    HIP call (the last case passes them and fails only at the device lookup, as there is no GPU here)."""
    if expect == Status.ERR_HIP and _has_gpu():
        pytest.skip("a GPU is present: the call would launch")
    assert _lp_noalloc(lib, **kw) == expect


def _has_gpu():
    import torch
    return torch.cuda.is_available()


def test_noalloc_scratch_limit_matches_the_header():
    text = open(HEADER).read()
    assert "#define TIM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)" in text
    assert tim.NOALLOC_SCRATCH_BYTES == 64 << 20
    # 7061 rows of partials at V = 151936 fit, the next row does not
    assert 7061 * 594 * 16 <= tim.NOALLOC_SCRATCH_BYTES < 7062 * 594 * 16


def test_logprobs_error_precedence(lib):
    # shape errors are reported before value errors, value before workspace
    assert _lp(lib, d=100, tau=-1.0, ws=None) == Status.ERR_SHAPE
    assert _lp(lib, tau=-1.0, ws=None) == Status.ERR_VALUE
    assert _lp(lib, hidden=None, d=100) == Status.ERR_NULL


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-3), Status.ERR_SHAPE),
    (dict(a=None), Status.ERR_NULL),
    (dict(b=None), Status.ERR_NULL),
    (dict(C=0.0), Status.ERR_VALUE),
    (dict(C=-2.0), Status.ERR_VALUE),
    (dict(C=float("nan")), Status.ERR_VALUE),
    (dict(C=float("inf")), Status.ERR_VALUE),
])
def test_mismatch_rejects(lib, kw, expect):
    a = kw.get("a", FAKE)
    b = kw.get("b", FAKE)
    assert lib.tim_mismatch(a, b, kw.get("T", 8), kw.get("C", 2.0), FAKE, FAKE, FAKE, None) == expect


def test_mismatch_noops(lib):
    assert lib.tim_mismatch(None, None, 0, 2.0, None, None, None, None) == Status.OK
    # every output NULL: nothing to compute, nothing launched
    assert lib.tim_mismatch(FAKE, FAKE, 8, 2.0, None, None, None, None) == Status.OK


def _seq(lib, **kw):
    a = kw.get("a", FAKE)
    b = kw.get("b", FAKE)
    return lib.tim_mismatch_seq(a, b, kw.get("T", 8), kw.get("cu", FAKE), kw.get("n", 2), kw.get("est", 3),
                                kw.get("C", 2.0), kw.get("tau", 1e-3), FAKE, FAKE, FAKE, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(n=-1), Status.ERR_SHAPE),
    (dict(n=2 ** 31), Status.ERR_SHAPE),
    (dict(cu=None), Status.ERR_NULL),
    (dict(a=None), Status.ERR_NULL),
    (dict(b=None), Status.ERR_NULL),
    (dict(est=2), Status.ERR_VALUE),
    (dict(est=0), Status.ERR_VALUE),
    (dict(C=0.0), Status.ERR_VALUE),
    (dict(C=-1.0), Status.ERR_VALUE),
    (dict(C=math.inf), Status.ERR_VALUE),
    (dict(C=math.nan), Status.ERR_VALUE),
    (dict(tau=math.nan), Status.ERR_VALUE),
])
def test_mismatch_seq_rejects(lib, kw, expect):
    assert _seq(lib, **kw) == expect


def test_mismatch_seq_noops(lib):
    # no responses: nothing is read, whatever the pointers
    assert lib.tim_mismatch_seq(None, None, 0, None, 0, 3, 2.0, 1e-3, None, None, None, None) == Status.OK
    assert lib.tim_mismatch_seq(None, None, 5, None, 0, 0, -1.0, math.nan, None, None, None, None) == Status.OK
    # all outputs NULL: validated, nothing enqueued
    assert lib.tim_mismatch_seq(FAKE, FAKE, 8, FAKE, 2, 1, 2.0, math.inf, None, None, None, None) == Status.OK
    # T == 0 with responses: logp arrays are never read, may be NULL (still rejected on other errors)
    assert lib.tim_mismatch_seq(None, None, 0, FAKE, 2, 4, 2.0, 1e-3, None, None, None, None) == Status.ERR_VALUE


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(out=None), Status.ERR_NULL),
    (dict(hidden=None), Status.ERR_NULL),
    (dict(d=96), Status.ERR_SHAPE),
    (dict(V=0), Status.ERR_SHAPE),
    (dict(tau=0.0), Status.ERR_VALUE),
    (dict(order=3), Status.ERR_VALUE),
    (dict(hidden=FAKE_MIS), Status.ERR_VALUE),
])
def test_logits_rejects(lib, kw, expect):
    args = dict(hidden=FAKE, w=FAKE, T=4, d=256, V=300, tau=1.0, order=0, out=FAKE)
    args.update(kw)
    assert lib.tim_logits(args["hidden"], args["w"], args["T"], args["d"], args["V"], args["tau"],
                          args["order"], args["out"], None) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(ws=None), Status.ERR_NULL),
    (dict(tokens=None), Status.ERR_NULL),
    (dict(logp=None), Status.ERR_NULL),
    (dict(V=0), Status.ERR_SHAPE),
    (dict(order=9), Status.ERR_VALUE),
])
def test_merge_rejects(lib, kw, expect):
    a = dict(ws=FAKE, tokens=FAKE, T=4, V=300, order=0, logp=FAKE)
    a.update(kw)
    assert lib.tim_logprobs_merge(a["ws"], a["tokens"], a["T"], a["V"], a["order"], a["logp"], None, None,
                                  None) == expect
    assert lib.tim_logprobs_merge(None, None, 0, 300, 0, None, None, None, None) == Status.OK


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(hidden=None), Status.ERR_NULL),
    (dict(ws=None), Status.ERR_NULL),
    (dict(d=100), Status.ERR_SHAPE),
    (dict(tau=0.0), Status.ERR_VALUE),
    (dict(mode=5), Status.ERR_VALUE),
    (dict(ws_bytes=4 * 2 * 16 - 1), Status.ERR_WORKSPACE),
])
def test_partials_rejects(lib, kw, expect):
    a = dict(hidden=FAKE, w=FAKE, tokens=FAKE, T=4, d=256, V=300, tau=1.0, mode=1, order=0, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    assert lib.tim_logprobs_partials(a["hidden"], a["w"], a["tokens"], a["T"], a["d"], a["V"], a["tau"],
                                     a["mode"], a["order"], a["ws"], a["ws_bytes"], None) == expect


def test_python_binding_rejects_cpu_tensors():
    import torch
    h = torch.zeros(4, 256, dtype=torch.bfloat16)
    w = torch.zeros(300, 256, dtype=torch.bfloat16)
    tok = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU"):
        tim.logprobs(h, w, tok)
    with pytest.raises(TypeError):
        tim.logprobs(h.float(), w, tok)
    with pytest.raises(TypeError):
        tim.logprobs(h, w, tok.long())
    with pytest.raises(ValueError, match="GPU"):
        tim.mismatch(torch.zeros(3), torch.zeros(3))


# ---------------------------------------------------------------- backward

def _bwd_size(T, d, V, mb):
    """Row words, then W^T, dlogits, dlogits^T and h^T in whole 256-row tiles."""
    step = mb if 0 < mb < T else T
    t_pad = -(-step // 128) * 128
    v_pad = -(-V // 256) * 256
    a = lambda x: -(-x // 256) * 256
    d_pad, step_pad = a(d), a(step)
    return a(step * 16) + a(2 * d_pad * v_pad) + a(2 * step_pad * v_pad) + a(2 * v_pad * t_pad) + a(2 * d_pad * t_pad)


@pytest.mark.parametrize("T,d,V,mb", [(700, 256, 4173, 128), (138564, 4096, 151936, 16384), (1, 128, 1, 0),
                                      (300, 640, 5000, 0), (300, 640, 5000, 1024)])
def test_backward_workspace_size_formula(lib, T, d, V, mb):
    assert tim.backward_workspace_size(T, d, V, mb) == _bwd_size(T, d, V, mb)


@pytest.mark.parametrize("args", [(0, 256, 4096, 0), (-1, 256, 4096, 0), (10, 100, 4096, 0), (10, 256, 0, 0),
                                  (10, 256, 4096, 100), (10, 256, 4096, -128), (2 ** 22 + 1, 128, 256, 0),
                                  (10, 256, 2048 * 256 + 1, 0)])
def test_backward_workspace_size_zero_when_invalid(lib, args):
    assert lib.tim_logprobs_backward_workspace_size(*args) == 0


def _bwd(lib, **kw):
    g = lambda k, v: kw.get(k, v)
    T, d, V, mb = g("T", 8), g("d", 256), g("V", 4096), g("mb", 0)
    ws_bytes = g("ws_bytes", _bwd_size(max(T, 1), d, V, mb))
    return lib.tim_logprobs_backward(g("hidden", FAKE), g("w", FAKE), g("tokens", FAKE), T, d, V, g("tau", 1.0),
                                     g("lse", FAKE), g("ent", FAKE), g("gl", FAKE), g("ge", FAKE), mb,
                                     g("gh", FAKE), g("gw", FAKE), g("acc", 0), g("ws", FAKE), ws_bytes, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(d=100), Status.ERR_SHAPE),
    (dict(d=0), Status.ERR_SHAPE),
    (dict(V=0), Status.ERR_SHAPE),
    (dict(V=2048 * 256 + 1), Status.ERR_SHAPE),
    (dict(tau=0.0), Status.ERR_VALUE),
    (dict(tau=math.nan), Status.ERR_VALUE),
    (dict(mb=100), Status.ERR_VALUE),
    (dict(mb=-128), Status.ERR_VALUE),
    (dict(acc=2), Status.ERR_VALUE),
    (dict(gh=FAKE_MIS), Status.ERR_VALUE),
    (dict(gw=FAKE_MIS), Status.ERR_VALUE),
    (dict(T=2 ** 22 + 1, d=128, V=256), Status.ERR_VALUE),
    (dict(hidden=None), Status.ERR_NULL),
    (dict(w=None), Status.ERR_NULL),
    (dict(tokens=None), Status.ERR_NULL),
    (dict(lse=None), Status.ERR_NULL),
    (dict(gl=None), Status.ERR_NULL),
    (dict(ent=None), Status.ERR_NULL),          # grad_entropy given without entropy
    (dict(hidden=FAKE_MIS), Status.ERR_VALUE),
    (dict(w=FAKE_MIS), Status.ERR_VALUE),
    (dict(ws=None), Status.ERR_WORKSPACE),
    (dict(ws=FAKE_MIS), Status.ERR_WORKSPACE),
    (dict(ws_bytes=100), Status.ERR_WORKSPACE),
])
def test_backward_rejects(lib, kw, expect):
    assert _bwd(lib, **kw) == expect


def test_backward_noops(lib):
    # no outputs requested: validated, nothing enqueued (inputs never read)
    assert _bwd(lib, gh=None, gw=None, hidden=None, lse=None, ws=None) == Status.OK
    # T == 0 without a weight gradient to clear
    assert _bwd(lib, T=0, gw=None, hidden=None, ws=None) == Status.OK
    assert _bwd(lib, T=0, acc=1, hidden=None, ws=None) == Status.OK
    # entropy may be NULL when grad_entropy is
    assert _bwd(lib, ent=None, ge=None, gh=None, gw=None) == Status.OK


def _lg(lib, **kw):
    g = lambda k, v: kw.get(k, v)
    T = g("T", 8)
    return lib.tim_logit_grads(g("hidden", FAKE), g("w", FAKE), g("tokens", FAKE), T, g("d", 256), g("V", 4096),
                               g("tau", 1.0), g("lse", FAKE), g("ent", FAKE), g("gl", FAKE), g("ge", FAKE),
                               g("out", FAKE), g("ws", FAKE), g("ws_bytes", 16 * max(T, 1)), None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(d=200), Status.ERR_SHAPE),
    (dict(out=None), Status.ERR_NULL),
    (dict(lse=None), Status.ERR_NULL),
    (dict(ent=None), Status.ERR_NULL),
    (dict(out=FAKE_MIS), Status.ERR_VALUE),
    (dict(tau=-1.0), Status.ERR_VALUE),
    (dict(ws_bytes=16 * 8 - 1), Status.ERR_WORKSPACE),
])
def test_logit_grads_rejects(lib, kw, expect):
    assert _lg(lib, **kw) == expect
    assert _lg(lib, T=0, out=None, hidden=None) == Status.OK


# ---------------------------------------------------------------- final RMS norm

@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(T=65535 * 256 + 1), Status.ERR_SHAPE),
    (dict(d=0), Status.ERR_SHAPE),
    (dict(d=12), Status.ERR_SHAPE),
    (dict(eps=-1e-6), Status.ERR_VALUE),
    (dict(eps=math.nan), Status.ERR_VALUE),
    (dict(eps=math.inf), Status.ERR_VALUE),
    (dict(x=None), Status.ERR_NULL),
    (dict(h=None), Status.ERR_NULL),
    (dict(x=FAKE_MIS), Status.ERR_VALUE),
    (dict(h=FAKE_MIS), Status.ERR_VALUE),
    (dict(gamma=FAKE_MIS), Status.ERR_VALUE),
])
def test_rmsnorm_rejects(lib, kw, expect):
    g = lambda k, v: kw.get(k, v)
    assert lib.tim_rmsnorm(g("x", FAKE), g("gamma", None), g("T", 8), g("d", 256), g("eps", 1e-6), g("h", FAKE),
                           None, None) == expect


def test_rmsnorm_T_zero_is_noop(lib):
    assert lib.tim_rmsnorm(None, None, 0, 256, 1e-6, None, None, None) == Status.OK


def _nb(lib, **kw):
    g = lambda k, v: kw.get(k, v)
    T, d = g("T", 8), g("d", 256)
    return lib.tim_rmsnorm_backward(g("x", FAKE), g("gamma", None), g("rstd", FAKE), g("gh", FAKE), T, d,
                                    g("gx", FAKE), g("gg", FAKE), g("acc", 0), g("ws", FAKE),
                                    g("ws_bytes", ((T + 255) // 256) * d * 4), None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(d=4), Status.ERR_SHAPE),
    (dict(acc=3), Status.ERR_VALUE),
    (dict(x=None), Status.ERR_NULL),
    (dict(rstd=None), Status.ERR_NULL),
    (dict(gh=None), Status.ERR_NULL),
    (dict(gh=FAKE_MIS), Status.ERR_VALUE),
    (dict(gx=FAKE_MIS), Status.ERR_VALUE),
    (dict(ws=None), Status.ERR_WORKSPACE),
    (dict(ws_bytes=100), Status.ERR_WORKSPACE),
])
def test_rmsnorm_backward_rejects(lib, kw, expect):
    assert _nb(lib, **kw) == expect


def test_rmsnorm_backward_noops_and_workspace(lib):
    assert _nb(lib, gx=None, gg=None, x=None, ws=None) == Status.OK
    assert _nb(lib, gg=None, ws=None, gx=None) == Status.OK
    assert _nb(lib, T=0, gx=None, acc=1, x=None, ws=None) == Status.OK
    assert lib.tim_rmsnorm_backward_workspace_size(1000, 4096) == 4 * 4096 * 4
    assert lib.tim_rmsnorm_backward_workspace_size(0, 4096) == 0
    assert lib.tim_rmsnorm_backward_workspace_size(10, 12) == 0


# ---------------------------------------------------------------- PPO / GRPO loss

def _ppo(lib, **kw):
    g = lambda k, v: kw.get(k, v)
    return lib.tim_ppo_loss(g("lp", FAKE), g("lo", FAKE), g("adv", FAKE), None, g("T", 8), g("cu", FAKE), g("n", 2),
                            g("el", 0.2), g("eh", 0.2), g("seq", FAKE), g("batch", None), None, None, None, None, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(T=-1), Status.ERR_SHAPE),
    (dict(n=-1), Status.ERR_SHAPE),
    (dict(n=2 ** 31), Status.ERR_SHAPE),
    (dict(el=-0.1), Status.ERR_VALUE),
    (dict(el=1.0), Status.ERR_VALUE),
    (dict(eh=-0.1), Status.ERR_VALUE),
    (dict(eh=math.nan), Status.ERR_VALUE),
    (dict(cu=None), Status.ERR_NULL),
    (dict(lp=None), Status.ERR_NULL),
    (dict(lo=None), Status.ERR_NULL),
    (dict(adv=None), Status.ERR_NULL),
    (dict(seq=None, batch=FAKE), Status.ERR_NULL),
])
def test_ppo_rejects(lib, kw, expect):
    assert _ppo(lib, **kw) == expect


def test_ppo_noops(lib):
    assert _ppo(lib, n=0, cu=None, lp=None) == Status.OK
    assert _ppo(lib, seq=None) == Status.OK          # no outputs requested
