"""Python binding of libtim.so: batch-invariant fused LM-head token log-probs
and training-inference mismatch statistics on MI355X (gfx950).

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI (include/tim.h). Tensors must live on the GPU; the
calls are enqueued on torch's current stream. There is no fallback: when the
library is missing or no GPU is present the calls raise.
"""

from __future__ import annotations

import ctypes
import enum
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtim.so")

VOCAB_TILE = 256
MAX_VOCAB = 2048 * VOCAB_TILE


class Status(enum.IntEnum):
    OK = 0
    ERR_NULL = 1
    ERR_SHAPE = 2
    ERR_VALUE = 3
    ERR_WORKSPACE = 4
    ERR_HIP = 5


class Mode(enum.IntEnum):
    ROLLOUT = 0
    TRAINING = 1


class Order(enum.IntEnum):
    INVARIANT = 0
    SPLITK4 = 1


class Estimator(enum.IntEnum):
    K1 = 1
    K3 = 3


class TimError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = Status(status)


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libtim.so and declare its C signatures. Raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2605_14220_amd.build`")
    lib = ctypes.CDLL(path)
    c = ctypes
    lib.tim_logprobs_rows_per_launch.restype = c.c_int64
    lib.tim_logprobs_rows_per_launch.argtypes = [c.c_int64, c.c_int32, c.c_int32, c.c_int64]
    lib.tim_logprobs_workspace_size.restype = c.c_size_t
    lib.tim_logprobs_workspace_size.argtypes = [c.c_int64, c.c_int32, c.c_int32, c.c_int32, c.c_int64]
    lib.tim_logprobs.restype = c.c_int
    lib.tim_logprobs.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32,
                                 c.c_float, c.c_int32, c.c_int64, c.c_int32, c.c_void_p, c.c_void_p,
                                 c.c_void_p, c.c_void_p, c.c_size_t, c.c_void_p]
    lib.tim_logprobs_noalloc.restype = c.c_int
    lib.tim_logprobs_noalloc.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32,
                                         c.c_float, c.c_int32, c.c_int64, c.c_int32, c.c_void_p, c.c_void_p,
                                         c.c_void_p, c.c_void_p]
    lib.tim_logprobs_partials.restype = c.c_int
    lib.tim_logprobs_partials.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32,
                                          c.c_int32, c.c_float, c.c_int32, c.c_int32, c.c_void_p,
                                          c.c_size_t, c.c_void_p]
    lib.tim_logprobs_merge.restype = c.c_int
    lib.tim_logprobs_merge.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32,
                                       c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p]
    lib.tim_mismatch.restype = c.c_int
    lib.tim_mismatch.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_float, c.c_void_p, c.c_void_p,
                                 c.c_void_p, c.c_void_p]
    lib.tim_mismatch_seq.restype = c.c_int
    lib.tim_mismatch_seq.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_void_p, c.c_int64, c.c_int32,
                                     c.c_float, c.c_double, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p]
    lib.tim_logprobs_backward_workspace_size.restype = c.c_size_t
    lib.tim_logprobs_backward_workspace_size.argtypes = [c.c_int64, c.c_int32, c.c_int32, c.c_int64]
    lib.tim_logprobs_backward.restype = c.c_int
    lib.tim_logprobs_backward.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32,
                                          c.c_float, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64,
                                          c.c_void_p, c.c_void_p, c.c_int32, c.c_void_p, c.c_size_t, c.c_void_p]
    lib.tim_logit_grads.restype = c.c_int
    lib.tim_logit_grads.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32,
                                    c.c_float, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p,
                                    c.c_void_p, c.c_size_t, c.c_void_p]
    lib.tim_rmsnorm.restype = c.c_int
    lib.tim_rmsnorm.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_float, c.c_void_p, c.c_void_p,
                                c.c_void_p]
    lib.tim_rmsnorm_backward_workspace_size.restype = c.c_size_t
    lib.tim_rmsnorm_backward_workspace_size.argtypes = [c.c_int64, c.c_int32]
    lib.tim_rmsnorm_backward.restype = c.c_int
    lib.tim_rmsnorm_backward.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_int32,
                                         c.c_void_p, c.c_void_p, c.c_int32, c.c_void_p, c.c_size_t, c.c_void_p]
    lib.tim_ppo_loss.restype = c.c_int
    lib.tim_ppo_loss.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64, c.c_void_p, c.c_int64,
                                 c.c_float, c.c_float, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p, c.c_void_p,
                                 c.c_void_p, c.c_void_p]
    lib.tim_logits.restype = c.c_int
    lib.tim_logits.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_int32, c.c_int32, c.c_float,
                               c.c_int32, c.c_void_p, c.c_void_p]
    lib.tim_status_string.restype = c.c_char_p
    lib.tim_status_string.argtypes = [c.c_int]
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        msg = load_library().tim_status_string(status).decode()
        raise TimError(status, msg)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _require_gpu(*tensors):
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise ValueError("tim: tensors must be on the GPU")
        if t is not None and not t.is_contiguous():
            raise ValueError("tim: tensors must be contiguous")


def rows_per_launch(T: int, d: int, mode: Mode = Mode.TRAINING, micro_batch: int = 0) -> int:
    """Rows tim_logprobs hands to one launch (0 for invalid arguments); see include/tim.h."""
    return int(load_library().tim_logprobs_rows_per_launch(int(T), int(d), int(mode), int(micro_batch)))


def workspace_size(T: int, d: int, V: int, mode: Mode = Mode.TRAINING, micro_batch: int = 0) -> int:
    """Bytes of workspace tim_logprobs needs (0 for T == 0 or invalid shapes)."""
    return int(load_library().tim_logprobs_workspace_size(int(T), int(d), int(V), int(mode), int(micro_batch)))


def logprobs(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor, temperature: float = 1.0,
             mode: Mode = Mode.TRAINING, micro_batch: int = 0, order: Order = Order.INVARIANT,
             entropy: bool = True, lse: bool = False, workspace: torch.Tensor | None = None,
             out: tuple | None = None):
    """Token log-probabilities (and entropies, log-normalisers) of T rows.

    hidden bf16 [T, d], w_vocab bf16 [V, d], tokens int32 [T], all on one GPU.
    Returns (logp, entropy or None, lse or None), fp32 [T] each."""
    lib = load_library()
    if hidden.dtype != torch.bfloat16 or w_vocab.dtype != torch.bfloat16:
        raise TypeError("tim.logprobs: hidden and w_vocab must be bfloat16")
    if tokens.dtype != torch.int32:
        raise TypeError("tim.logprobs: tokens must be int32")
    if hidden.dim() != 2 or w_vocab.dim() != 2 or hidden.shape[1] != w_vocab.shape[1]:
        raise ValueError("tim.logprobs: hidden [T, d] and w_vocab [V, d] must share d")
    T, d = hidden.shape
    V = w_vocab.shape[0]
    if tokens.shape != (T,):
        raise ValueError("tim.logprobs: tokens must be [T]")
    _require_gpu(hidden, w_vocab, tokens, workspace)
    dev = hidden.device
    if out is None:
        lp = torch.empty(T, dtype=torch.float32, device=dev)
        ent = torch.empty(T, dtype=torch.float32, device=dev) if entropy else None
        ls = torch.empty(T, dtype=torch.float32, device=dev) if lse else None
    else:
        lp, ent, ls = out
        _require_gpu(lp, ent, ls)
    if T == 0:
        return lp, ent, ls
    need = workspace_size(T, d, V, mode, micro_batch)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib.tim_logprobs(_ptr(hidden), _ptr(w_vocab), _ptr(tokens), T, d, V, float(temperature),
                            int(mode), int(micro_batch), int(order), _ptr(lp), _ptr(ent), _ptr(ls),
                            _ptr(workspace), ws_bytes, _stream(dev)))
    return lp, ent, ls


NOALLOC_SCRATCH_BYTES = 64 << 20  # TIM_NOALLOC_SCRATCH_BYTES


def logprobs_noalloc(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor, temperature: float = 1.0,
                     mode: Mode = Mode.TRAINING, micro_batch: int = 0, order: Order = Order.INVARIANT,
                     out: tuple | None = None):
    """tim_logprobs_noalloc: logprobs() with the partials in the library's per-GPU device array instead of a
    workspace (the call allocates no device memory; pass `out` = (logp, entropy or None, lse or None) to keep
    the binding from allocating the outputs). Needs workspace_size(T, d, V, mode, micro_batch) <=
    NOALLOC_SCRATCH_BYTES."""
    lib = load_library()
    if hidden.dtype != torch.bfloat16 or w_vocab.dtype != torch.bfloat16:
        raise TypeError("tim.logprobs_noalloc: hidden and w_vocab must be bfloat16")
    if tokens.dtype != torch.int32:
        raise TypeError("tim.logprobs_noalloc: tokens must be int32")
    if hidden.dim() != 2 or w_vocab.dim() != 2 or hidden.shape[1] != w_vocab.shape[1]:
        raise ValueError("tim.logprobs_noalloc: hidden [T, d] and w_vocab [V, d] must share d")
    T, d = hidden.shape
    V = w_vocab.shape[0]
    if tokens.shape != (T,):
        raise ValueError("tim.logprobs_noalloc: tokens must be [T]")
    _require_gpu(hidden, w_vocab, tokens)
    dev = hidden.device
    if out is None:
        out = (torch.empty(T, dtype=torch.float32, device=dev), torch.empty(T, dtype=torch.float32, device=dev),
               None)
    lp, ent, ls = out
    _require_gpu(lp, ent, ls)
    _check(lib.tim_logprobs_noalloc(_ptr(hidden), _ptr(w_vocab), _ptr(tokens), T, d, V, float(temperature),
                                    int(mode), int(micro_batch), int(order), _ptr(lp), _ptr(ent), _ptr(ls),
                                    _stream(dev)))
    return lp, ent, ls


def logprobs_partials(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor,
                      workspace: torch.Tensor, temperature: float = 1.0, mode: Mode = Mode.TRAINING,
                      order: Order = Order.INVARIANT):
    """First stage of logprobs over all rows in one launch: per-(row, vocab tile)
    partials written into `workspace` (see include/tim.h)."""
    lib = load_library()
    _require_gpu(hidden, w_vocab, tokens, workspace)
    T, d = hidden.shape
    V = w_vocab.shape[0]
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib.tim_logprobs_partials(_ptr(hidden), _ptr(w_vocab), _ptr(tokens), T, d, V, float(temperature),
                                     int(mode), int(order), _ptr(workspace), ws_bytes, _stream(hidden.device)))


def logprobs_merge(workspace: torch.Tensor, tokens: torch.Tensor, V: int, order: Order = Order.INVARIANT,
                   out: tuple | None = None):
    """Second stage: partials in `workspace` -> (logp, entropy, lse) for len(tokens) rows."""
    lib = load_library()
    _require_gpu(workspace, tokens)
    T = tokens.numel()
    if out is None:
        out = tuple(torch.empty(T, dtype=torch.float32, device=tokens.device) for _ in range(3))
    _require_gpu(*out)
    _check(lib.tim_logprobs_merge(_ptr(workspace), _ptr(tokens), T, int(V), int(order), _ptr(out[0]),
                                  _ptr(out[1]), _ptr(out[2]), _stream(tokens.device)))
    return out


def mismatch(logp_a: torch.Tensor, logp_b: torch.Tensor, C: float = 2.0, out: tuple | None = None):
    """(log_ratio, k3, is_weight) fp32 [T]: delta = a - b, k3 = expm1(delta) - delta,
    w = min(exp(delta), C). a is the trainer's log-prob, b the rollout engine's."""
    lib = load_library()
    if logp_a.dtype != torch.float32 or logp_b.dtype != torch.float32 or logp_a.shape != logp_b.shape:
        raise TypeError("tim.mismatch: logp_a and logp_b must be fp32 of one shape")
    _require_gpu(logp_a, logp_b)
    T = logp_a.numel()
    if out is None:
        out = tuple(torch.empty_like(logp_a) for _ in range(3))
    _require_gpu(*out)
    _check(lib.tim_mismatch(_ptr(logp_a), _ptr(logp_b), T, float(C), _ptr(out[0]), _ptr(out[1]),
                            _ptr(out[2]), _stream(logp_a.device)))
    return out


def mismatch_seq(logp_a: torch.Tensor, logp_b: torch.Tensor, cu_seqlens: torch.Tensor, C: float = 2.0,
                 tau_seq: float = 1e-3, estimator: Estimator = Estimator.K3, out: tuple | None = None):
    """Per-response mismatch score, keep mask and per-token weights of a packed stream.

    logp_a (trainer) and logp_b (rollout) fp32 [T]; cu_seqlens int64 [n + 1] offsets of the
    n responses. Returns (score fp64 [n], keep uint8 [n], weight fp32 [T]) with
    score = sum_t K(delta_t) (K1 = -delta, K3 = expm1(delta) - delta), keep = score <= tau_seq,
    weight = keep * min(exp(delta), C). See include/tim.h."""
    lib = load_library()
    if logp_a.dtype != torch.float32 or logp_b.dtype != torch.float32 or logp_a.shape != logp_b.shape:
        raise TypeError("tim.mismatch_seq: logp_a and logp_b must be fp32 of one shape")
    if cu_seqlens.dtype != torch.int64 or cu_seqlens.dim() != 1 or cu_seqlens.numel() < 1:
        raise TypeError("tim.mismatch_seq: cu_seqlens must be a non-empty int64 vector")
    _require_gpu(logp_a, logp_b, cu_seqlens)
    T = logp_a.numel()
    n = cu_seqlens.numel() - 1
    dev = logp_a.device
    if out is None:
        out = (torch.empty(n, dtype=torch.float64, device=dev), torch.empty(n, dtype=torch.uint8, device=dev),
               torch.zeros(T, dtype=torch.float32, device=dev))
    _require_gpu(*out)
    _check(lib.tim_mismatch_seq(_ptr(logp_a), _ptr(logp_b), T, _ptr(cu_seqlens), n, int(estimator), float(C),
                                float(tau_seq), _ptr(out[0]), _ptr(out[1]), _ptr(out[2]), _stream(dev)))
    return out


def logits(hidden: torch.Tensor, w_vocab: torch.Tensor, temperature: float = 1.0,
           order: Order = Order.INVARIANT) -> torch.Tensor:
    """fp32 [T, V] logits exactly as tim_logprobs forms them (test/debug aid)."""
    lib = load_library()
    _require_gpu(hidden, w_vocab)
    T, d = hidden.shape
    V = w_vocab.shape[0]
    z = torch.empty((T, V), dtype=torch.float32, device=hidden.device)
    _check(lib.tim_logits(_ptr(hidden), _ptr(w_vocab), T, d, V, float(temperature), int(order), _ptr(z),
                          _stream(hidden.device)))
    return z


def backward_workspace_size(T: int, d: int, V: int, micro_batch: int = 0) -> int:
    """Bytes of workspace tim_logprobs_backward needs (0 for T == 0 or invalid arguments)."""
    return int(load_library().tim_logprobs_backward_workspace_size(int(T), int(d), int(V), int(micro_batch)))


def _grad_inputs(name, hidden, w_vocab, tokens, lse, grad_logp, entropy, grad_entropy):
    if hidden.dtype != torch.bfloat16 or w_vocab.dtype != torch.bfloat16:
        raise TypeError(f"tim.{name}: hidden and w_vocab must be bfloat16")
    if tokens.dtype != torch.int32:
        raise TypeError(f"tim.{name}: tokens must be int32")
    if hidden.dim() != 2 or w_vocab.dim() != 2 or hidden.shape[1] != w_vocab.shape[1]:
        raise ValueError(f"tim.{name}: hidden [T, d] and w_vocab [V, d] must share d")
    T = hidden.shape[0]
    for t in (tokens, lse, grad_logp, entropy, grad_entropy):
        if t is not None and t.shape != (T,):
            raise ValueError(f"tim.{name}: per-row arrays must be [T]")
    for t in (lse, grad_logp, entropy, grad_entropy):
        if t is not None and t.dtype != torch.float32:
            raise TypeError(f"tim.{name}: lse, entropy and the upstream gradients must be fp32")
    _require_gpu(hidden, w_vocab, tokens, lse, grad_logp, entropy, grad_entropy)


def logprobs_backward(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor, lse: torch.Tensor,
                      grad_logp: torch.Tensor, temperature: float = 1.0, entropy: torch.Tensor | None = None,
                      grad_entropy: torch.Tensor | None = None, micro_batch: int = 0, want_hidden: bool = True,
                      want_w: bool = True, grad_w: torch.Tensor | None = None, accumulate: bool = False,
                      workspace: torch.Tensor | None = None):
    """Gradients of sum_t grad_logp[t] logp[t] + grad_entropy[t] entropy[t] with respect
    to hidden [T, d] and w_vocab [V, d], as fp32 (grad_hidden or None, grad_w or None).

    lse (and entropy, when grad_entropy is given) are tim.logprobs' outputs for the same
    inputs. grad_w, if given, is the fp32 [V, d] output buffer; with accumulate=True the
    gradient is added to its contents. See include/tim.h."""
    lib = load_library()
    _grad_inputs("logprobs_backward", hidden, w_vocab, tokens, lse, grad_logp, entropy, grad_entropy)
    T, d = hidden.shape
    V = w_vocab.shape[0]
    dev = hidden.device
    gh = torch.empty((T, d), dtype=torch.float32, device=dev) if want_hidden else None
    if want_w and grad_w is None:
        if accumulate:
            raise ValueError("tim.logprobs_backward: accumulate needs the grad_w buffer")
        grad_w = torch.empty((V, d), dtype=torch.float32, device=dev)
    gw = grad_w if want_w else None
    if gw is not None and (gw.dtype != torch.float32 or gw.shape != (V, d)):
        raise ValueError("tim.logprobs_backward: grad_w must be fp32 [V, d]")
    _require_gpu(gh, gw, workspace)
    need = backward_workspace_size(T, d, V, micro_batch)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib.tim_logprobs_backward(_ptr(hidden), _ptr(w_vocab), _ptr(tokens), T, d, V, float(temperature),
                                     _ptr(lse), _ptr(entropy), _ptr(grad_logp), _ptr(grad_entropy),
                                     int(micro_batch), _ptr(gh), _ptr(gw), 1 if accumulate else 0,
                                     _ptr(workspace), ws_bytes, _stream(dev)))
    return gh, gw


def logit_grads(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor, lse: torch.Tensor,
                grad_logp: torch.Tensor, temperature: float = 1.0, entropy: torch.Tensor | None = None,
                grad_entropy: torch.Tensor | None = None) -> torch.Tensor:
    """bf16 [T, ceil(V / 256) * 256] gradients with respect to the LM-head contraction,
    exactly as the backward's first pass forms them (test/debug aid)."""
    lib = load_library()
    _grad_inputs("logit_grads", hidden, w_vocab, tokens, lse, grad_logp, entropy, grad_entropy)
    T, d = hidden.shape
    V = w_vocab.shape[0]
    dev = hidden.device
    v_pad = (V + VOCAB_TILE - 1) // VOCAB_TILE * VOCAB_TILE
    out = torch.empty((T, v_pad), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(max(T * 16, 16), dtype=torch.uint8, device=dev)
    _check(lib.tim_logit_grads(_ptr(hidden), _ptr(w_vocab), _ptr(tokens), T, d, V, float(temperature), _ptr(lse),
                               _ptr(entropy), _ptr(grad_logp), _ptr(grad_entropy), _ptr(out), _ptr(ws),
                               ws.numel(), _stream(dev)))
    return out


def rmsnorm(x: torch.Tensor, gamma: torch.Tensor | None = None, eps: float = 1e-6, out: torch.Tensor | None = None):
    """Final RMS norm: (h bf16 [T, d], rstd fp32 [T]) of x bf16 [T, d] (see include/tim.h)."""
    lib = load_library()
    if x.dtype != torch.bfloat16 or x.dim() != 2 or (gamma is not None and gamma.dtype != torch.bfloat16):
        raise TypeError("tim.rmsnorm: x must be bf16 [T, d] and gamma bf16 [d]")
    T, d = x.shape
    if gamma is not None and gamma.shape != (d,):
        raise ValueError("tim.rmsnorm: gamma must be [d]")
    _require_gpu(x, gamma, out)
    h = torch.empty_like(x) if out is None else out
    rstd = torch.empty(T, dtype=torch.float32, device=x.device)
    _check(lib.tim_rmsnorm(_ptr(x), _ptr(gamma), T, d, float(eps), _ptr(h), _ptr(rstd), _stream(x.device)))
    return h, rstd


def rmsnorm_backward(x: torch.Tensor, gamma: torch.Tensor | None, rstd: torch.Tensor, grad_h: torch.Tensor,
                     want_x: bool = True, want_gamma: bool = True, grad_gamma: torch.Tensor | None = None,
                     accumulate: bool = False):
    """(grad_x fp32 [T, d] or None, grad_gamma fp32 [d] or None) of the final RMS norm."""
    lib = load_library()
    T, d = x.shape
    if grad_h.dtype != torch.float32 or grad_h.shape != (T, d) or rstd.shape != (T,):
        raise ValueError("tim.rmsnorm_backward: grad_h fp32 [T, d] and rstd [T]")
    _require_gpu(x, gamma, rstd, grad_h, grad_gamma)
    dev = x.device
    gx = torch.empty((T, d), dtype=torch.float32, device=dev) if want_x else None
    if want_gamma and grad_gamma is None:
        if accumulate:
            raise ValueError("tim.rmsnorm_backward: accumulate needs the grad_gamma buffer")
        grad_gamma = torch.empty(d, dtype=torch.float32, device=dev)
    gg = grad_gamma if want_gamma else None
    ws = torch.empty(max(int(lib.tim_rmsnorm_backward_workspace_size(T, d)), 16), dtype=torch.uint8, device=dev)
    _check(lib.tim_rmsnorm_backward(_ptr(x), _ptr(gamma), _ptr(rstd), _ptr(grad_h), T, d, _ptr(gx), _ptr(gg),
                                    1 if accumulate else 0, _ptr(ws), ws.numel(), _stream(dev)))
    return gx, gg


def logprobs_from_residual(x: torch.Tensor, gamma: torch.Tensor | None, w_vocab: torch.Tensor, tokens: torch.Tensor,
                           eps: float = 1e-6, temperature: float = 1.0, **kw):
    """The final norm followed by the LM-head log-probs: (logp, entropy, lse, h, rstd).
    Two C-ABI calls on the same stream; keyword arguments go to logprobs()."""
    h, rstd = rmsnorm(x, gamma, eps)
    lp, ent, lse = logprobs(h, w_vocab, tokens, temperature, **kw)
    return lp, ent, lse, h, rstd


def ppo_loss(logp: torch.Tensor, logp_old: torch.Tensor, advantages: torch.Tensor, cu_seqlens: torch.Tensor,
             eps_low: float = 0.2, eps_high: float = 0.2, weight: torch.Tensor | None = None,
             out: dict | None = None) -> dict:
    """Clipped PPO/GRPO loss of a packed stream (see include/tim.h): dict with seq_loss fp64 [n],
    batch_loss fp64 [1], token_loss / grad / contribution fp32 [T] and clipped uint8 [T]
    (freshly allocated outputs are zero outside every response; `out` reuses a previous dict)."""
    lib = load_library()
    for t in (logp, logp_old, advantages, weight):
        if t is not None and (t.dtype != torch.float32 or t.shape != logp.shape):
            raise TypeError("tim.ppo_loss: per-token inputs must be fp32 of one shape")
    if cu_seqlens.dtype != torch.int64 or cu_seqlens.dim() != 1 or cu_seqlens.numel() < 1:
        raise TypeError("tim.ppo_loss: cu_seqlens must be a non-empty int64 vector")
    _require_gpu(logp, logp_old, advantages, weight, cu_seqlens)
    T = logp.numel()
    n = cu_seqlens.numel() - 1
    dev = logp.device
    if out is not None:
        _require_gpu(*out.values())
    out = out or {"seq_loss": torch.zeros(n, dtype=torch.float64, device=dev),
           "batch_loss": torch.zeros(1, dtype=torch.float64, device=dev),
           "token_loss": torch.zeros(T, dtype=torch.float32, device=dev),
           "grad": torch.zeros(T, dtype=torch.float32, device=dev),
           "contribution": torch.zeros(T, dtype=torch.float32, device=dev),
           "clipped": torch.zeros(T, dtype=torch.uint8, device=dev)}
    _check(lib.tim_ppo_loss(_ptr(logp), _ptr(logp_old), _ptr(advantages), _ptr(weight), T, _ptr(cu_seqlens), n,
                            float(eps_low), float(eps_high), _ptr(out["seq_loss"]), _ptr(out["batch_loss"]),
                            _ptr(out["token_loss"]), _ptr(out["grad"]), _ptr(out["contribution"]),
                            _ptr(out["clipped"]), _stream(dev)))
    return out
