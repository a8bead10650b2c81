"""ctypes binding of libforkstep.so (the C ABI in include/fork_step.h).

Argument marshalling only: shapes, dtypes, devices and contiguity are checked,
then raw device pointers and the current HIP stream are handed to the library,
where every step of the computation runs in HIP kernels.  There is no CPU or
PyTorch fallback: if the library is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libforkstep.so")

FORK_OK = 0
FORK_EINVAL = -1
FORK_EUNSUPPORTED = -2
FORK_EHIP = -3
FORK_ENOMEM = -4
FORK_BF16 = 0
FORK_F32 = 1
FORK_RULE_LEFTMOST = 0
FORK_RULE_MAXCONF = 1
FORK_RULE_MINCONF = 2
FORK_RULE_MAXENT = 3
FORK_RULE_RANDOM = 4
FORK_ROWS_ALL = 0
FORK_ROWS_ACTIVE = 1
FORK_NOALLOC_SCRATCH_BYTES = 64 << 20
FORK_LAYOUT_ROW_MAJOR = 0
FORK_LAYOUT_POSITION_MAJOR = 1

_P = ctypes.c_void_p
_I32 = ctypes.c_int32


class ForkStepArgs(ctypes.Structure):
    _fields_ = [
        ("hidden", _P), ("W_head", _P), ("tokens", _P), ("mask", _P),
        ("block_start", _P), ("block_len", _I32), ("tau", ctypes.c_float),
        ("out_conf", _P), ("out_entropy", _P), ("out_logp", _P),
        ("out_fallback", _P),
        ("B", _I32), ("L", _I32), ("d", _I32), ("V", _I32), ("dtype", _I32),
        ("stream", _P),
        ("out_lse", _P), ("out_argmax", _P), ("out_ncommit", _P),
        ("out_commit_pos", _P), ("rule", _I32),
        ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
        ("ev_lmhead_begin", _P), ("ev_lmhead_end", _P),
        ("fallback_uniform", _P), ("rows_mode", _I32),
        ("sample_temperature", ctypes.c_float), ("sample_counter", ctypes.c_uint32),
        ("sample_seed", ctypes.c_uint64),
    ]


class ForkLogprobArgs(ctypes.Structure):
    _fields_ = [
        ("hidden", _P), ("W_head", _P), ("rows", _P), ("tokens", _P),
        ("out_logp", _P), ("out_q", _P), ("out_entropy", _P), ("out_lse", _P),
        ("n", _I32), ("M", _I32), ("d", _I32), ("V", _I32), ("dtype", _I32),
        ("stream", _P), ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
        ("ev_lmhead_begin", _P), ("ev_lmhead_end", _P),
    ]


class ForkGrpoArgs(ctypes.Structure):
    _fields_ = [
        ("n_groups", _I32), ("G", _I32), ("n", _I32),
        ("rewards", _P), ("offsets", _P), ("lp_new", _P), ("lp_old", _P),
        ("eps", ctypes.c_float),
        ("out_adv", _P), ("out_ratio", _P), ("out_term", _P), ("out_rollout_obj", _P),
        ("out_group_obj", _P), ("out_skipped", _P), ("out_J", _P),
        ("stream", _P),
    ]


class ForkSelectArgs(ctypes.Structure):
    _fields_ = [
        ("conf", _P), ("entropy", _P), ("uniform", _P), ("argmax", _P),
        ("tokens", _P), ("mask", _P), ("block_start", _P),
        ("out_fallback", _P), ("out_ncommit", _P), ("out_commit_pos", _P),
        ("B", _I32), ("L", _I32), ("block_len", _I32), ("tau", ctypes.c_float),
        ("rule", _I32), ("stream", _P), ("layout", _I32),
    ]


class ForkError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("fork_step failed (%d): %s" % (code, msg))
        self.code = code


_lib = None


def lib():
    """Load libforkstep.so (after torch, so that the HIP runtime torch already
    loaded is the one the library binds to)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libforkstep.so is not built (expected at %s); run "
                "`python -c 'import __graft_entry__ as g; g.build()'` or "
                "`python -m paper_2609_39859_amd.build`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        L.fork_step.restype = ctypes.c_int
        L.fork_step.argtypes = [_P, _P, _P, _P, _P, _I32, ctypes.c_float, _P, _P,
                                _P, _P, _I32, _I32, _I32, _I32, _I32, _P]
        L.fork_step_ex.restype = ctypes.c_int
        L.fork_step_ex.argtypes = [ctypes.POINTER(ForkStepArgs)]
        L.fork_step_noalloc.restype = ctypes.c_int
        L.fork_step_noalloc.argtypes = [ctypes.POINTER(ForkStepArgs)]
        L.fork_workspace_bytes.restype = ctypes.c_size_t
        L.fork_workspace_bytes.argtypes = [_I32, _I32, _I32]
        L.fork_last_error.restype = ctypes.c_char_p
        L.fork_last_error.argtypes = []
        L.fork_release.restype = None
        L.fork_release.argtypes = []
        L.fork_version.restype = ctypes.c_int
        L.fork_version.argtypes = []
        L.fork_logprob.restype = ctypes.c_int
        L.fork_logprob.argtypes = [ctypes.POINTER(ForkLogprobArgs)]
        L.fork_logprob_workspace_bytes.restype = ctypes.c_size_t
        L.fork_logprob_workspace_bytes.argtypes = [_I32, _I32]
        L.fork_grpo_objective.restype = ctypes.c_int
        L.fork_grpo_objective.argtypes = [ctypes.POINTER(ForkGrpoArgs)]
        L.fork_select.restype = ctypes.c_int
        L.fork_select.argtypes = [ctypes.POINTER(ForkSelectArgs)]
        L.fork_top_entropy.restype = ctypes.c_int
        L.fork_top_entropy.argtypes = [_P, _I32, _I32, _I32, _P, _P]
        _lib = L
    return _lib


def _check(t: torch.Tensor, name: str, dtype, numel: int, device) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (name, t.numel(), numel))
    return t.data_ptr()


def _opt(t: Optional[torch.Tensor], name, dtype, numel, device):
    return None if t is None else _check(t, name, dtype, numel, device)


def _stream_handle(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream


def fork_step(hidden: torch.Tensor, W_head: torch.Tensor, tokens: torch.Tensor,
              mask: torch.Tensor, block_start: torch.Tensor, block_len: int,
              tau: float, out_conf: torch.Tensor, out_entropy: torch.Tensor,
              out_logp: torch.Tensor, out_fallback: torch.Tensor, *,
              B: int, L: int, stream=None) -> None:
    """One denoising step on the GPU (see include/fork_step.h, fork_step)."""
    fork_step_ex(hidden, W_head, tokens, mask, block_start, block_len, tau,
                 out_conf, out_entropy, out_logp, out_fallback, B=B, L=L,
                 stream=stream)


def fork_step_ex(hidden: torch.Tensor, W_head: torch.Tensor, tokens: torch.Tensor,
                 mask: torch.Tensor, block_start: torch.Tensor, block_len: int,
                 tau: float, out_conf: torch.Tensor, out_entropy: torch.Tensor,
                 out_logp: torch.Tensor, out_fallback: torch.Tensor, *,
                 B: int, L: int, out_lse=None, out_argmax=None, out_ncommit=None,
                 out_commit_pos=None, rule: int = FORK_RULE_LEFTMOST,
                 workspace: Optional[torch.Tensor] = None, stream=None,
                 events=None, fallback_uniform=None, rows_mode: int = FORK_ROWS_ALL,
                 temperature: float = 0.0, seed: int = 0, counter: int = 0) -> None:
    """fork_step_ex of the C ABI; optional outputs may be None.  ``events``
    is an optional pair of raw hipEvent_t handles (ints) recorded around the
    LM-head kernel."""
    a = _step_args(hidden, W_head, tokens, mask, block_start, block_len, tau, out_conf,
                   out_entropy, out_logp, out_fallback, B, L, out_lse, out_argmax,
                   out_ncommit, out_commit_pos, rule, workspace, stream, events,
                   fallback_uniform, rows_mode, temperature, seed, counter)
    _raise_on(lib().fork_step_ex(ctypes.byref(a)))


def fork_step_noalloc(hidden: torch.Tensor, W_head: torch.Tensor, tokens: torch.Tensor,
                      mask: torch.Tensor, block_start: torch.Tensor, block_len: int,
                      tau: float, out_conf: torch.Tensor, out_entropy: torch.Tensor,
                      out_logp: torch.Tensor, out_fallback: torch.Tensor, *,
                      B: int, L: int, out_lse=None, out_argmax=None, out_ncommit=None,
                      out_commit_pos=None, rule: int = FORK_RULE_LEFTMOST, stream=None,
                      events=None, fallback_uniform=None, rows_mode: int = FORK_ROWS_ALL,
                      temperature: float = 0.0, seed: int = 0, counter: int = 0) -> None:
    """fork_step_noalloc of the C ABI: fork_step_ex on the library's static
    device scratch (allocates nothing)."""
    a = _step_args(hidden, W_head, tokens, mask, block_start, block_len, tau, out_conf,
                   out_entropy, out_logp, out_fallback, B, L, out_lse, out_argmax,
                   out_ncommit, out_commit_pos, rule, None, stream, events,
                   fallback_uniform, rows_mode, temperature, seed, counter)
    _raise_on(lib().fork_step_noalloc(ctypes.byref(a)))


def _step_args(hidden, W_head, tokens, mask, block_start, block_len, tau, out_conf,
               out_entropy, out_logp, out_fallback, B, L, out_lse, out_argmax, out_ncommit,
               out_commit_pos, rule, workspace, stream, events, fallback_uniform, rows_mode,
               temperature, seed, counter) -> ForkStepArgs:
    if hidden.dim() != 2 or W_head.dim() != 2:
        raise ValueError("hidden and W_head must be 2-D")
    device = hidden.device
    if device.type != "cuda":
        raise ValueError("fork_step runs on the GPU; hidden is on %s" % device)
    M, d = hidden.shape
    V = W_head.shape[0]
    if M != B * L:
        raise ValueError("hidden has %d rows, expected B*L = %d" % (M, B * L))
    if hidden.dtype == torch.bfloat16:
        dt = FORK_BF16
    elif hidden.dtype == torch.float32:
        dt = FORK_F32
    else:
        raise TypeError("hidden must be bfloat16 or float32")
    a = ForkStepArgs()
    a.hidden = _check(hidden, "hidden", hidden.dtype, M * d, device)
    a.W_head = _check(W_head, "W_head", hidden.dtype, V * d, device)
    a.tokens = _check(tokens, "tokens", torch.int32, M, device)
    a.mask = _check(mask, "mask", torch.uint8, M, device)
    a.block_start = _check(block_start, "block_start", torch.int32, B, device)
    a.block_len = int(block_len)
    a.tau = float(tau)
    a.out_conf = _check(out_conf, "out_conf", torch.float32, M, device)
    a.out_entropy = _check(out_entropy, "out_entropy", torch.float32, M, device)
    a.out_logp = _check(out_logp, "out_logp", torch.float32, M, device)
    a.out_fallback = _check(out_fallback, "out_fallback", torch.int32, B, device)
    a.B, a.L, a.d, a.V, a.dtype = B, L, d, V, dt
    a.stream = _stream_handle(stream, device)
    a.out_lse = _opt(out_lse, "out_lse", torch.float32, M, device)
    a.out_argmax = _opt(out_argmax, "out_argmax", torch.int32, M, device)
    a.out_ncommit = _opt(out_ncommit, "out_ncommit", torch.int32, B, device)
    a.out_commit_pos = _opt(out_commit_pos, "out_commit_pos", torch.int32,
                            B * int(block_len), device)
    a.rule = int(rule)
    if workspace is not None:
        if workspace.device != device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on %s" % device)
        a.workspace = workspace.data_ptr()
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    if events is not None:
        a.ev_lmhead_begin, a.ev_lmhead_end = events
    a.fallback_uniform = _opt(fallback_uniform, "fallback_uniform", torch.float32, B, device)
    a.rows_mode = int(rows_mode)
    a.sample_temperature = float(temperature)
    a.sample_counter = int(counter) & 0xFFFFFFFF
    a.sample_seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return a


def _raise_on(rc: int) -> None:
    if rc != FORK_OK:
        raise ForkError(rc, lib().fork_last_error().decode())


def logprob(hidden: torch.Tensor, W_head: torch.Tensor, tokens: torch.Tensor,
            out_logp: torch.Tensor, *, rows: Optional[torch.Tensor] = None, out_q=None,
            out_entropy=None, out_lse=None, workspace=None, stream=None, events=None) -> None:
    """fork_logprob of the C ABI: log q(tokens[e]) at hidden row rows[e]
    (row e without ``rows``) under W_head."""
    if hidden.dim() != 2 or W_head.dim() != 2:
        raise ValueError("hidden and W_head must be 2-D")
    device = hidden.device
    if device.type != "cuda":
        raise ValueError("fork_logprob runs on the GPU; hidden is on %s" % device)
    M, d = hidden.shape
    V = W_head.shape[0]
    n = tokens.numel()
    if hidden.dtype == torch.bfloat16:
        dt = FORK_BF16
    elif hidden.dtype == torch.float32:
        dt = FORK_F32
    else:
        raise TypeError("hidden must be bfloat16 or float32")
    a = ForkLogprobArgs()
    a.hidden = _check(hidden, "hidden", hidden.dtype, M * d, device)
    a.W_head = _check(W_head, "W_head", hidden.dtype, V * d, device)
    a.rows = _opt(rows, "rows", torch.int32, n, device)
    a.tokens = _check(tokens, "tokens", torch.int32, n, device)
    a.out_logp = _check(out_logp, "out_logp", torch.float32, n, device)
    a.out_q = _opt(out_q, "out_q", torch.float32, n, device)
    a.out_entropy = _opt(out_entropy, "out_entropy", torch.float32, n, device)
    a.out_lse = _opt(out_lse, "out_lse", torch.float32, n, device)
    a.n, a.M, a.d, a.V, a.dtype = n, M, d, V, dt
    a.stream = _stream_handle(stream, device)
    if workspace is not None:
        a.workspace = workspace.data_ptr()
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    if events is not None:
        a.ev_lmhead_begin, a.ev_lmhead_end = events
    _raise_on(lib().fork_logprob(ctypes.byref(a)))


def grpo_objective(rewards: torch.Tensor, offsets: torch.Tensor, lp_new: torch.Tensor,
                   lp_old: torch.Tensor, G: int, eps: float, out_group_obj: torch.Tensor,
                   out_skipped: torch.Tensor, out_J: torch.Tensor, *, out_adv=None,
                   out_ratio=None, out_term=None, out_rollout_obj=None, stream=None) -> None:
    """fork_grpo_objective of the C ABI (rewards [n_groups*G], offsets
    [n_groups*G + 1], lp_new / lp_old [n])."""
    device = rewards.device
    if device.type != "cuda":
        raise ValueError("fork_grpo_objective runs on the GPU")
    R = rewards.numel()
    if R % G:
        raise ValueError("rewards must hold n_groups * G entries")
    ng = R // G
    n = lp_new.numel()
    a = ForkGrpoArgs()
    a.n_groups, a.G, a.n = ng, int(G), n
    a.rewards = _check(rewards, "rewards", torch.float32, R, device)
    a.offsets = _check(offsets, "offsets", torch.int32, R + 1, device)
    a.lp_new = _check(lp_new, "lp_new", torch.float32, n, device)
    a.lp_old = _check(lp_old, "lp_old", torch.float32, n, device)
    a.eps = float(eps)
    a.out_adv = _opt(out_adv, "out_adv", torch.float32, R, device)
    a.out_ratio = _opt(out_ratio, "out_ratio", torch.float32, n, device)
    a.out_term = _opt(out_term, "out_term", torch.float32, n, device)
    a.out_rollout_obj = _opt(out_rollout_obj, "out_rollout_obj", torch.float32, R, device)
    a.out_group_obj = _check(out_group_obj, "out_group_obj", torch.float32, ng, device)
    a.out_skipped = _check(out_skipped, "out_skipped", torch.uint8, ng, device)
    a.out_J = _check(out_J, "out_J", torch.float32, 1, device)
    a.stream = _stream_handle(stream, device)
    _raise_on(lib().fork_grpo_objective(ctypes.byref(a)))


def top_entropy(entropy: torch.Tensor, k: int, out_sel: torch.Tensor, stream=None) -> None:
    """fork_top_entropy of the C ABI on an [R, Lg] float32 tensor."""
    if entropy.dim() != 2:
        raise ValueError("entropy must be [R, Lg]")
    device = entropy.device
    if device.type != "cuda":
        raise ValueError("fork_top_entropy runs on the GPU")
    R, Lg = entropy.shape
    e = _check(entropy, "entropy", torch.float32, R * Lg, device)
    o = _check(out_sel, "out_sel", torch.uint8, R * Lg, device)
    _raise_on(lib().fork_top_entropy(e, R, Lg, int(k), o, _stream_handle(stream, device)))


def select(conf: torch.Tensor, argmax: torch.Tensor, tokens: torch.Tensor, mask: torch.Tensor,
           block_start: torch.Tensor, block_len: int, tau: float, out_fallback: torch.Tensor, *,
           B: int, L: int, rule: int = FORK_RULE_LEFTMOST, entropy=None, uniform=None,
           out_ncommit=None, out_commit_pos=None, stream=None,
           layout: int = FORK_LAYOUT_ROW_MAJOR) -> None:
    """fork_select of the C ABI: the unmasking rule alone, in place.  With
    FORK_LAYOUT_POSITION_MAJOR the per-position tensors hold position k of
    sequence b at k*B + b."""
    device = conf.device
    if device.type != "cuda":
        raise ValueError("fork_select runs on the GPU")
    M = B * L
    a = ForkSelectArgs()
    a.conf = _check(conf, "conf", torch.float32, M, device)
    a.entropy = _opt(entropy, "entropy", torch.float32, M, device)
    a.uniform = _opt(uniform, "uniform", torch.float32, B, device)
    a.argmax = _check(argmax, "argmax", torch.int32, M, device)
    a.tokens = _check(tokens, "tokens", torch.int32, M, device)
    a.mask = _check(mask, "mask", torch.uint8, M, device)
    a.block_start = _check(block_start, "block_start", torch.int32, B, device)
    a.out_fallback = _check(out_fallback, "out_fallback", torch.int32, B, device)
    a.out_ncommit = _opt(out_ncommit, "out_ncommit", torch.int32, B, device)
    a.out_commit_pos = _opt(out_commit_pos, "out_commit_pos", torch.int32, B * int(block_len),
                            device)
    a.B, a.L, a.block_len, a.tau, a.rule = B, L, int(block_len), float(tau), int(rule)
    a.layout = int(layout)
    a.stream = _stream_handle(stream, device)
    _raise_on(lib().fork_select(ctypes.byref(a)))


def logprob_workspace_bytes(n: int, V: int) -> int:
    return int(lib().fork_logprob_workspace_bytes(n, V))


def workspace_bytes(B: int, L: int, V: int) -> int:
    return int(lib().fork_workspace_bytes(B, L, V))


def release() -> None:
    lib().fork_release()


def version() -> int:
    return int(lib().fork_version())
