"""ctypes binding of libsao (include/sao.h).

Argument marshalling only: every step of the pass runs in the library's HIP
kernels. torch supplies device memory (outputs and workspace) and the current
stream. There is no CPU fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsao.so")

SAO_BF16, SAO_F32 = 0, 1
(OP_LOGPROB, OP_ADVANTAGE, OP_LOSS, OP_BACKWARD, OP_VALUE, OP_PPO_LOSS, OP_EXPLAINED_VARIANCE,
 OP_STEP_ADVANTAGE, OP_GROUP_ADVANTAGE, OP_RUNNING_MEAN_ADVANTAGE) = range(10)
STEP_AVERAGE, STEP_LAST = 0, 1
STATUS_TARGET_RANGE, STATUS_SEGMENTS, STATUS_NONFINITE, STATUS_KEY_RANGE = 1, 2, 4, 8
FLAG_MASKED, FLAG_USED, FLAG_LOW, FLAG_HIGH, FLAG_NONFINITE = 0, 1, 2, 3, 4

EXPORTS = ("sao_status_string", "sao_last_error_message", "sao_version", "sao_workspace_size",
           "sao_token_logprob", "sao_advantage", "sao_clipped_loss", "sao_loss_backward",
           "sao_value_forward", "sao_value_loss", "sao_ppo_loss", "sao_explained_variance", "sao_step_advantage",
           "sao_group_advantage", "sao_running_mean_advantage", "sao_clipped_loss_noalloc",
           "sao_debug_time_kernel", "sao_debug_clock_samples")
KERNEL_NONE, KERNEL_HEAD_FORWARD, KERNEL_BACKWARD_DZ, KERNEL_BACKWARD_DH, KERNEL_BACKWARD_DW = 0, 1, 2, 3, 4


class SaoError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{message} (status {code})")
        self.code = code


_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_SIGS = {
    "sao_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "sao_last_error_message": (ctypes.c_char_p, []),
    "sao_version": (ctypes.c_char_p, []),
    "sao_workspace_size": (ctypes.c_size_t, [ctypes.c_int, _i64, _i64, _i64, ctypes.c_int]),
    "sao_token_logprob": (ctypes.c_int, [_p, _i64, _p, _i64, _p, _p, _i64, _i64, _i64, ctypes.c_int,
                                         _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "sao_advantage": (ctypes.c_int, [_p, _p, _p, _p, ctypes.c_int32, _i64, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_double, _p, _p, _p, _p, _p,
                                     ctypes.c_size_t, _p]),
    "sao_clipped_loss": (ctypes.c_int, [_p, _p, _p, _p, _i64, ctypes.c_float, ctypes.c_float, _p, _p,
                                        _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "sao_clipped_loss_noalloc": (ctypes.c_int, [_p, _p, _p, _p, _i64, ctypes.c_float, ctypes.c_float, _p, _p,
                                                _p, _p, _p, _p]),
    "sao_loss_backward": (ctypes.c_int, [_p, _i64, _p, _i64, _p, _p, _p, _i64, _i64, _i64,
                                         ctypes.c_int, _p, _p, _p, ctypes.c_size_t, _p]),
    "sao_value_forward": (ctypes.c_int, [_p, _i64, _p, _i64, _i64, ctypes.c_int, _p, _p, ctypes.c_size_t, _p]),
    "sao_value_loss": (ctypes.c_int, [_p, _i64, _p, _p, _p, _p, _i64, _i64, _p, ctypes.c_int, _p, _p, _p, _p,
                                      ctypes.c_size_t, _p]),
    "sao_ppo_loss": (ctypes.c_int, [_p, _p, _p, _p, _p, _i64, ctypes.c_float, ctypes.c_float, _p, _p, _p, _p,
                                    _p, _p, ctypes.c_size_t, _p]),
    "sao_explained_variance": (ctypes.c_int, [_p, _p, _p, _i64, _p, _p, _p, ctypes.c_size_t, _p]),
    "sao_step_advantage": (ctypes.c_int, [_p, _p, _p, _p, ctypes.c_int32, _i64, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_double, ctypes.c_int, _p, _p, _p, _p, _p, _p, ctypes.c_size_t,
                                          _p]),
    "sao_group_advantage": (ctypes.c_int, [_p, _p, _p, ctypes.c_int32, _i64, ctypes.c_int32, ctypes.c_double, _p, _p,
                                           _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "sao_running_mean_advantage": (ctypes.c_int, [_p, _p, _p, ctypes.c_int32, _i64, _p, ctypes.c_int32,
                                                  ctypes.c_int32, _p, _p, _p, _p, _p, _p, _p, _p, ctypes.c_size_t,
                                                  _p]),
    "sao_debug_time_kernel": (None, [ctypes.c_int, _p, _p]),
    "sao_debug_clock_samples": (None, [ctypes.c_int, _p, _i64]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libsao.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_07508_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(code: int) -> None:
    if code != 0:
        raise SaoError(code, lib().sao_last_error_message().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SAO_BF16
    if t.dtype == torch.float32:
        return SAO_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _rows(t: torch.Tensor, name: str) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a row-major 2-D tensor with unit column stride")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    return t.stride(0)


def _vec(t: Optional[torch.Tensor], name: str, dtype: torch.dtype, n: int, device: torch.device,
         optional: bool = False) -> None:
    """A per-token array: on `device`, of `dtype`, contiguous, at least n elements."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, not {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, not {t.dtype}")
    if not t.is_contiguous() or t.numel() < n:
        raise ValueError(f"{name} must be contiguous with at least {n} elements")


def workspace_size(op: int, T: int, H: int, V: int, dtype: int) -> int:
    return int(lib().sao_workspace_size(op, T, H, V, dtype))


def _workspace(nbytes: int, device) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _head_shapes(hidden: torch.Tensor, w_head: torch.Tensor) -> None:
    if hidden.dim() != 2 or w_head.dim() != 2 or w_head.shape[1] != hidden.shape[1]:
        raise ValueError("hidden [T, H] and w_head [V, H] must share H")
    if w_head.device != hidden.device:
        raise ValueError("hidden and w_head must be on the same device")


def token_logprob(hidden: torch.Tensor, w_head: torch.Tensor, target: torch.Tensor,
                  mask: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
                  out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None):
    """Per-token (logp, lse) of the LM head; rows with mask 0 get 0."""
    T, H = hidden.shape
    V = w_head.shape[0]
    dt = _dtype_code(hidden)
    if _dtype_code(w_head) != dt:
        raise TypeError("hidden and w_head must share a dtype")
    dev = hidden.device
    _head_shapes(hidden, w_head)
    _vec(target, "target", torch.int32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev, optional=True)
    _vec(status, "status", torch.int32, 1, dev, optional=True)
    logp, lse = out if out is not None else (torch.empty(T, dtype=torch.float32, device=dev),
                                             torch.empty(T, dtype=torch.float32, device=dev))
    _vec(logp, "logp", torch.float32, T, dev)
    _vec(lse, "lse", torch.float32, T, dev)
    ws = _workspace(workspace_size(OP_LOGPROB, T, H, V, dt), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_token_logprob(
            _ptr(hidden), _rows(hidden, "hidden"), _ptr(w_head), _rows(w_head, "w_head"), _ptr(target),
            _ptr(mask), T, H, V, dt, _ptr(logp), _ptr(lse), _ptr(status), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return logp, lse


def advantage(values: torch.Tensor, rewards: torch.Tensor, mask: torch.Tensor, cu_seqlens: torch.Tensor,
              gamma: float = 1.0, lam: float = 1.0, alpha: float = 0.0,
              status: Optional[torch.Tensor] = None, want_count: bool = True):
    """Skip-observation GAE: (adv, ret, n_tokens) with n_tokens a device int64 scalar."""
    T = values.shape[0]
    B = cu_seqlens.shape[0] - 1
    dev = values.device
    _vec(values, "values", torch.float32, T, dev)
    _vec(rewards, "rewards", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(cu_seqlens, "cu_seqlens", torch.int32, B + 1, dev)
    _vec(status, "status", torch.int32, 1, dev, optional=True)
    adv = torch.empty(T, dtype=torch.float32, device=dev)
    ret = torch.empty(T, dtype=torch.float32, device=dev)
    n_tok = torch.zeros(1, dtype=torch.int64, device=dev) if want_count else None
    ws = _workspace(workspace_size(OP_ADVANTAGE, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_advantage(
            _ptr(values), _ptr(rewards), _ptr(mask), _ptr(cu_seqlens), B, T, float(gamma), float(lam),
            float(alpha), _ptr(adv), _ptr(ret), _ptr(n_tok), _ptr(status), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return adv, ret, n_tok


def step_advantage(values: torch.Tensor, rewards: torch.Tensor, mask: torch.Tensor, cu_seqlens: torch.Tensor,
                   gamma: float = 1.0, lam: float = 1.0, alpha: float = 0.0, step_value: str = "average",
                   status: Optional[torch.Tensor] = None, want_last: bool = True, want_count: bool = True):
    """Step-level GAE: (adv, ret, last or None, n_tokens or None); step_value "average" or "last"."""
    T = values.shape[0]
    B = cu_seqlens.shape[0] - 1
    dev = values.device
    form = {"average": STEP_AVERAGE, "last": STEP_LAST}.get(step_value)
    if form is None:
        raise ValueError(f"step_value must be 'average' or 'last', not {step_value!r}")
    _vec(values, "values", torch.float32, T, dev)
    _vec(rewards, "rewards", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(cu_seqlens, "cu_seqlens", torch.int32, B + 1, dev)
    _vec(status, "status", torch.int32, 1, dev, optional=True)
    adv = torch.empty(T, dtype=torch.float32, device=dev)
    ret = torch.empty(T, dtype=torch.float32, device=dev)
    last = torch.empty(T, dtype=torch.uint8, device=dev) if want_last else None
    n_tok = torch.zeros(1, dtype=torch.int64, device=dev) if want_count else None
    ws = _workspace(workspace_size(OP_STEP_ADVANTAGE, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_step_advantage(
            _ptr(values), _ptr(rewards), _ptr(mask), _ptr(cu_seqlens), B, T, float(gamma), float(lam),
            float(alpha), form, _ptr(adv), _ptr(ret), _ptr(last), _ptr(n_tok), _ptr(status), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return adv, ret, last, n_tok


def _segment_inputs(rewards, mask, cu_seqlens, status):
    T = rewards.shape[0]
    B = cu_seqlens.shape[0] - 1
    dev = rewards.device
    _vec(rewards, "rewards", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(cu_seqlens, "cu_seqlens", torch.int32, B + 1, dev)
    _vec(status, "status", torch.int32, 1, dev, optional=True)
    return T, B, dev


def group_advantage(rewards: torch.Tensor, mask: torch.Tensor, cu_seqlens: torch.Tensor, group_size: int,
                    eps_stab: float, status: Optional[torch.Tensor] = None, want_count: bool = True):
    """GRPO advantage: (adv [T] f32, traj_adv [B] f64, traj_reward [B] f64, n_tokens or None)."""
    T, B, dev = _segment_inputs(rewards, mask, cu_seqlens, status)
    adv = torch.empty(T, dtype=torch.float32, device=dev)
    traj_reward = torch.empty(B, dtype=torch.float64, device=dev)
    traj_adv = torch.empty(B, dtype=torch.float64, device=dev)
    n_tok = torch.zeros(1, dtype=torch.int64, device=dev) if want_count else None
    ws = _workspace(workspace_size(OP_GROUP_ADVANTAGE, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_group_advantage(
            _ptr(rewards), _ptr(mask), _ptr(cu_seqlens), B, T, int(group_size), float(eps_stab), _ptr(adv),
            _ptr(traj_reward), _ptr(traj_adv), _ptr(n_tok), _ptr(status), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return adv, traj_adv, traj_reward, n_tok


def running_mean_state(n_keys: int, window: int, device) -> Tuple[torch.Tensor, torch.Tensor]:
    """Zeroed (history [n_keys, window] f64, seen [n_keys] i64) for running_mean_advantage."""
    return (torch.zeros((n_keys, window), dtype=torch.float64, device=device),
            torch.zeros(n_keys, dtype=torch.int64, device=device))


def running_mean_advantage(rewards: torch.Tensor, mask: torch.Tensor, cu_seqlens: torch.Tensor,
                           history: torch.Tensor, seen: torch.Tensor, keys: Optional[torch.Tensor] = None,
                           status: Optional[torch.Tensor] = None, want_count: bool = True):
    """Running-mean baseline over a window of history.shape[1] rewards per key; updates
    (history, seen) in place. Returns (adv [T] f32, traj_adv [B] f64, traj_reward [B] f64, n_tokens)."""
    T, B, dev = _segment_inputs(rewards, mask, cu_seqlens, status)
    if history.dim() != 2:
        raise ValueError("history must be [n_keys, window]")
    n_keys, window = history.shape
    _vec(history, "history", torch.float64, n_keys * window, dev)
    _vec(seen, "seen", torch.int64, n_keys, dev)
    _vec(keys, "keys", torch.int32, B, dev, optional=True)
    adv = torch.empty(T, dtype=torch.float32, device=dev)
    traj_reward = torch.empty(B, dtype=torch.float64, device=dev)
    traj_adv = torch.empty(B, dtype=torch.float64, device=dev)
    n_tok = torch.zeros(1, dtype=torch.int64, device=dev) if want_count else None
    ws = _workspace(workspace_size(OP_RUNNING_MEAN_ADVANTAGE, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_running_mean_advantage(
            _ptr(rewards), _ptr(mask), _ptr(cu_seqlens), B, T, _ptr(keys), n_keys, window, _ptr(history),
            _ptr(seen), _ptr(adv), _ptr(traj_reward), _ptr(traj_adv), _ptr(n_tok), _ptr(status), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return adv, traj_adv, traj_reward, n_tok


def clipped_loss(logp: torch.Tensor, logp_rollout: torch.Tensor, adv: torch.Tensor, mask: torch.Tensor,
                 eps_low: float, eps_high: float, n_tokens: Optional[torch.Tensor] = None,
                 loss: Optional[torch.Tensor] = None, counts: Optional[torch.Tensor] = None):
    """DIS loss: (loss[2] f64 +=, g, flags, counts[5] i64 +=). Zeroed accumulators are made if not given."""
    T = logp.shape[0]
    dev = logp.device
    _vec(logp, "logp", torch.float32, T, dev)
    _vec(logp_rollout, "logp_rollout", torch.float32, T, dev)
    _vec(adv, "adv", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(n_tokens, "n_tokens", torch.int64, 1, dev, optional=True)
    if loss is None:
        loss = torch.zeros(2, dtype=torch.float64, device=dev)
    if counts is None:
        counts = torch.zeros(5, dtype=torch.int64, device=dev)
    _vec(loss, "loss", torch.float64, 2, dev)
    _vec(counts, "counts", torch.int64, 5, dev)
    g = torch.empty(T, dtype=torch.float32, device=dev)
    flags = torch.empty(T, dtype=torch.uint8, device=dev)
    ws = _workspace(workspace_size(OP_LOSS, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_clipped_loss(
            _ptr(logp), _ptr(logp_rollout), _ptr(adv), _ptr(mask), T, float(eps_low), float(eps_high),
            _ptr(n_tokens), _ptr(loss), _ptr(g), _ptr(flags), _ptr(counts), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return loss, g, flags, counts


def clipped_loss_noalloc(logp: torch.Tensor, logp_rollout: torch.Tensor, adv: torch.Tensor, mask: torch.Tensor,
                         eps_low: float, eps_high: float, n_tokens: Optional[torch.Tensor] = None,
                         loss: Optional[torch.Tensor] = None, counts: Optional[torch.Tensor] = None):
    """clipped_loss through sao_clipped_loss_noalloc: the library's static per-device
    scratch instead of a workspace. Same results; calls that overlap on one GPU race."""
    T = logp.shape[0]
    dev = logp.device
    _vec(logp, "logp", torch.float32, T, dev)
    _vec(logp_rollout, "logp_rollout", torch.float32, T, dev)
    _vec(adv, "adv", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(n_tokens, "n_tokens", torch.int64, 1, dev, optional=True)
    if loss is None:
        loss = torch.zeros(2, dtype=torch.float64, device=dev)
    if counts is None:
        counts = torch.zeros(5, dtype=torch.int64, device=dev)
    _vec(loss, "loss", torch.float64, 2, dev)
    _vec(counts, "counts", torch.int64, 5, dev)
    g = torch.empty(T, dtype=torch.float32, device=dev)
    flags = torch.empty(T, dtype=torch.uint8, device=dev)
    if T:
        _check(lib().sao_clipped_loss_noalloc(
            _ptr(logp), _ptr(logp_rollout), _ptr(adv), _ptr(mask), T, float(eps_low), float(eps_high),
            _ptr(n_tokens), _ptr(loss), _ptr(g), _ptr(flags), _ptr(counts), _stream(dev)))
    return loss, g, flags, counts


def ppo_loss(logp: torch.Tensor, logp_old: torch.Tensor, adv: torch.Tensor, mask: torch.Tensor,
             eps_low: float, eps_high: float, n_tokens: Optional[torch.Tensor] = None,
             logp_behav: Optional[torch.Tensor] = None, loss: Optional[torch.Tensor] = None,
             counts: Optional[torch.Tensor] = None):
    """Clipped surrogate (standard, clip-higher, or decoupled with logp_behav):
    (loss[1] f64 +=, g, flags, counts[5] i64 +=). Zeroed accumulators are made if not given."""
    T = logp.shape[0]
    dev = logp.device
    _vec(logp, "logp", torch.float32, T, dev)
    _vec(logp_old, "logp_old", torch.float32, T, dev)
    _vec(logp_behav, "logp_behav", torch.float32, T, dev, optional=True)
    _vec(adv, "adv", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(n_tokens, "n_tokens", torch.int64, 1, dev, optional=True)
    if loss is None:
        loss = torch.zeros(1, dtype=torch.float64, device=dev)
    if counts is None:
        counts = torch.zeros(5, dtype=torch.int64, device=dev)
    _vec(loss, "loss", torch.float64, 1, dev)
    _vec(counts, "counts", torch.int64, 5, dev)
    g = torch.empty(T, dtype=torch.float32, device=dev)
    flags = torch.empty(T, dtype=torch.uint8, device=dev)
    ws = _workspace(workspace_size(OP_PPO_LOSS, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_ppo_loss(
            _ptr(logp), _ptr(logp_old), _ptr(logp_behav), _ptr(adv), _ptr(mask), T, float(eps_low), float(eps_high),
            _ptr(n_tokens), _ptr(loss), _ptr(g), _ptr(flags), _ptr(counts), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return loss, g, flags, counts


def explained_variance(values: torch.Tensor, ret: torch.Tensor, mask: torch.Tensor,
                       moments: Optional[torch.Tensor] = None):
    """(ev [1] f64, moments [5] f64): EV = 1 - Var(R - V) / Var(R) over mask tokens, with this
    call's tokens combined into `moments` (zeroed if not given) so chunked calls cover a batch."""
    T = values.shape[0]
    dev = values.device
    _vec(values, "values", torch.float32, T, dev)
    _vec(ret, "ret", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    if moments is None:
        moments = torch.zeros(5, dtype=torch.float64, device=dev)
    _vec(moments, "moments", torch.float64, 5, dev)
    ev = torch.full((1,), float("nan"), dtype=torch.float64, device=dev)
    ws = _workspace(workspace_size(OP_EXPLAINED_VARIANCE, T, 1, 1, SAO_F32), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_explained_variance(
            _ptr(values), _ptr(ret), _ptr(mask), T, _ptr(moments), _ptr(ev), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return ev, moments


def loss_backward(hidden: torch.Tensor, w_head: torch.Tensor, target: torch.Tensor, lse: torch.Tensor,
                  g: torch.Tensor, dw_head: Optional[torch.Tensor] = None,
                  dhidden: Optional[torch.Tensor] = None):
    """(dhidden [T,H] in hidden's dtype, dw_head [V,H] f32 +=; zeroed if not given)."""
    T, H = hidden.shape
    V = w_head.shape[0]
    dt = _dtype_code(hidden)
    if _dtype_code(w_head) != dt:
        raise TypeError("hidden and w_head must share a dtype")
    dev = hidden.device
    _head_shapes(hidden, w_head)
    _vec(target, "target", torch.int32, T, dev)
    _vec(lse, "lse", torch.float32, T, dev)
    _vec(g, "g", torch.float32, T, dev)
    if dhidden is None:
        dhidden = torch.empty((T, H), dtype=hidden.dtype, device=dev)
    if dw_head is None:
        dw_head = torch.zeros((V, H), dtype=torch.float32, device=dev)
    _vec(dhidden, "dhidden", hidden.dtype, T * H, dev)
    _vec(dw_head, "dw_head", torch.float32, V * H, dev)
    ws = _workspace(workspace_size(OP_BACKWARD, T, H, V, dt), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_loss_backward(
            _ptr(hidden), _rows(hidden, "hidden"), _ptr(w_head), _rows(w_head, "w_head"), _ptr(target),
            _ptr(lse), _ptr(g), T, H, V, dt, _ptr(dhidden), _ptr(dw_head), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return dhidden, dw_head


def value_forward(hidden: torch.Tensor, w_value: torch.Tensor, v: Optional[torch.Tensor] = None) -> torch.Tensor:
    """v [T] f32 = hidden . w_value (bias-free critic head)."""
    T, H = hidden.shape
    dev = hidden.device
    _vec(w_value, "w_value", hidden.dtype, H, dev)
    if v is None:
        v = torch.empty(T, dtype=torch.float32, device=dev)
    _vec(v, "v", torch.float32, T, dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_value_forward(_ptr(hidden), _rows(hidden, "hidden"), _ptr(w_value), T, H,
                                       _dtype_code(hidden), _ptr(v), None, 0, _stream(dev)))
    return v


def value_loss(hidden: torch.Tensor, w_value: torch.Tensor, v: torch.Tensor, ret: torch.Tensor,
               mask: torch.Tensor, n_tokens: Optional[torch.Tensor] = None,
               loss: Optional[torch.Tensor] = None, dw_value: Optional[torch.Tensor] = None,
               dhidden: Optional[torch.Tensor] = None):
    """(loss_v [1] f64 +=, dhidden_v [T,H] in hidden's dtype, dw_value [H] f32 +=)."""
    T, H = hidden.shape
    dt = _dtype_code(hidden)
    dev = hidden.device
    _vec(w_value, "w_value", hidden.dtype, H, dev)
    _vec(v, "v", torch.float32, T, dev)
    _vec(ret, "ret", torch.float32, T, dev)
    _vec(mask, "mask", torch.uint8, T, dev)
    _vec(n_tokens, "n_tokens", torch.int64, 1, dev, optional=True)
    if loss is None:
        loss = torch.zeros(1, dtype=torch.float64, device=dev)
    if dw_value is None:
        dw_value = torch.zeros(H, dtype=torch.float32, device=dev)
    if dhidden is None:
        dhidden = torch.empty((T, H), dtype=hidden.dtype, device=dev)
    _vec(loss, "loss", torch.float64, 1, dev)
    _vec(dw_value, "dw_value", torch.float32, H, dev)
    _vec(dhidden, "dhidden", hidden.dtype, T * H, dev)
    ws = _workspace(workspace_size(OP_VALUE, T, H, 1, dt), dev)
    if T:  # T == 0 is a no-op: empty tensors carry null pointers
        _check(lib().sao_value_loss(
            _ptr(hidden), _rows(hidden, "hidden"), _ptr(w_value), _ptr(v), _ptr(ret), _ptr(mask), T, H,
            _ptr(n_tokens), dt, _ptr(loss), _ptr(dhidden), _ptr(dw_value), _ptr(ws),
            0 if ws is None else ws.numel(), _stream(dev)))
    return loss, dhidden, dw_value


def time_kernel(kernel: int, start: Optional[torch.cuda.Event], stop: Optional[torch.cuda.Event]) -> None:
    """Bracket the next launches of `kernel` with two timing events (None disables)."""
    if start is None or stop is None:
        lib().sao_debug_time_kernel(KERNEL_NONE, None, None)
        return
    lib().sao_debug_time_kernel(kernel, start.cuda_event, stop.cuda_event)


CLOCK_RECORD = ("hw_id", "wall_start", "wall_end", "clk_start", "clk_prologue", "clk_loop", "clk_end", "tile")


def clock_samples(records: Optional[torch.Tensor], kernel: int = KERNEL_HEAD_FORWARD) -> None:
    """Make the next launches of `kernel` (KERNEL_*; the backward ones on their
    first vocabulary block) record each workgroup's timeline (fields CLOCK_RECORD)
    into `records` (int64 [slots, 8] on the device); None disables."""
    if records is None:
        lib().sao_debug_clock_samples(KERNEL_NONE, None, 0)
        return
    if records.dtype != torch.int64 or records.dim() != 2 or records.shape[1] != 8 or not records.is_contiguous():
        raise ValueError("records must be a contiguous int64 [slots, 8] tensor")
    lib().sao_debug_clock_samples(kernel, records.data_ptr(), records.shape[0])
