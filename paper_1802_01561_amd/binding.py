"""Torch-tensor front end of libvtrace: argument marshalling only.

Every step of the computation runs in the HIP kernels behind the C ABI; torch
only provides device memory and the current HIP stream.  Function names match
the C entry points in include/vtrace.h.
"""

from __future__ import annotations

import contextlib
import ctypes
from typing import NamedTuple, Optional

import torch

from ._lib import (BEHAVIOUR_INPUTS, CORRECTIONS, Q_ESTIMATES, REWARD_TRANSFORMS, VTRACE_BF16,
                   VTRACE_F32, Variant, check, lib)

__all__ = [
    "HeadLossGrad",
    "LossGrad",
    "Workspace",
    "vtrace_abi_version",
    "vtrace_error_flag",
    "vtrace_gather_logits",
    "vtrace_head_loss_grad",
    "vtrace_head_workspace_bytes",
    "vtrace_loss_grad",
    "vtrace_loss_grad_static",
    "vtrace_max_elements",
    "vtrace_targets",
    "vtrace_workspace_bytes",
]


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _allocating_on(stream):
    """Allocations made for a call on ``stream`` (workspace, outputs) are made
    with ``stream`` current, so that torch's caching allocator ties them to the
    stream the kernels use: a temporary workspace is then not handed out again
    before the call that uses it has run."""
    return contextlib.nullcontext() if stream is None else torch.cuda.stream(stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return VTRACE_F32
    if t.dtype == torch.bfloat16:
        return VTRACE_BF16
    raise TypeError(f"logits must be float32 or bfloat16, got {t.dtype}")


def _require(t: torch.Tensor, name: str, shape, dtype, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _inputs(target_logits, behaviour_logits, actions, rewards, discounts, values, bootstrap_value,
            behaviour="logits"):
    if target_logits.dim() != 3:
        raise ValueError("target_logits must be [T, B, A]")
    T, B, A = target_logits.shape
    dev = target_logits.device
    if dev.type != "cuda":
        raise ValueError("inputs must be on a GPU device")
    code = _dtype_code(target_logits)
    _require(target_logits, "target_logits", (T, B, A), None, dev)
    if behaviour == "log_probs":
        _require(behaviour_logits, "behaviour log-probabilities", (T, B), torch.float32, dev)
    else:
        _require(behaviour_logits, "behaviour_logits", (T, B, A), target_logits.dtype, dev)
    _require(actions, "actions", (T, B), torch.int32, dev)
    for name, t in (("rewards", rewards), ("discounts", discounts), ("values", values)):
        _require(t, name, (T, B), torch.float32, dev)
    _require(bootstrap_value, "bootstrap_value", (B,), torch.float32, dev)
    return T, B, A, code, dev


def _variant(correction="vtrace", q_estimate="vtrace", epsilon=1e-6, behaviour="logits",
             reward_transform=None, grad_dtype=torch.float32):
    """A vtrace_variant for the _ex entry points (Sec. 5.2.3, App. D, App. E.3)."""
    try:
        gd = {torch.float32: VTRACE_F32, torch.bfloat16: VTRACE_BF16}[grad_dtype]
        return Variant(CORRECTIONS[correction], Q_ESTIMATES[q_estimate], float(epsilon),
                       BEHAVIOUR_INPUTS[behaviour], REWARD_TRANSFORMS[reward_transform], gd)
    except KeyError as e:
        raise ValueError(f"unknown variant setting: {e}") from None


def vtrace_abi_version() -> int:
    return lib().vtrace_abi_version()


def vtrace_max_elements() -> int:
    return lib().vtrace_max_elements()


def vtrace_workspace_bytes(T: int, B: int, A: int) -> int:
    return lib().vtrace_workspace_bytes(T, B, A)


def vtrace_head_workspace_bytes(T: int, B: int, A: int, H: int) -> int:
    return lib().vtrace_head_workspace_bytes(T, B, A, H)


class Workspace:
    """Device workspace for vtrace_loss_grad (or, with H, for
    vtrace_head_loss_grad), cleared on creation."""

    def __init__(self, T: int, B: int, A: int, device=None, stream=None, *, H: Optional[int] = None):
        n = vtrace_workspace_bytes(T, B, A) if H is None else vtrace_head_workspace_bytes(T, B, A, H)
        if n == 0:
            raise ValueError(f"invalid batch shape T={T} B={B} A={A} H={H}")
        self.nbytes = n
        with _allocating_on(stream):
            self.tensor = torch.empty(n, dtype=torch.uint8, device=device or "cuda")
        check(lib().vtrace_workspace_init(_p(self.tensor), n, _stream(stream)))

    def fits(self, T: int, B: int, A: int, H: Optional[int] = None) -> bool:
        need = vtrace_workspace_bytes(T, B, A) if H is None else vtrace_head_workspace_bytes(T, B, A, H)
        return self.nbytes >= need


class LossGrad(NamedTuple):
    losses: torch.Tensor  # [4] total, policy gradient, baseline, entropy
    d_logits: torch.Tensor  # [T,B,A]
    d_values: torch.Tensor  # [T,B]
    vs: Optional[torch.Tensor]
    pg_advantages: Optional[torch.Tensor]
    lane_losses: Optional[torch.Tensor]


def vtrace_targets(target_logits, behaviour_logits, actions, rewards, discounts, values,
                   bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0, *, vs=None,
                   pg_advantages=None, workspace: Optional[Workspace] = None, stream=None,
                   correction="vtrace", q_estimate="vtrace", epsilon=1e-6, behaviour="logits",
                   reward_transform=None):
    """V-trace targets v_s and advantages; returns (vs, pg_advantages).

    ``correction`` ("vtrace", "none", "epsilon", "one_step_is") and
    ``q_estimate`` ("vtrace", "baseline") select the paper's variants;
    behaviour="log_probs" takes ``behaviour_logits`` as [T, B] float32
    log mu(a_t|x_t); ``reward_transform`` is None, "clip" or "asymmetric"."""
    variant = _variant(correction, q_estimate, epsilon, behaviour, reward_transform)
    T, B, A, code, dev = _inputs(target_logits, behaviour_logits, actions, rewards, discounts,
                                 values, bootstrap_value, behaviour)
    with _allocating_on(stream):
        if vs is None:
            vs = torch.empty((T, B), dtype=torch.float32, device=dev)
        if pg_advantages is None:
            pg_advantages = torch.empty((T, B), dtype=torch.float32, device=dev)
    _require(vs, "vs", (T, B), torch.float32, dev)
    _require(pg_advantages, "pg_advantages", (T, B), torch.float32, dev)
    ws, nws = (None, 0) if workspace is None else (_p(workspace.tensor), workspace.nbytes)
    check(lib().vtrace_targets_ex(
        T, B, A, code, _p(target_logits), _p(behaviour_logits), _p(actions), _p(rewards),
        _p(discounts), _p(values), _p(bootstrap_value), rho_bar, c_bar, lam,
        ctypes.byref(variant), _p(vs), _p(pg_advantages), ws, nws, _stream(stream)))
    return vs, pg_advantages


def vtrace_loss_grad(target_logits, behaviour_logits, actions, rewards, discounts, values,
                     bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0, baseline_cost=0.5,
                     entropy_cost=0.01, *, workspace: Optional[Workspace] = None,
                     with_vs=False, with_pg_advantages=False, with_lane_losses=False,
                     out: Optional[LossGrad] = None, stream=None, correction="vtrace",
                     q_estimate="vtrace", epsilon=1e-6, behaviour="logits",
                     reward_transform=None, grad_dtype=torch.float32) -> LossGrad:
    """Fused V-trace targets, losses and gradients w.r.t. logits and values.

    ``out`` may hold preallocated output tensors (fields left None are skipped
    when optional, allocated when required).  The variant arguments are as in
    vtrace_targets; ``grad_dtype`` (float32 or bfloat16) is d_logits' type."""
    variant = _variant(correction, q_estimate, epsilon, behaviour, reward_transform, grad_dtype)
    T, B, A, code, dev = _inputs(target_logits, behaviour_logits, actions, rewards, discounts,
                                 values, bootstrap_value, behaviour)
    if workspace is None:
        workspace = Workspace(T, B, A, device=dev, stream=stream)
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        with _allocating_on(stream):
            out = LossGrad(
                torch.empty(4, **f32), torch.empty((T, B, A), dtype=grad_dtype, device=dev),
                torch.empty((T, B), **f32),
                torch.empty((T, B), **f32) if with_vs else None,
                torch.empty((T, B), **f32) if with_pg_advantages else None,
                torch.empty((B, 3), **f32) if with_lane_losses else None)
    _require(out.losses, "losses", (4,), torch.float32, dev)
    _require(out.d_logits, "d_logits", (T, B, A), grad_dtype, dev)
    _require(out.d_values, "d_values", (T, B), torch.float32, dev)
    if out.vs is not None:
        _require(out.vs, "vs", (T, B), torch.float32, dev)
    if out.pg_advantages is not None:
        _require(out.pg_advantages, "pg_advantages", (T, B), torch.float32, dev)
    if out.lane_losses is not None:
        _require(out.lane_losses, "lane_losses", (B, 3), torch.float32, dev)
    check(lib().vtrace_loss_grad_ex(
        T, B, A, code, _p(target_logits), _p(behaviour_logits), _p(actions), _p(rewards),
        _p(discounts), _p(values), _p(bootstrap_value), rho_bar, c_bar, lam,
        baseline_cost, entropy_cost, ctypes.byref(variant), _p(out.losses), _p(out.d_logits),
        _p(out.d_values),
        _p(out.vs), _p(out.pg_advantages), _p(out.lane_losses),
        _p(workspace.tensor), workspace.nbytes, _stream(stream)))
    return out


def vtrace_loss_grad_static(target_logits, behaviour_logits, actions, rewards, discounts, values,
                            bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0, baseline_cost=0.5,
                            entropy_cost=0.01, *, with_vs=False, with_pg_advantages=False,
                            with_lane_losses=False, out: Optional[LossGrad] = None, stream=None,
                            correction="vtrace", q_estimate="vtrace", epsilon=1e-6,
                            behaviour="logits", reward_transform=None,
                            grad_dtype=torch.float32) -> LossGrad:
    """vtrace_loss_grad without a workspace: the library keeps the loss partials
    in a fixed device array (B <= VTRACE_STATIC_MAX_LANES).  The C call
    allocates nothing; pass ``out`` to allocate nothing here either.  Calls
    that overlap on one device race on that array."""
    variant = _variant(correction, q_estimate, epsilon, behaviour, reward_transform, grad_dtype)
    T, B, A, code, dev = _inputs(target_logits, behaviour_logits, actions, rewards, discounts,
                                 values, bootstrap_value, behaviour)
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        with _allocating_on(stream):
            out = LossGrad(
                torch.empty(4, **f32), torch.empty((T, B, A), dtype=grad_dtype, device=dev),
                torch.empty((T, B), **f32),
                torch.empty((T, B), **f32) if with_vs else None,
                torch.empty((T, B), **f32) if with_pg_advantages else None,
                torch.empty((B, 3), **f32) if with_lane_losses else None)
    _require(out.losses, "losses", (4,), torch.float32, dev)
    _require(out.d_logits, "d_logits", (T, B, A), grad_dtype, dev)
    _require(out.d_values, "d_values", (T, B), torch.float32, dev)
    for name, t, shape in (("vs", out.vs, (T, B)), ("pg_advantages", out.pg_advantages, (T, B)),
                           ("lane_losses", out.lane_losses, (B, 3))):
        if t is not None:
            _require(t, name, shape, torch.float32, dev)
    check(lib().vtrace_loss_grad_static(
        T, B, A, code, _p(target_logits), _p(behaviour_logits), _p(actions), _p(rewards),
        _p(discounts), _p(values), _p(bootstrap_value), rho_bar, c_bar, lam,
        baseline_cost, entropy_cost, ctypes.byref(variant), _p(out.losses), _p(out.d_logits),
        _p(out.d_values), _p(out.vs), _p(out.pg_advantages), _p(out.lane_losses), _stream(stream)))
    return out


class HeadLossGrad(NamedTuple):
    losses: torch.Tensor  # [4] total, policy gradient, baseline, entropy
    d_hidden: torch.Tensor  # [T,B,H]
    d_weight: torch.Tensor  # [H,A+1]
    d_bias: torch.Tensor  # [A+1]
    vs: Optional[torch.Tensor]
    pg_advantages: Optional[torch.Tensor]
    lane_losses: Optional[torch.Tensor]
    outputs: Optional[torch.Tensor]  # [T,B,A+1] the layer's outputs


def vtrace_head_loss_grad(hidden, head_weight, head_bias, behaviour_logits, actions, rewards,
                          discounts, bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0,
                          baseline_cost=0.5, entropy_cost=0.01, *,
                          workspace: Optional[Workspace] = None, with_vs=False,
                          with_pg_advantages=False, with_lane_losses=False, with_outputs=False,
                          out: Optional[HeadLossGrad] = None, stream=None, correction="vtrace",
                          q_estimate="vtrace", epsilon=1e-6, behaviour="logits",
                          reward_transform=None, grad_dtype=torch.float32) -> HeadLossGrad:
    """Output layer o = hidden @ head_weight + head_bias (policy logits, then the
    baseline), the V-trace losses on it and the gradients through the layer.

    hidden [T,B,H] and head_weight [H,A+1] are bfloat16; the variant arguments
    are as in vtrace_loss_grad; ``grad_dtype`` is d_hidden's type."""
    variant = _variant(correction, q_estimate, epsilon, behaviour, reward_transform, grad_dtype)
    if hidden.dim() != 3 or head_weight.dim() != 2:
        raise ValueError("hidden must be [T, B, H] and head_weight [H, A + 1]")
    T, B, H = hidden.shape
    A = head_weight.shape[1] - 1
    dev = hidden.device
    if dev.type != "cuda":
        raise ValueError("inputs must be on a GPU device")
    _require(hidden, "hidden", (T, B, H), torch.bfloat16, dev)
    _require(head_weight, "head_weight", (H, A + 1), torch.bfloat16, dev)
    _require(head_bias, "head_bias", (A + 1,), torch.float32, dev)
    if behaviour == "log_probs":
        _require(behaviour_logits, "behaviour log-probabilities", (T, B), torch.float32, dev)
        code = VTRACE_F32
    else:
        _require(behaviour_logits, "behaviour_logits", (T, B, A), None, dev)
        code = _dtype_code(behaviour_logits)
    _require(actions, "actions", (T, B), torch.int32, dev)
    for name, t in (("rewards", rewards), ("discounts", discounts)):
        _require(t, name, (T, B), torch.float32, dev)
    _require(bootstrap_value, "bootstrap_value", (B,), torch.float32, dev)
    if workspace is None:
        workspace = Workspace(T, B, A, device=dev, stream=stream, H=H)
    if out is None:
        f32 = dict(dtype=torch.float32, device=dev)
        with _allocating_on(stream):
            out = HeadLossGrad(
                torch.empty(4, **f32), torch.empty((T, B, H), dtype=grad_dtype, device=dev),
                torch.empty((H, A + 1), **f32), torch.empty(A + 1, **f32),
                torch.empty((T, B), **f32) if with_vs else None,
                torch.empty((T, B), **f32) if with_pg_advantages else None,
                torch.empty((B, 3), **f32) if with_lane_losses else None,
                torch.empty((T, B, A + 1), **f32) if with_outputs else None)
    _require(out.losses, "losses", (4,), torch.float32, dev)
    _require(out.d_hidden, "d_hidden", (T, B, H), grad_dtype, dev)
    _require(out.d_weight, "d_weight", (H, A + 1), torch.float32, dev)
    _require(out.d_bias, "d_bias", (A + 1,), torch.float32, dev)
    for name, t, shape in (("vs", out.vs, (T, B)), ("pg_advantages", out.pg_advantages, (T, B)),
                           ("lane_losses", out.lane_losses, (B, 3)),
                           ("outputs", out.outputs, (T, B, A + 1))):
        if t is not None:
            _require(t, name, shape, torch.float32, dev)
    check(lib().vtrace_head_loss_grad(
        T, B, A, H, code, _p(hidden), _p(head_weight), _p(head_bias), _p(behaviour_logits),
        _p(actions), _p(rewards), _p(discounts), _p(bootstrap_value), rho_bar, c_bar, lam,
        baseline_cost, entropy_cost, ctypes.byref(variant), _p(out.losses), _p(out.d_hidden),
        _p(out.d_weight), _p(out.d_bias), _p(out.vs), _p(out.pg_advantages), _p(out.lane_losses),
        _p(out.outputs), _p(workspace.tensor), workspace.nbytes, _stream(stream)))
    return out


def vtrace_gather_logits(target_logits, behaviour_logits, actions, *, gathered=None, stream=None):
    """[T,B,2] bit copies of the target and behaviour logits at the taken actions."""
    if target_logits.dim() != 3:
        raise ValueError("target_logits must be [T, B, A]")
    T, B, A = target_logits.shape
    dev = target_logits.device
    code = _dtype_code(target_logits)
    _require(behaviour_logits, "behaviour_logits", (T, B, A), target_logits.dtype, dev)
    _require(actions, "actions", (T, B), torch.int32, dev)
    if gathered is None:
        with _allocating_on(stream):
            gathered = torch.empty((T, B, 2), dtype=target_logits.dtype, device=dev)
    _require(gathered, "gathered", (T, B, 2), target_logits.dtype, dev)
    check(lib().vtrace_gather_logits(T, B, A, code, _p(target_logits), _p(behaviour_logits),
                                     _p(actions), _p(gathered), _stream(stream)))
    return gathered


def vtrace_error_flag(workspace: Workspace, stream=None) -> int:
    """Synchronises the stream and returns the sticky out-of-range-action flag."""
    flag = ctypes.c_int32(0)
    check(lib().vtrace_error_flag(_p(workspace.tensor), ctypes.byref(flag), _stream(stream)))
    return int(flag.value)
