"""MI355X (gfx950) library for the multi-step GRPO token loss of AsyncWebRL.

Thin torch-facing binding of libgrpo's C ABI (include/grpo.h): every function
here marshals tensors into pointers and calls the entry point of the same
name; all arithmetic runs in the HIP kernels.  torch provides device memory
and the current stream only.  There is no CPU fallback: the functions raise
if the library is not built or a tensor is not on a GPU.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field

import torch

from . import _lib
from ._lib import (GRPO_ADV_GROUP_NORM, GRPO_ADV_SUCCESS_FILTER, GRPO_BF16, GRPO_F32,  # noqa: F401
                   GRPO_FLAG_ACTION, GRPO_FLAG_NONFINITE, GRPO_FLAG_OFFSETS, GRPO_NORM_CONST_K,
                   GRPO_NORM_TRAJ_STEPS, GrpoError)

__all__ = ["grpo_advantages", "grpo_advantages_ex", "grpo_loss_workspace_bytes", "grpo_loss_fwd_bwd", "fused_lmhead_workspace_bytes",
           "fused_lmhead_grpo", "fused_lmhead_blocked_workspace_bytes", "fused_lmhead_grpo_blocked", "grpo_token_logp", "grpo_vocab_shard_stats", "grpo_loss_fwd_bwd_vocab_shard",
           "vocab_stats_fields", "fused_lmhead_vocab_shard_stats", "fused_lmhead_grpo_vocab_shard",
           "vocab_shard_logits_buffer", "GrpoLoss", "FusedLmHeadGrpoLoss", "loss",
           "fused_lmhead_token_logp",
           "grpo_status_str", "LossAux", "GrpoError"]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (no CPU path)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _workspace(workspace, need, device):
    """The caller's workspace (a contiguous tensor of any dtype on the inputs' device; its size in bytes is what the
    library is told) or a new one of ``need`` bytes."""
    if workspace is None:
        return torch.empty(max(int(need), 1), dtype=torch.uint8, device=device)
    _dev(workspace, "workspace")
    if workspace.device != torch.device(device):
        raise ValueError("workspace must be on the inputs' device")
    return workspace


def _nbytes(t):
    return t.numel() * t.element_size()


def _loss_out(loss_out, device):
    """The caller's fp64 loss scalar on the inputs' device, or a new one."""
    if loss_out is None:
        return torch.empty(1, dtype=torch.float64, device=device)
    _dev(loss_out, "loss_out")
    if loss_out.dtype != torch.float64 or loss_out.numel() < 1 or loss_out.device != torch.device(device):
        raise ValueError("loss_out must be a float64 GPU tensor of at least one element on the inputs' device")
    return loss_out


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, what):
    if status != _lib.GRPO_OK:
        raise GrpoError(status, what)


def grpo_status_str(status: int) -> str:
    return _lib.status_str(status)


def grpo_advantages(rewards: torch.Tensor, group_size: int, ddof: int = 1, std_eps: float = 0.0,
                    out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Group-relative advantages A_i (fp32 [N]) from rewards (fp32 [N])."""
    _dev(rewards, "rewards")
    if rewards.dtype != torch.float32:
        raise TypeError("rewards must be float32")
    out = torch.empty_like(rewards) if out is None else _dev(out, "out")
    st = _lib.load().grpo_advantages(_ptr(rewards), rewards.numel(), int(group_size), int(ddof), float(std_eps),
                                     _ptr(out), _stream(stream))
    _check(st, "grpo_advantages")
    return out


def grpo_advantages_ex(rewards: torch.Tensor, group_size: int, mode: int = GRPO_ADV_GROUP_NORM, ddof: int = 1,
                       std_eps: float = 0.0, out: torch.Tensor | None = None, mixed: bool = True, stream=None):
    """Advantages under ``mode`` (group-normalised, or the RAFT++ success filter) and, with ``mixed``, DAPO's
    mixed-group mask (int32 [N / G]) and count (int32 [1]).  Returns (adv, group_mixed or None, n_mixed or None)."""
    _dev(rewards, "rewards")
    if rewards.dtype != torch.float32:
        raise TypeError("rewards must be float32")
    out = torch.empty_like(rewards) if out is None else _dev(out, "out")
    gm = nm = None
    if mixed:
        gm = torch.empty(max(rewards.numel() // max(int(group_size), 1), 1), dtype=torch.int32, device=rewards.device)
        nm = torch.empty(1, dtype=torch.int32, device=rewards.device)
    st = _lib.load().grpo_advantages_ex(_ptr(rewards), rewards.numel(), int(group_size), int(mode), int(ddof),
                                        float(std_eps), _ptr(out), _ptr(gm), _ptr(nm), _stream(stream))
    _check(st, "grpo_advantages_ex")
    return out, gm, nm


def grpo_loss_workspace_bytes(T: int, n_traj: int) -> int:
    return int(_lib.load().grpo_loss_workspace_bytes(int(T), int(n_traj)))


def loss(logits: torch.Tensor, actions: torch.Tensor, old_logp: torch.Tensor, rewards: torch.Tensor,
         step_tok_off: torch.Tensor, traj_step_off: torch.Tensor, group_size: int, *, ddof: int = 1,
         std_eps: float = 0.0, stream=None, **opts):
    """The loss and dlogits from rewards: the group-relative advantages of Sec. 3.2 (``grpo_advantages``), then
    ``grpo_loss_fwd_bwd`` with ``old_logp`` as the behaviour log-probs, on the same stream.  ``opts``: the keyword
    options of ``grpo_loss_fwd_bwd``.  Returns (loss [1] fp64, dlogits)."""
    adv = grpo_advantages(rewards, group_size, ddof=ddof, std_eps=std_eps, stream=stream)
    return grpo_loss_fwd_bwd(logits, actions, old_logp, adv, step_tok_off, traj_step_off, group_size,
                             stream=stream, **opts)


def fused_lmhead_workspace_bytes(T: int, H: int, V: int, vocab_chunk: int, n_traj: int) -> int:
    return int(_lib.load().fused_lmhead_workspace_bytes(int(T), int(H), int(V), int(vocab_chunk), int(n_traj)))


def fused_lmhead_blocked_workspace_bytes(T: int, H: int, V: int, token_block: int, n_traj: int) -> int:
    return int(_lib.load().fused_lmhead_blocked_workspace_bytes(int(T), int(H), int(V), int(token_block),
                                                                int(n_traj)))


@dataclass
class LossAux:
    """Optional outputs of the loss entry points (allocate with ``LossAux.alloc``)."""
    token_logp: torch.Tensor | None = None
    tok_traj: torch.Tensor | None = None
    traj_tok_off: torch.Tensor | None = None
    gather_idx: torch.Tensor | None = None
    traj_loss: torch.Tensor | None = None
    clip_counts: torch.Tensor | None = None
    ratio_stats: torch.Tensor | None = None
    error_flags: torch.Tensor | None = None
    hot_events: tuple | None = field(default=None)  # (begin, end) raw hipEvent_t handles

    @staticmethod
    def alloc(T: int, n_traj: int, device, which=("token_logp", "tok_traj", "traj_tok_off", "gather_idx",
                                                   "traj_loss", "clip_counts", "ratio_stats",
                                                   "error_flags")) -> "LossAux":
        mk = {
            "token_logp": lambda: torch.empty(T, dtype=torch.float32, device=device),
            "tok_traj": lambda: torch.empty(T, dtype=torch.int32, device=device),
            "traj_tok_off": lambda: torch.empty(n_traj + 1, dtype=torch.int32, device=device),
            "gather_idx": lambda: torch.empty(T, dtype=torch.int64, device=device),
            "traj_loss": lambda: torch.empty(n_traj, dtype=torch.float64, device=device),
            "clip_counts": lambda: torch.empty(2, dtype=torch.int64, device=device),
            "ratio_stats": lambda: torch.empty(8, dtype=torch.float64, device=device),
            "error_flags": lambda: torch.empty(1, dtype=torch.int32, device=device),
        }
        return LossAux(**{k: mk[k]() for k in which})

    def _c(self, T: int, n_traj: int):
        a = _lib.Aux()
        want = {"token_logp": (torch.float32, T), "tok_traj": (torch.int32, T), "traj_tok_off": (torch.int32, n_traj + 1),
                "gather_idx": (torch.int64, T), "traj_loss": (torch.float64, n_traj), "clip_counts": (torch.int64, 2),
                "ratio_stats": (torch.float64, 8), "error_flags": (torch.int32, 1)}
        for name, (dt, n) in want.items():
            t = getattr(self, name)
            if t is not None:
                _dev(t, name)
                if t.dtype != dt or t.numel() < n:
                    raise ValueError(f"aux.{name} must be {dt} with at least {n} elements")
            setattr(a, name, None if t is None else t.data_ptr())
        if self.hot_events is not None:
            a.hot_begin, a.hot_end = self.hot_events
        return a


def _segments(step_tok_off, traj_step_off, group_size):
    _dev(step_tok_off, "step_tok_off")
    _dev(traj_step_off, "traj_step_off")
    if step_tok_off.dtype != torch.int32 or traj_step_off.dtype != torch.int32:
        raise TypeError("offsets must be int32")
    seg = _lib.Segments()
    seg.n_traj = traj_step_off.numel() - 1
    seg.group_size = int(group_size)
    seg.n_steps = step_tok_off.numel() - 1
    seg.step_tok_off = step_tok_off.data_ptr()
    seg.traj_step_off = traj_step_off.data_ptr()
    return seg


def _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total):
    p = _lib.LossParams()
    p.norm = int(norm)
    p.k = float(k)
    p.eps_low = float(eps_low)
    p.eps_high = float(eps_high)
    p.dual_clip_c = float(dual_clip_c)
    p.grad_scale = float(grad_scale)
    p.n_groups_total = float(n_groups_total)
    return p


def _f32(t, name):
    if t is None:
        return None
    _dev(t, name)
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")
    return t


def grpo_loss_fwd_bwd(logits: torch.Tensor, actions: torch.Tensor, behave_logp: torch.Tensor, adv: torch.Tensor,
                      step_tok_off: torch.Tensor, traj_step_off: torch.Tensor, group_size: int, *,
                      V: int | None = None, prox_logp: torch.Tensor | None = None, norm: int = GRPO_NORM_CONST_K,
                      k: float = 10.0, eps_low: float = 0.2, eps_high: float = 0.2, dual_clip_c: float = 0.0,
                      grad_scale: float = 1.0, n_groups_total: float = 0.0, dlogits=True,
                      aux: LossAux | None = None, workspace: torch.Tensor | None = None,
                      loss_out: torch.Tensor | None = None, stream=None):
    """Loss (fp64 device scalar) and dlogits of Eq. 1 from logits [T, ld].

    ``dlogits``: True allocates a [T, ld] tensor like ``logits``; None/False is
    forward only; a tensor is written in place (it may be ``logits`` itself).
    Returns (loss [1] fp64, dlogits or None).
    """
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be [T, ld] with unit column stride")
    if not logits.is_cuda:
        raise ValueError("logits must be a GPU tensor (no CPU path)")
    dt = {torch.bfloat16: GRPO_BF16, torch.float32: GRPO_F32}.get(logits.dtype)
    if dt is None:
        raise TypeError("logits must be bfloat16 or float32")
    T = logits.shape[0]
    ld = logits.stride(0) if T > 0 else logits.shape[1]
    Vv = logits.shape[1] if V is None else int(V)
    _dev(actions, "actions")
    if actions.dtype != torch.int32:
        raise TypeError("actions must be int32")
    seg = _segments(step_tok_off, traj_step_off, group_size)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    if dlogits is True:
        dlogits = torch.empty_like(logits)
    elif dlogits is False:
        dlogits = None
    if dlogits is not None and (dlogits.shape != logits.shape or dlogits.stride() != logits.stride()
                                or dlogits.dtype != logits.dtype):
        raise ValueError("dlogits must match logits in shape, stride and dtype")
    need = grpo_loss_workspace_bytes(T, seg.n_traj)
    workspace = _workspace(workspace, need, logits.device)
    loss_out = _loss_out(loss_out, logits.device)
    ca = aux._c(T, seg.n_traj) if aux is not None else None
    st = _lib.load().grpo_loss_fwd_bwd(
        _ptr(logits), dt, T, Vv, ld, _ptr(actions), _ptr(_f32(behave_logp, "behave_logp")),
        _ptr(_f32(prox_logp, "prox_logp")), _ptr(_f32(adv, "adv")), ctypes.byref(seg), ctypes.byref(par),
        _ptr(loss_out), _ptr(dlogits), ctypes.byref(ca) if ca is not None else None, _ptr(workspace),
        _nbytes(workspace), _stream(stream))
    _check(st, "grpo_loss_fwd_bwd")
    return loss_out, dlogits


def _fused_call(entry: str, ws_bytes, hidden, w_lm, actions, behave_logp, adv, step_tok_off, traj_step_off,
                group_size, sched, prox_logp, norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total,
                dhidden, dw_lm, accumulate_dw, aux, workspace, loss_out, stream, extra=()):
    _dev(hidden, "hidden")
    _dev(w_lm, "w_lm")
    if hidden.dtype != torch.bfloat16 or w_lm.dtype != torch.bfloat16:
        raise TypeError("hidden and w_lm must be bfloat16")
    T, H = hidden.shape
    H2, V = w_lm.shape
    if H2 != H:
        raise ValueError("hidden and w_lm disagree on H")
    _dev(actions, "actions")
    seg = _segments(step_tok_off, traj_step_off, group_size)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    if dhidden is None:
        dhidden = torch.empty_like(hidden)
    if dw_lm is None:
        dw_lm = torch.empty((H, V), dtype=torch.float32, device=hidden.device)
    _dev(dhidden, "dhidden")
    _dev(dw_lm, "dw_lm")
    need = ws_bytes(T, H, V, sched, seg.n_traj)
    workspace = _workspace(workspace, need, hidden.device)
    loss_out = _loss_out(loss_out, hidden.device)
    ca = aux._c(T, seg.n_traj) if aux is not None else None
    st = getattr(_lib.load(), entry)(
        _ptr(hidden), _ptr(w_lm), T, H, V, int(sched), _ptr(actions), _ptr(_f32(behave_logp, "behave_logp")),
        _ptr(_f32(prox_logp, "prox_logp")), _ptr(_f32(adv, "adv")), ctypes.byref(seg), ctypes.byref(par),
        _ptr(loss_out), _ptr(dhidden), _ptr(dw_lm), int(bool(accumulate_dw)),
        ctypes.byref(ca) if ca is not None else None, _ptr(workspace), _nbytes(workspace), _stream(stream), *extra)
    _check(st, entry)
    return loss_out, dhidden, dw_lm


def fused_lmhead_grpo(hidden: torch.Tensor, w_lm: torch.Tensor, actions: torch.Tensor, behave_logp: torch.Tensor,
                      adv: torch.Tensor, step_tok_off: torch.Tensor, traj_step_off: torch.Tensor, group_size: int, *,
                      vocab_chunk: int = 8192, prox_logp: torch.Tensor | None = None,
                      norm: int = GRPO_NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2, eps_high: float = 0.2,
                      dual_clip_c: float = 0.0, grad_scale: float = 1.0, n_groups_total: float = 0.0,
                      dhidden: torch.Tensor | None = None, dw_lm: torch.Tensor | None = None,
                      accumulate_dw: bool = False, aux: LossAux | None = None,
                      workspace: torch.Tensor | None = None, loss_out: torch.Tensor | None = None, stream=None):
    """Loss, dhidden (bf16 [T, H]) and dW (fp32 [H, V]) from hidden [T, H] and W [H, V] (bf16), over vocabulary
    chunks with the logits recomputed for the backward products.

    Returns (loss [1] fp64, dhidden, dw_lm).
    """
    return _fused_call("fused_lmhead_grpo", fused_lmhead_workspace_bytes, hidden, w_lm, actions, behave_logp, adv,
                       step_tok_off, traj_step_off, group_size, vocab_chunk, prox_logp, norm, k, eps_low, eps_high,
                       dual_clip_c, grad_scale, n_groups_total, dhidden, dw_lm, accumulate_dw, aux, workspace,
                       loss_out, stream)


def fused_lmhead_grpo_blocked(hidden: torch.Tensor, w_lm: torch.Tensor, actions: torch.Tensor,
                              behave_logp: torch.Tensor, adv: torch.Tensor, step_tok_off: torch.Tensor,
                              traj_step_off: torch.Tensor, group_size: int, *, token_block: int = 8192,
                              prox_logp: torch.Tensor | None = None, norm: int = GRPO_NORM_CONST_K, k: float = 10.0,
                              eps_low: float = 0.2, eps_high: float = 0.2, dual_clip_c: float = 0.0,
                              grad_scale: float = 1.0, n_groups_total: float = 0.0,
                              dhidden: torch.Tensor | None = None, dw_lm: torch.Tensor | None = None,
                              accumulate_dw: bool = False, aux: LossAux | None = None,
                              workspace: torch.Tensor | None = None, loss_out: torch.Tensor | None = None,
                              stream=None, aux_stream=None):
    """As fused_lmhead_grpo, over blocks of `token_block` tokens whose fp32 logits are kept in the workspace
    between the forward and backward products (three products instead of four).  With `aux_stream` (a second
    torch.cuda.Stream on the same device), each block's D pass runs on it beside the next block's forward
    product; the results are complete in `stream`'s order either way.

    Returns (loss [1] fp64, dhidden, dw_lm).
    """
    if aux_stream is not None and aux_stream.device != hidden.device:
        raise ValueError("aux_stream must be on hidden's device")
    return _fused_call("fused_lmhead_grpo_blocked", fused_lmhead_blocked_workspace_bytes, hidden, w_lm, actions,
                       behave_logp, adv, step_tok_off, traj_step_off, group_size, token_block, prox_logp, norm, k,
                       eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total, dhidden, dw_lm, accumulate_dw,
                       aux, workspace, loss_out, stream,
                       extra=(None if aux_stream is None else ctypes.c_void_p(aux_stream.cuda_stream),))


def grpo_token_logp(logits: torch.Tensor, actions: torch.Tensor, *, V: int | None = None, entropy: bool = True,
                    error_flags: torch.Tensor | None = None, stream=None):
    """Forward only: each token row's action log-prob and (optionally) policy entropy, both fp32 [T].

    ``logits`` is [T, ld] (bf16 or fp32, unit column stride); V defaults to the column count.
    ``error_flags`` (int32 [1], optional) receives GRPO_FLAG_* bits.  Returns (logp, entropy or None).
    """
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be [T, ld] with unit column stride")
    if not logits.is_cuda:
        raise ValueError("logits must be a GPU tensor (no CPU path)")
    dt = {torch.bfloat16: GRPO_BF16, torch.float32: GRPO_F32}.get(logits.dtype)
    if dt is None:
        raise TypeError("logits must be bfloat16 or float32")
    T = logits.shape[0]
    ld = logits.stride(0) if T > 0 else logits.shape[1]
    Vv = logits.shape[1] if V is None else int(V)
    _dev(actions, "actions")
    if actions.dtype != torch.int32:
        raise TypeError("actions must be int32")
    logp = torch.empty(T, dtype=torch.float32, device=logits.device)
    ent = torch.empty(T, dtype=torch.float32, device=logits.device) if entropy else None
    if error_flags is not None and (error_flags.dtype != torch.int32 or not error_flags.is_cuda):
        raise ValueError("error_flags must be an int32 GPU tensor")
    st = _lib.load().grpo_token_logp(_ptr(logits), dt, T, Vv, ld, _ptr(actions), _ptr(logp), _ptr(ent),
                                     _ptr(error_flags), _stream(stream))
    _check(st, "grpo_token_logp")
    return logp, ent


VOCAB_STATS_BYTES = 24  # one grpo_vocab_stats record: fp64 m, s, z_a


def fused_lmhead_token_logp(hidden: torch.Tensor, w_lm: torch.Tensor, actions: torch.Tensor, *,
                            entropy: bool = True, error_flags: torch.Tensor | None = None,
                            workspace: torch.Tensor | None = None, stream=None):
    """Forward only from hidden states: the action's log-prob (fp32 [T]) and, if ``entropy``, the policy entropy
    (fp32 [T]) of softmax(h W) per token, without storing the logits.  Returns (token_logp, token_entropy or
    None)."""
    _dev(hidden, "hidden")
    _dev(w_lm, "w_lm")
    if hidden.dtype != torch.bfloat16 or w_lm.dtype != torch.bfloat16:
        raise TypeError("hidden and w_lm must be bfloat16")
    T, H = hidden.shape
    H2, V = w_lm.shape
    if H2 != H:
        raise ValueError("hidden and w_lm disagree on H")
    _dev(actions, "actions")
    if actions.dtype != torch.int32:
        raise TypeError("actions must be int32")
    if error_flags is not None and (error_flags.dtype != torch.int32 or not error_flags.is_cuda):
        raise ValueError("error_flags must be an int32 GPU tensor")
    lib = _lib.load()
    need = int(lib.fused_lmhead_token_logp_workspace_bytes(T, H, V))
    workspace = _workspace(workspace, need, hidden.device)
    logp = torch.empty(T, dtype=torch.float32, device=hidden.device)
    ent = torch.empty(T, dtype=torch.float32, device=hidden.device) if entropy else None
    st = lib.fused_lmhead_token_logp(_ptr(hidden), _ptr(w_lm), T, H, V, _ptr(actions), _ptr(logp), _ptr(ent),
                                     _ptr(error_flags), _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "fused_lmhead_token_logp")
    return logp, ent


def vocab_stats_fields(stats: torch.Tensor):
    """Views of a uint8 [..., T, 24] record tensor as (m, z_a, s), each fp64 [..., T]."""
    f64 = stats.view(torch.float64)
    return f64[..., 0], f64[..., 2], f64[..., 1]


def _logits2d(logits, name="logits"):
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError(f"{name} must be [T, ld] with unit column stride")
    if not logits.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (no CPU path)")
    dt = {torch.bfloat16: GRPO_BF16, torch.float32: GRPO_F32}.get(logits.dtype)
    if dt is None:
        raise TypeError(f"{name} must be bfloat16 or float32")
    T = logits.shape[0]
    ld = logits.stride(0) if T > 0 else logits.shape[1]
    return dt, T, ld


def grpo_vocab_shard_stats(logits: torch.Tensor, actions: torch.Tensor, v_begin: int, *, V: int | None = None,
                           stats: torch.Tensor | None = None, error_flags: torch.Tensor | None = None, stream=None):
    """Step 1 of the vocabulary-sharded loss: each row of the shard (global columns [v_begin, v_begin + V)) reduced
    to its record.  Returns uint8 [T, 24] records (read them with ``vocab_stats_fields``)."""
    dt, T, ld = _logits2d(logits)
    Vv = logits.shape[1] if V is None else int(V)
    _dev(actions, "actions")
    if actions.dtype != torch.int32:
        raise TypeError("actions must be int32")
    if stats is None:
        stats = torch.empty((T, VOCAB_STATS_BYTES), dtype=torch.uint8, device=logits.device)
    _dev(stats, "stats")
    if stats.dtype != torch.uint8 or tuple(stats.shape) != (T, VOCAB_STATS_BYTES):
        raise ValueError(f"stats must be uint8 [T, {VOCAB_STATS_BYTES}]")
    if error_flags is not None and (error_flags.dtype != torch.int32 or not error_flags.is_cuda):
        raise ValueError("error_flags must be an int32 GPU tensor")
    st = _lib.load().grpo_vocab_shard_stats(_ptr(logits), dt, T, Vv, ld, int(v_begin), _ptr(actions), _ptr(stats),
                                            _ptr(error_flags), _stream(stream))
    _check(st, "grpo_vocab_shard_stats")
    return stats


def grpo_loss_fwd_bwd_vocab_shard(logits: torch.Tensor, stats_all: torch.Tensor, v_begin: int, V_total: int,
                                  actions: torch.Tensor, behave_logp: torch.Tensor, adv: torch.Tensor,
                                  step_tok_off: torch.Tensor, traj_step_off: torch.Tensor, group_size: int, *,
                                  V: int | None = None, prox_logp: torch.Tensor | None = None,
                                  norm: int = GRPO_NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2,
                                  eps_high: float = 0.2, dual_clip_c: float = 0.0, grad_scale: float = 1.0,
                                  n_groups_total: float = 0.0, dlogits=True, aux: LossAux | None = None,
                                  workspace: torch.Tensor | None = None, loss_out: torch.Tensor | None = None,
                                  stream=None):
    """Step 2 of the vocabulary-sharded loss: the loss (fp64 [1], the whole rows') and this shard's dlogits, from
    the shard's logits and every shard's records ``stats_all`` (uint8 [n_shards, T, 24], in shard order).

    ``dlogits``: True allocates a tensor like ``logits``; None/False is forward only; a tensor is written in place.
    Returns (loss, dlogits or None).
    """
    dt, T, ld = _logits2d(logits)
    Vv = logits.shape[1] if V is None else int(V)
    _dev(actions, "actions")
    if actions.dtype != torch.int32:
        raise TypeError("actions must be int32")
    _dev(stats_all, "stats_all")
    if stats_all.dtype != torch.uint8 or stats_all.dim() != 3 or tuple(stats_all.shape[1:]) != (T, VOCAB_STATS_BYTES):
        raise ValueError(f"stats_all must be uint8 [n_shards, T, {VOCAB_STATS_BYTES}]")
    n_shards = stats_all.shape[0]
    seg = _segments(step_tok_off, traj_step_off, group_size)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    if dlogits is True:
        dlogits = torch.empty_like(logits)
    elif dlogits is False:
        dlogits = None
    if dlogits is not None and (dlogits.shape != logits.shape or dlogits.stride() != logits.stride()
                                or dlogits.dtype != logits.dtype):
        raise ValueError("dlogits must match logits in shape, stride and dtype")
    need = grpo_loss_workspace_bytes(T, seg.n_traj)
    workspace = _workspace(workspace, need, logits.device)
    loss_out = _loss_out(loss_out, logits.device)
    ca = aux._c(T, seg.n_traj) if aux is not None else None
    st = _lib.load().grpo_loss_fwd_bwd_vocab_shard(
        _ptr(logits), dt, T, Vv, ld, int(v_begin), int(V_total), _ptr(stats_all), int(n_shards), _ptr(actions),
        _ptr(_f32(behave_logp, "behave_logp")), _ptr(_f32(prox_logp, "prox_logp")), _ptr(_f32(adv, "adv")),
        ctypes.byref(seg), ctypes.byref(par), _ptr(loss_out), _ptr(dlogits),
        ctypes.byref(ca) if ca is not None else None, _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "grpo_loss_fwd_bwd_vocab_shard")
    return loss_out, dlogits


def vocab_shard_logits_buffer(T: int, V_shard: int, device) -> torch.Tensor:
    """An fp32 buffer for the shard's logits kept between the two steps of the sharded fused LM head."""
    n = int(_lib.load().fused_lmhead_vocab_shard_logits_bytes(int(T), int(V_shard))) // 4
    return torch.empty(max(n, 1), dtype=torch.float32, device=device)


def _check_logits_buffer(buf: torch.Tensor, T: int, V_shard: int):
    _dev(buf, "logits buffer")
    need = int(_lib.load().fused_lmhead_vocab_shard_logits_bytes(int(T), int(V_shard)))
    if buf.dtype != torch.float32 or not buf.is_contiguous() or buf.numel() * 4 < need:
        raise ValueError(f"the logits buffer must be contiguous float32 of at least {need} bytes")


def fused_lmhead_vocab_shard_stats(hidden: torch.Tensor, w_shard: torch.Tensor, actions: torch.Tensor, v_begin: int,
                                   *, stats: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                                   logits_out: torch.Tensor | None = None, stream=None):
    """Step 1 of the vocabulary-sharded fused LM head: each row of h W_shard (W's columns [v_begin, v_begin +
    V_shard)) reduced to its record.  Returns uint8 [T, 24] records (read them with ``vocab_stats_fields``).
    ``logits_out`` (fp32, ``fused_lmhead_vocab_shard_logits_bytes(T, V_shard) / 4`` elements, see
    ``vocab_shard_logits_buffer``) also receives the shard's logits for step 2."""
    _dev(hidden, "hidden")
    _dev(w_shard, "w_shard")
    if hidden.dtype != torch.bfloat16 or w_shard.dtype != torch.bfloat16:
        raise TypeError("hidden and w_shard must be bfloat16")
    T, H = hidden.shape
    H2, Vs = w_shard.shape
    if H2 != H:
        raise ValueError("hidden and w_shard disagree on H")
    _dev(actions, "actions")
    if stats is None:
        stats = torch.empty((T, VOCAB_STATS_BYTES), dtype=torch.uint8, device=hidden.device)
    _dev(stats, "stats")
    if stats.dtype != torch.uint8 or tuple(stats.shape) != (T, VOCAB_STATS_BYTES):
        raise ValueError(f"stats must be uint8 [T, {VOCAB_STATS_BYTES}]")
    lib = _lib.load()
    need = lib.fused_lmhead_vocab_shard_stats_workspace_bytes(T, H, Vs)
    workspace = _workspace(workspace, need, hidden.device)
    if logits_out is not None:
        _check_logits_buffer(logits_out, T, Vs)
    st = lib.fused_lmhead_vocab_shard_stats(_ptr(hidden), _ptr(w_shard), T, H, Vs, int(v_begin), _ptr(actions),
                                            _ptr(stats), _ptr(logits_out), _ptr(workspace), _nbytes(workspace),
                                            _stream(stream))
    _check(st, "fused_lmhead_vocab_shard_stats")
    return stats


def fused_lmhead_grpo_vocab_shard(hidden: torch.Tensor, w_shard: torch.Tensor, stats_all: torch.Tensor, v_begin: int,
                                  V_total: int, actions: torch.Tensor, behave_logp: torch.Tensor, adv: torch.Tensor,
                                  step_tok_off: torch.Tensor, traj_step_off: torch.Tensor, group_size: int, *,
                                  vocab_chunk: int = 8192, prox_logp: torch.Tensor | None = None,
                                  norm: int = GRPO_NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2,
                                  eps_high: float = 0.2, dual_clip_c: float = 0.0, grad_scale: float = 1.0,
                                  n_groups_total: float = 0.0, dhidden_partial: torch.Tensor | None = None,
                                  dw_shard: torch.Tensor | None = None, accumulate_dw: bool = False,
                                  aux: LossAux | None = None, workspace: torch.Tensor | None = None,
                                  loss_out: torch.Tensor | None = None, logits_in: torch.Tensor | None = None,
                                  stream=None):
    """Step 2 of the vocabulary-sharded fused LM head: the loss (fp64 [1]), this shard's partial dhidden (fp32
    [T, H], to be summed over the shards) and its dW columns (fp32 [H, V_shard]), from every shard's records
    ``stats_all`` (uint8 [n_shards, T, 24], in shard order).  With ``logits_in`` (the buffer step 1 filled), D
    comes from the kept logits instead of a recomputed product.  Returns (loss, dhidden_partial, dw_shard)."""
    _dev(hidden, "hidden")
    _dev(w_shard, "w_shard")
    if hidden.dtype != torch.bfloat16 or w_shard.dtype != torch.bfloat16:
        raise TypeError("hidden and w_shard must be bfloat16")
    T, H = hidden.shape
    H2, Vs = w_shard.shape
    if H2 != H:
        raise ValueError("hidden and w_shard disagree on H")
    _dev(actions, "actions")
    _dev(stats_all, "stats_all")
    if stats_all.dtype != torch.uint8 or stats_all.dim() != 3 or tuple(stats_all.shape[1:]) != (T, VOCAB_STATS_BYTES):
        raise ValueError(f"stats_all must be uint8 [n_shards, T, {VOCAB_STATS_BYTES}]")
    seg = _segments(step_tok_off, traj_step_off, group_size)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    if dhidden_partial is None:
        dhidden_partial = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    if dw_shard is None:
        dw_shard = torch.empty((H, Vs), dtype=torch.float32, device=hidden.device)
    _dev(dhidden_partial, "dhidden_partial")
    _dev(dw_shard, "dw_shard")
    if dhidden_partial.dtype != torch.float32 or dw_shard.dtype != torch.float32:
        raise TypeError("dhidden_partial and dw_shard must be float32")
    if logits_in is not None:
        _check_logits_buffer(logits_in, T, Vs)
        vocab_chunk = (Vs + 255) // 256 * 256  # the whole shard as one chunk
    need = fused_lmhead_workspace_bytes(T, H, Vs, vocab_chunk, seg.n_traj)
    workspace = _workspace(workspace, need, hidden.device)
    loss_out = _loss_out(loss_out, hidden.device)
    ca = aux._c(T, seg.n_traj) if aux is not None else None
    st = _lib.load().fused_lmhead_grpo_vocab_shard(
        _ptr(hidden), _ptr(w_shard), T, H, Vs, int(v_begin), int(V_total), int(vocab_chunk), _ptr(stats_all),
        int(stats_all.shape[0]), _ptr(actions), _ptr(_f32(behave_logp, "behave_logp")),
        _ptr(_f32(prox_logp, "prox_logp")), _ptr(_f32(adv, "adv")), ctypes.byref(seg), ctypes.byref(par),
        _ptr(loss_out), _ptr(dhidden_partial), _ptr(dw_shard), int(bool(accumulate_dw)),
        ctypes.byref(ca) if ca is not None else None, _ptr(logits_in), _ptr(workspace), _nbytes(workspace),
        _stream(stream))
    _check(st, "fused_lmhead_grpo_vocab_shard")
    return loss_out, dhidden_partial, dw_shard


from .autograd import FusedLmHeadGrpoLoss, GrpoLoss  # noqa: E402  (needs the entry points above)
