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
                   GRPO_FLAG_ACTION, GRPO_FLAG_NONFINITE, GRPO_FLAG_OFFSETS, GRPO_NOALLOC_SCRATCH_BYTES,
                   GRPO_NORM_CONST_K, GRPO_NORM_TRAJ_STEPS, GrpoError)

__all__ = ["grpo_advantages", "grpo_advantages_ex", "grpo_loss_workspace_bytes", "grpo_loss_fwd_bwd",
           "grpo_loss_fwd_bwd_noalloc", "fused_lmhead_workspace_bytes",
           "fused_lmhead_grpo", "fused_lmhead_blocked_workspace_bytes", "fused_lmhead_grpo_blocked", "grpo_token_logp", "grpo_vocab_shard_stats", "grpo_loss_fwd_bwd_vocab_shard",
           "vocab_stats_fields", "fused_lmhead_vocab_shard_stats", "fused_lmhead_grpo_vocab_shard",
           "vocab_shard_logits_buffer", "GrpoLoss", "FusedLmHeadGrpoLoss", "loss",
           "fused_lmhead_token_logp",
           "grpo_status_str", "LossAux", "GrpoError"]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# Argument checks run in two stages, so that each is seen whatever the other would say: first every tensor's dtype
# and size (_meta), then where the tensors live (_placed: GPU, the inputs' device, contiguous).  Nothing reaches the
# library before both pass, so the library is never handed a host pointer or a buffer it would overrun.

def _meta(t, name, dtype, n=None, shape=None, optional=False):
    """dtype and size of a caller tensor: dtype (None = any), at least n elements, or exactly this shape."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if n is not None and t.numel() < n:
        raise ValueError(f"{name} must hold at least {n} elements, got {t.numel()}")
    return t


def _placed(device, strided=(), **tensors):
    """Every tensor given is on the GPU, on `device`, and contiguous (those named in `strided` only need a unit
    column stride, checked with their shape)."""
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor (no CPU path)")
        if t.device != device:
            raise ValueError(f"{name} must be on {device} (the inputs' device), got {t.device}")
        if name not in strided and not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")


def _logits2d(logits, name="logits"):
    """dtype code, rows and row stride of a [T, ld] logits tensor with unit column stride."""
    _meta(logits, name, None)
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError(f"{name} must be [T, ld] with unit column stride")
    dt = {torch.bfloat16: GRPO_BF16, torch.float32: GRPO_F32}.get(logits.dtype)
    if dt is None:
        raise TypeError(f"{name} must be bfloat16 or float32")
    T = logits.shape[0]
    ld = logits.stride(0) if T > 0 else logits.shape[1]
    return dt, T, ld


def _hidden_w(hidden, w, w_name):
    """(T, H, V) of bf16 hidden [T, H] and weight [H, V]."""
    _meta(hidden, "hidden", torch.bfloat16)
    _meta(w, w_name, torch.bfloat16)
    if hidden.dim() != 2 or w.dim() != 2:
        raise ValueError(f"hidden and {w_name} must be 2-D")
    T, H = hidden.shape
    H2, V = w.shape
    if H2 != H:
        raise ValueError(f"hidden and {w_name} disagree on H")
    return T, H, V


def _dlogits_arg(dlogits, logits):
    if dlogits is True:
        return torch.empty_like(logits)
    if dlogits is False or dlogits is None:
        return None
    _meta(dlogits, "dlogits", logits.dtype)
    if dlogits.shape != logits.shape or dlogits.stride() != logits.stride():
        raise ValueError("dlogits must match logits in shape, stride and dtype")
    return dlogits


def _workspace(workspace, need, device):
    """The caller's workspace (a contiguous GPU tensor of any dtype on the inputs' device; its size in bytes is what
    the library is told, and the library refuses one that is too small) or a new one of ``need`` bytes."""
    if workspace is None:
        return torch.empty(max(int(need), 1), dtype=torch.uint8, device=device)
    _placed(device, workspace=workspace)
    return workspace


def _nbytes(t):
    return t.numel() * t.element_size()


def _loss_out(loss_out, device):
    """The caller's fp64 loss scalar on the inputs' device, or a new one."""
    if loss_out is None:
        return torch.empty(1, dtype=torch.float64, device=device)
    _meta(loss_out, "loss_out", torch.float64, n=1)
    _placed(device, loss_out=loss_out)
    return loss_out


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, what):
    if status != _lib.GRPO_OK:
        raise GrpoError(status, what)


def _n_traj(traj_step_off):
    return max(traj_step_off.numel() - 1, 0)


def grpo_status_str(status: int) -> str:
    return _lib.status_str(status)


def grpo_advantages(rewards: torch.Tensor, group_size: int, ddof: int = 1, std_eps: float = 0.0,
                    out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Group-relative advantages A_i (fp32 [N]) from rewards (fp32 [N])."""
    _meta(rewards, "rewards", torch.float32)
    _meta(out, "out", torch.float32, n=rewards.numel(), optional=True)
    _placed(rewards.device, rewards=rewards, out=out)
    out = torch.empty_like(rewards) if out is None else out
    st = _lib.load().grpo_advantages(_ptr(rewards), rewards.numel(), int(group_size), int(ddof), float(std_eps),
                                     _ptr(out), _stream(stream))
    _check(st, "grpo_advantages")
    return out


def grpo_advantages_ex(rewards: torch.Tensor, group_size: int, mode: int = GRPO_ADV_GROUP_NORM, ddof: int = 1,
                       std_eps: float = 0.0, out: torch.Tensor | None = None, mixed: bool = True, stream=None):
    """Advantages under ``mode`` (group-normalised, or the RAFT++ success filter) and, with ``mixed``, DAPO's
    mixed-group mask (int32 [N / G]) and count (int32 [1]).  Returns (adv, group_mixed or None, n_mixed or None)."""
    _meta(rewards, "rewards", torch.float32)
    _meta(out, "out", torch.float32, n=rewards.numel(), optional=True)
    _placed(rewards.device, rewards=rewards, out=out)
    out = torch.empty_like(rewards) if out is None else out
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

    _WANT = {"token_logp": torch.float32, "tok_traj": torch.int32, "traj_tok_off": torch.int32,
             "gather_idx": torch.int64, "traj_loss": torch.float64, "clip_counts": torch.int64,
             "ratio_stats": torch.float64, "error_flags": torch.int32}

    def _meta(self, T: int, n_traj: int):
        """dtype and size of every output given (checked with the other arguments' before any device check)."""
        n = {"token_logp": T, "tok_traj": T, "traj_tok_off": n_traj + 1, "gather_idx": T, "traj_loss": n_traj,
             "clip_counts": 2, "ratio_stats": 8, "error_flags": 1}
        for name, dt in self._WANT.items():
            _meta(getattr(self, name), f"aux.{name}", dt, n=n[name], optional=True)

    def _c(self, T: int, n_traj: int, device):
        a = _lib.Aux()
        self._meta(T, n_traj)
        got = {name: getattr(self, name) for name in self._WANT}
        _placed(device, **{f"aux.{name}": t for name, t in got.items()})
        for name, t in got.items():
            setattr(a, name, None if t is None else t.data_ptr())
        if self.hot_events is not None:
            a.hot_begin, a.hot_end = self.hot_events
        return a


def _segments(step_tok_off, traj_step_off, group_size):
    """The CSR offsets (int32) as a grpo_segments struct (their device is checked with the other tensors)."""
    _meta(step_tok_off, "step_tok_off", torch.int32, n=1)
    _meta(traj_step_off, "traj_step_off", torch.int32, n=1)
    seg = _lib.Segments()
    seg.n_traj = _n_traj(traj_step_off)
    seg.group_size = int(group_size)
    seg.n_steps = step_tok_off.numel() - 1
    seg.step_tok_off = step_tok_off.data_ptr()
    seg.traj_step_off = traj_step_off.data_ptr()
    return seg


def _outputs_meta(T, n_traj, aux, loss_out):
    """dtypes and sizes of a loss call's optional outputs."""
    if aux is not None:
        aux._meta(T, n_traj)
    _meta(loss_out, "loss_out", torch.float64, n=1, optional=True)


def _token_inputs(T, n_traj, actions, behave_logp, prox_logp, adv):
    """dtypes and sizes of the per-token and per-trajectory inputs of a loss call."""
    _meta(actions, "actions", torch.int32, n=T)
    _meta(behave_logp, "behave_logp", torch.float32, n=T)
    _meta(prox_logp, "prox_logp", torch.float32, n=T, optional=True)
    _meta(adv, "adv", torch.float32, n=n_traj)


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
    return _logits_loss(True, logits, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, V,
                        prox_logp, norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total, dlogits, aux,
                        workspace, loss_out, stream)


def grpo_loss_fwd_bwd_noalloc(logits: torch.Tensor, actions: torch.Tensor, behave_logp: torch.Tensor,
                              adv: torch.Tensor, step_tok_off: torch.Tensor, traj_step_off: torch.Tensor,
                              group_size: int, *, V: int | None = None, prox_logp: torch.Tensor | None = None,
                              norm: int = GRPO_NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2,
                              eps_high: float = 0.2, dual_clip_c: float = 0.0, grad_scale: float = 1.0,
                              n_groups_total: float = 0.0, dlogits=True, aux: LossAux | None = None,
                              loss_out: torch.Tensor | None = None, stream=None):
    """grpo_loss_fwd_bwd with the library's own per-device scratch array as the workspace (the entry point allocates
    nothing; pass ``dlogits`` and ``loss_out`` tensors for a call in which nothing is allocated at all).  Calls that
    overlap on one device race on the array; the batch must fit it (grpo_loss_workspace_bytes(T, n_traj) <=
    GRPO_NOALLOC_SCRATCH_BYTES).  Returns (loss [1] fp64, dlogits or None)."""
    return _logits_loss(False, logits, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, V,
                        prox_logp, norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total, dlogits, aux,
                        None, loss_out, stream)


def _logits_loss(with_ws, logits, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, V, prox_logp,
                 norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total, dlogits, aux, workspace,
                 loss_out, stream):
    dt, T, ld = _logits2d(logits)
    Vv = logits.shape[1] if V is None else int(V)
    seg = _segments(step_tok_off, traj_step_off, group_size)
    _token_inputs(T, seg.n_traj, actions, behave_logp, prox_logp, adv)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    dlogits = _dlogits_arg(dlogits, logits) if dlogits is not True else True
    _outputs_meta(T, seg.n_traj, aux, loss_out)
    dev = logits.device
    _placed(dev, strided=("logits", "dlogits"), logits=logits, dlogits=None if dlogits is True else dlogits,
            actions=actions, behave_logp=behave_logp, prox_logp=prox_logp, adv=adv, step_tok_off=step_tok_off,
            traj_step_off=traj_step_off)
    ca = aux._c(T, seg.n_traj, dev) if aux is not None else None
    loss_out = _loss_out(loss_out, dev)
    dlogits = _dlogits_arg(dlogits, logits)
    args = (_ptr(logits), dt, T, Vv, ld, _ptr(actions), _ptr(behave_logp), _ptr(prox_logp), _ptr(adv),
            ctypes.byref(seg), ctypes.byref(par), _ptr(loss_out), _ptr(dlogits),
            ctypes.byref(ca) if ca is not None else None)
    if with_ws:
        workspace = _workspace(workspace, grpo_loss_workspace_bytes(T, seg.n_traj), dev)
        st = _lib.load().grpo_loss_fwd_bwd(*args, _ptr(workspace), _nbytes(workspace), _stream(stream))
        _check(st, "grpo_loss_fwd_bwd")
    else:
        st = _lib.load().grpo_loss_fwd_bwd_noalloc(*args, _stream(stream))
        _check(st, "grpo_loss_fwd_bwd_noalloc")
    return loss_out, dlogits


def _fused_call(entry: str, ws_bytes, hidden, w_lm, actions, behave_logp, adv, step_tok_off, traj_step_off,
                group_size, sched, prox_logp, norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total,
                dhidden, dw_lm, accumulate_dw, aux, workspace, loss_out, stream, extra=()):
    T, H, V = _hidden_w(hidden, w_lm, "w_lm")
    seg = _segments(step_tok_off, traj_step_off, group_size)
    _token_inputs(T, seg.n_traj, actions, behave_logp, prox_logp, adv)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    _meta(dhidden, "dhidden", torch.bfloat16, shape=(T, H), optional=True)
    _meta(dw_lm, "dw_lm", torch.float32, n=H * V, optional=True)
    _outputs_meta(T, seg.n_traj, aux, loss_out)
    dev = hidden.device
    _placed(dev, hidden=hidden, w_lm=w_lm, actions=actions, behave_logp=behave_logp, prox_logp=prox_logp, adv=adv,
            step_tok_off=step_tok_off, traj_step_off=traj_step_off, dhidden=dhidden, dw_lm=dw_lm)
    ca = aux._c(T, seg.n_traj, dev) if aux is not None else None
    if dhidden is None:
        dhidden = torch.empty_like(hidden)
    if dw_lm is None:
        dw_lm = torch.empty((H, V), dtype=torch.float32, device=dev)
    need = ws_bytes(T, H, V, sched, seg.n_traj)
    workspace = _workspace(workspace, need, dev)
    loss_out = _loss_out(loss_out, dev)
    st = getattr(_lib.load(), entry)(
        _ptr(hidden), _ptr(w_lm), T, H, V, int(sched), _ptr(actions), _ptr(behave_logp), _ptr(prox_logp), _ptr(adv),
        ctypes.byref(seg), ctypes.byref(par), _ptr(loss_out), _ptr(dhidden), _ptr(dw_lm), int(bool(accumulate_dw)),
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
    """As fused_lmhead_grpo, over blocks of `token_block` tokens whose logits are kept in the workspace between
    the forward and backward products, as fp16 terms exp(z - m) (three products instead of four).  With `aux_stream` (a second
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
    dt, T, ld = _logits2d(logits)
    Vv = logits.shape[1] if V is None else int(V)
    _meta(actions, "actions", torch.int32, n=T)
    _meta(error_flags, "error_flags", torch.int32, n=1, optional=True)
    _placed(logits.device, strided=("logits",), logits=logits, actions=actions, error_flags=error_flags)
    logp = torch.empty(T, dtype=torch.float32, device=logits.device)
    ent = torch.empty(T, dtype=torch.float32, device=logits.device) if entropy else None
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
    T, H, V = _hidden_w(hidden, w_lm, "w_lm")
    _meta(actions, "actions", torch.int32, n=T)
    _meta(error_flags, "error_flags", torch.int32, n=1, optional=True)
    dev = hidden.device
    _placed(dev, hidden=hidden, w_lm=w_lm, actions=actions, error_flags=error_flags)
    lib = _lib.load()
    need = int(lib.fused_lmhead_token_logp_workspace_bytes(T, H, V))
    workspace = _workspace(workspace, need, dev)
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    ent = torch.empty(T, dtype=torch.float32, device=dev) if entropy else None
    st = lib.fused_lmhead_token_logp(_ptr(hidden), _ptr(w_lm), T, H, V, _ptr(actions), _ptr(logp), _ptr(ent),
                                     _ptr(error_flags), _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "fused_lmhead_token_logp")
    return logp, ent


def vocab_stats_fields(stats: torch.Tensor):
    """Views of a uint8 [..., T, 24] record tensor as (m, z_a, s), each fp64 [..., T]."""
    f64 = stats.view(torch.float64)
    return f64[..., 0], f64[..., 2], f64[..., 1]


def grpo_vocab_shard_stats(logits: torch.Tensor, actions: torch.Tensor, v_begin: int, *, V: int | None = None,
                           stats: torch.Tensor | None = None, error_flags: torch.Tensor | None = None, stream=None):
    """Step 1 of the vocabulary-sharded loss: each row of the shard (global columns [v_begin, v_begin + V)) reduced
    to its record.  Returns uint8 [T, 24] records (read them with ``vocab_stats_fields``)."""
    dt, T, ld = _logits2d(logits)
    Vv = logits.shape[1] if V is None else int(V)
    _meta(actions, "actions", torch.int32, n=T)
    _meta(stats, "stats", torch.uint8, shape=(T, VOCAB_STATS_BYTES), optional=True)
    _meta(error_flags, "error_flags", torch.int32, n=1, optional=True)
    _placed(logits.device, strided=("logits",), logits=logits, actions=actions, stats=stats, error_flags=error_flags)
    if stats is None:
        stats = torch.empty((T, VOCAB_STATS_BYTES), dtype=torch.uint8, device=logits.device)
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
    _stats_all(stats_all, T)
    n_shards = stats_all.shape[0]
    seg = _segments(step_tok_off, traj_step_off, group_size)
    _token_inputs(T, seg.n_traj, actions, behave_logp, prox_logp, adv)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    dlogits = _dlogits_arg(dlogits, logits) if dlogits is not True else True
    _outputs_meta(T, seg.n_traj, aux, loss_out)
    dev = logits.device
    _placed(dev, strided=("logits", "dlogits"), logits=logits, dlogits=None if dlogits is True else dlogits,
            stats_all=stats_all, actions=actions, behave_logp=behave_logp, prox_logp=prox_logp, adv=adv,
            step_tok_off=step_tok_off, traj_step_off=traj_step_off)
    ca = aux._c(T, seg.n_traj, dev) if aux is not None else None
    need = grpo_loss_workspace_bytes(T, seg.n_traj)
    workspace = _workspace(workspace, need, dev)
    loss_out = _loss_out(loss_out, dev)
    dlogits = _dlogits_arg(dlogits, logits)
    st = _lib.load().grpo_loss_fwd_bwd_vocab_shard(
        _ptr(logits), dt, T, Vv, ld, int(v_begin), int(V_total), _ptr(stats_all), int(n_shards), _ptr(actions),
        _ptr(behave_logp), _ptr(prox_logp), _ptr(adv), ctypes.byref(seg), ctypes.byref(par), _ptr(loss_out),
        _ptr(dlogits), ctypes.byref(ca) if ca is not None else None, _ptr(workspace), _nbytes(workspace),
        _stream(stream))
    _check(st, "grpo_loss_fwd_bwd_vocab_shard")
    return loss_out, dlogits


def _stats_all(stats_all, T):
    _meta(stats_all, "stats_all", torch.uint8)
    if stats_all.dim() != 3 or tuple(stats_all.shape[1:]) != (T, VOCAB_STATS_BYTES):
        raise ValueError(f"stats_all must be uint8 [n_shards, T, {VOCAB_STATS_BYTES}]")


def vocab_shard_logits_buffer(T: int, V_shard: int, device) -> torch.Tensor:
    """An fp32 buffer for the shard's logits kept between the two steps of the sharded fused LM head."""
    n = int(_lib.load().fused_lmhead_vocab_shard_logits_bytes(int(T), int(V_shard))) // 4
    return torch.empty(max(n, 1), dtype=torch.float32, device=device)


def _check_logits_buffer(buf: torch.Tensor, T: int, V_shard: int, name: str):
    need = int(_lib.load().fused_lmhead_vocab_shard_logits_bytes(int(T), int(V_shard)))
    _meta(buf, name, torch.float32, n=(need + 3) // 4)


def fused_lmhead_vocab_shard_stats(hidden: torch.Tensor, w_shard: torch.Tensor, actions: torch.Tensor, v_begin: int,
                                   *, stats: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                                   logits_out: torch.Tensor | None = None, stream=None):
    """Step 1 of the vocabulary-sharded fused LM head: each row of h W_shard (W's columns [v_begin, v_begin +
    V_shard)) reduced to its record.  Returns uint8 [T, 24] records (read them with ``vocab_stats_fields``).
    ``logits_out`` (fp32, ``fused_lmhead_vocab_shard_logits_bytes(T, V_shard) / 4`` elements, see
    ``vocab_shard_logits_buffer``) also receives the shard's logits for step 2."""
    T, H, Vs = _hidden_w(hidden, w_shard, "w_shard")
    _meta(actions, "actions", torch.int32, n=T)
    _meta(stats, "stats", torch.uint8, shape=(T, VOCAB_STATS_BYTES), optional=True)
    if logits_out is not None:
        _check_logits_buffer(logits_out, T, Vs, "logits_out")
    dev = hidden.device
    _placed(dev, hidden=hidden, w_shard=w_shard, actions=actions, stats=stats, logits_out=logits_out)
    if stats is None:
        stats = torch.empty((T, VOCAB_STATS_BYTES), dtype=torch.uint8, device=dev)
    lib = _lib.load()
    need = lib.fused_lmhead_vocab_shard_stats_workspace_bytes(T, H, Vs)
    workspace = _workspace(workspace, need, dev)
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
    T, H, Vs = _hidden_w(hidden, w_shard, "w_shard")
    _stats_all(stats_all, T)
    seg = _segments(step_tok_off, traj_step_off, group_size)
    _token_inputs(T, seg.n_traj, actions, behave_logp, prox_logp, adv)
    par = _params(norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total)
    _meta(dhidden_partial, "dhidden_partial", torch.float32, shape=(T, H), optional=True)
    _meta(dw_shard, "dw_shard", torch.float32, n=H * Vs, optional=True)
    if logits_in is not None:
        _check_logits_buffer(logits_in, T, Vs, "logits_in")
        vocab_chunk = (Vs + 255) // 256 * 256  # the whole shard as one chunk
    _outputs_meta(T, seg.n_traj, aux, loss_out)
    dev = hidden.device
    _placed(dev, hidden=hidden, w_shard=w_shard, stats_all=stats_all, actions=actions, behave_logp=behave_logp,
            prox_logp=prox_logp, adv=adv, step_tok_off=step_tok_off, traj_step_off=traj_step_off,
            dhidden_partial=dhidden_partial, dw_shard=dw_shard, logits_in=logits_in)
    ca = aux._c(T, seg.n_traj, dev) if aux is not None else None
    if dhidden_partial is None:
        dhidden_partial = torch.empty((T, H), dtype=torch.float32, device=dev)
    if dw_shard is None:
        dw_shard = torch.empty((H, Vs), dtype=torch.float32, device=dev)
    need = fused_lmhead_workspace_bytes(T, H, Vs, vocab_chunk, seg.n_traj)
    workspace = _workspace(workspace, need, dev)
    loss_out = _loss_out(loss_out, dev)
    st = _lib.load().fused_lmhead_grpo_vocab_shard(
        _ptr(hidden), _ptr(w_shard), T, H, Vs, int(v_begin), int(V_total), int(vocab_chunk), _ptr(stats_all),
        int(stats_all.shape[0]), _ptr(actions), _ptr(behave_logp), _ptr(prox_logp), _ptr(adv), ctypes.byref(seg),
        ctypes.byref(par), _ptr(loss_out), _ptr(dhidden_partial), _ptr(dw_shard), int(bool(accumulate_dw)),
        ctypes.byref(ca) if ca is not None else None, _ptr(logits_in), _ptr(workspace), _nbytes(workspace),
        _stream(stream))
    _check(st, "fused_lmhead_grpo_vocab_shard")
    return loss_out, dhidden_partial, dw_shard


from .autograd import FusedLmHeadGrpoLoss, GrpoLoss  # noqa: E402  (needs the entry points above)
