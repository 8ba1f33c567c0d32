"""torch.autograd wrappers of the loss entry points, for training loops that call ``loss.backward()``.

Each forward runs one library call that produces the loss and its gradients together (the GRPO loss of Eq. 1,
dual clip of Eq. 2), saves the gradients, and returns the loss as a 0-dim fp64 tensor; backward hands the saved
gradients back.  Behaviour and advantages are constants (no gradient), as in the paper's objective.

Neither direction synchronises with the host.  How backward treats the incoming gradient g of the loss is the
``upstream`` option:
  "scale" (default)  the saved gradients times g, on the device (an elementwise pass over them; exact when g is
                     1 or a power of two);
  "unit"             the saved gradients as the library wrote them: the caller guarantees g = 1 (``loss.backward()``
                     on this loss, or on a sum it enters with weight 1) and folds any known factor into the forward's
                     ``grad_scale``.  No extra pass: the right mode for the logits path, whose gradient is as large
                     as the logits.
"""
from __future__ import annotations

import torch

from . import fused_lmhead_grpo, fused_lmhead_grpo_blocked, grpo_loss_fwd_bwd

_UPSTREAM = ("scale", "unit")


def _upstream(opts):
    mode = opts.pop("upstream", "scale")
    if mode not in _UPSTREAM:
        raise ValueError(f"upstream must be one of {_UPSTREAM}, got {mode!r}")
    return mode


def _apply_upstream(mode, grads, grad_output):
    if mode == "unit":
        return grads
    return tuple(None if t is None else torch.mul(t, grad_output.to(t.dtype)) for t in grads)


class GrpoLoss(torch.autograd.Function):
    """``loss = GrpoLoss.apply(logits, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, opts)``

    logits [T, V] (bf16 or fp32, on the GPU); ``opts`` is a dict of the keyword options of ``grpo_loss_fwd_bwd``
    (prox_logp, norm, k, eps_low, eps_high, dual_clip_c, grad_scale, n_groups_total, aux, stream) plus
    ``upstream`` (above).  dlogits are formed in the same pass over the logits as the loss when ``logits``
    requires grad.
    """

    @staticmethod
    def forward(ctx, logits, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, opts=None):
        opts = dict(opts or {})
        ctx.upstream = _upstream(opts)
        want = bool(ctx.needs_input_grad[0])
        loss, dlogits = grpo_loss_fwd_bwd(logits.detach(), actions, behave_logp, adv, step_tok_off, traj_step_off,
                                          group_size, dlogits=want, **opts)
        ctx.save_for_backward(dlogits if want else None)
        return loss.view(())

    @staticmethod
    def backward(ctx, grad_output):
        (dlogits,) = ctx.saved_tensors
        (dlogits,) = _apply_upstream(ctx.upstream, (dlogits,), grad_output)
        return dlogits, None, None, None, None, None, None, None


class FusedLmHeadGrpoLoss(torch.autograd.Function):
    """``loss = FusedLmHeadGrpoLoss.apply(hidden, w_lm, actions, behave_logp, adv, step_tok_off, traj_step_off,
    group_size, opts)``

    hidden [T, H] and w_lm [H, V], bf16 on the GPU.  ``opts``: the keyword options of ``fused_lmhead_grpo_blocked``
    (token_block, aux_stream, ...), or with ``schedule="chunked"`` those of ``fused_lmhead_grpo`` (vocab_chunk, ...),
    plus ``upstream`` (above).  dhidden and dW come from the same call as the loss.  The library's dW is fp32;
    autograd needs the gradient in w_lm's dtype, so it is rounded to bf16 here (call the entry point directly to
    keep the fp32 dW).
    """

    @staticmethod
    def forward(ctx, hidden, w_lm, actions, behave_logp, adv, step_tok_off, traj_step_off, group_size, opts=None):
        opts = dict(opts or {})
        ctx.upstream = _upstream(opts)
        entry = fused_lmhead_grpo if opts.pop("schedule", "blocked") == "chunked" else fused_lmhead_grpo_blocked
        loss, dhidden, dw = entry(hidden.detach(), w_lm.detach(), actions, behave_logp, adv, step_tok_off,
                                  traj_step_off, group_size, **opts)
        ctx.save_for_backward(dhidden, dw)
        ctx.w_dtype = w_lm.dtype
        return loss.view(())

    @staticmethod
    def backward(ctx, grad_output):
        dhidden, dw = ctx.saved_tensors
        dhidden, dw = _apply_upstream(ctx.upstream, (dhidden, dw), grad_output)
        dh = dhidden if ctx.needs_input_grad[0] else None
        dW = dw.to(ctx.w_dtype) if ctx.needs_input_grad[1] else None
        return dh, dW, None, None, None, None, None, None, None
