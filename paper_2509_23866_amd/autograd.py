"""torch.autograd wrappers around the C ABI: the DART policy loss as a
differentiable function of the logits, or of the LM head's inputs.

The forward runs the first pass and the loss (token statistics, step
selection, TIS-weighted clipped loss, Sec. 4.3-4.4, Eq. 2); the backward runs
the second pass with the per-token coefficient scaled by the incoming
gradient, so the two-pass structure is kept: the logits (or h W^T) are read
once in each direction. Every step runs in the library's kernels; the wrappers
only marshal tensors and scale the [T] coefficient.

    loss = dart_policy_loss(logits, target, lp_old, lp_roll, adv, offsets, rho,
                            eps_low, eps_high, C)
    loss.backward()          # logits.grad = dL/dlogits

    loss = dart_lmhead_policy_loss(hidden, weight, target, lp_old, lp_roll, adv,
                                   offsets, rho, eps_low, eps_high, C)
    loss.backward()          # hidden.grad, weight.grad
"""

import torch

from . import (dart_lmhead_backward, dart_lmhead_tok_stats, dart_step_select, dart_tis_grad,
               dart_tis_loss_fwd, dart_tok_stats)


def _scaled(coef, grad):
    """coef * grad for the scalar incoming gradient, on the device (exact when
    the gradient is 1)."""
    if grad.numel() != 1:
        raise ValueError("the DART loss is a scalar")
    return coef * grad.reshape(()).to(torch.float32)


def _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low, eps_high, C):
    _, mask, _ = dart_step_select(ent, step_offsets, rho)
    loss, coef, _ = dart_tis_loss_fwd(logp, logp_old, logp_rollout, adv, step_offsets, mask,
                                      eps_low, eps_high, C, with_stats=False)
    return loss.reshape(()), coef


class DartPolicyLoss(torch.autograd.Function):
    """Scalar DART loss (float64) of logits [T, V] (float32 or bfloat16)."""

    @staticmethod
    def forward(ctx, logits, target, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                eps_high, C):
        logits = logits.detach()
        logp, ent, lse = dart_tok_stats(logits, target)
        loss, coef = _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                           eps_high, C)
        ctx.save_for_backward(logits, target, logp, lse, coef)
        return loss

    @staticmethod
    def backward(ctx, grad):
        logits, target, logp, lse, coef = ctx.saved_tensors
        dz = dart_tis_grad(logits, target, logp, lse, _scaled(coef, grad))
        return (dz,) + (None,) * 9


class DartLmHeadPolicyLoss(torch.autograd.Function):
    """Scalar DART loss (float64) of hidden [T, d] and weight [V, d] (bfloat16)
    through logits h W^T that are never written to memory."""

    @staticmethod
    def forward(ctx, hidden, weight, target, logp_old, logp_rollout, adv, step_offsets, rho,
                eps_low, eps_high, C, chunk_rows):
        hidden, weight = hidden.detach(), weight.detach()
        logp, ent, lse = dart_lmhead_tok_stats(hidden, weight, target)
        loss, coef = _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                           eps_high, C)
        ctx.chunk_rows = chunk_rows
        ctx.save_for_backward(hidden, weight, target, logp, lse, coef)
        return loss

    @staticmethod
    def backward(ctx, grad):
        hidden, weight, target, logp, lse, coef = ctx.saved_tensors
        dh, dw = dart_lmhead_backward(hidden, weight, target, lse, logp, _scaled(coef, grad),
                                      chunk_rows=ctx.chunk_rows)
        return (dh.to(hidden.dtype), dw.to(weight.dtype)) + (None,) * 10


def dart_policy_loss(logits, target, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                     eps_high, C):
    """Differentiable DART loss of the logits (see the module docstring)."""
    return DartPolicyLoss.apply(logits, target, logp_old, logp_rollout, adv, step_offsets, rho,
                                eps_low, eps_high, C)


def dart_lmhead_policy_loss(hidden, weight, target, logp_old, logp_rollout, adv, step_offsets,
                            rho, eps_low, eps_high, C, chunk_rows=1024):
    """Differentiable DART loss of the LM head's inputs (see the module
    docstring); the backward forms dlogits chunk_rows rows at a time."""
    return DartLmHeadPolicyLoss.apply(hidden, weight, target, logp_old, logp_rollout, adv,
                                      step_offsets, rho, eps_low, eps_high, C, chunk_rows)
