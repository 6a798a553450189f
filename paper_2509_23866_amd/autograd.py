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
    loss.backward()          # hidden.grad, weight.grad (bfloat16)

Both take inv_temp (default 1, the paper's value): the policy is then
softmax(inv_temp z), as for dart_tok_stats_ex and dart_tis_grad_ex.

The LM-head backward writes its gradients in bfloat16 directly and, unless
told otherwise, forms the dlogits in the blocks of rows x vocabulary entries
that lmhead_backward_plan picks for a 512 MiB workspace.
"""

import torch

from . import (DART_LMHEAD_BF16_GRADS, dart_lmhead_backward_ex, dart_lmhead_tok_stats_ex,
               dart_select_tis_loss_fwd, dart_tis_grad, dart_tok_stats, lmhead_backward_plan)


def _scaled(coef, grad):
    """coef * grad for the scalar incoming gradient, on the device (exact when
    the gradient is 1)."""
    if grad.numel() != 1:
        raise ValueError("the DART loss is a scalar")
    return coef * grad.reshape(()).to(torch.float32)


def _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low, eps_high, C):
    _, _, _, loss, coef, _ = dart_select_tis_loss_fwd(ent, logp, logp_old, logp_rollout, adv,
                                                      step_offsets, rho, eps_low, eps_high, C,
                                                      with_stats=False)
    return loss.reshape(()), coef


class DartPolicyLoss(torch.autograd.Function):
    """Scalar DART loss (float64) of logits [T, V] (float32 or bfloat16)."""

    @staticmethod
    def forward(ctx, logits, target, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                eps_high, C, inv_temp):
        logits = logits.detach()
        logp, ent, lse = dart_tok_stats(logits, target, inv_temp=inv_temp)
        loss, coef = _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                           eps_high, C)
        ctx.inv_temp = inv_temp
        ctx.save_for_backward(logits, target, logp, lse, coef)
        return loss

    @staticmethod
    def backward(ctx, grad):
        logits, target, logp, lse, coef = ctx.saved_tensors
        dz = dart_tis_grad(logits, target, logp, lse, _scaled(coef, grad), inv_temp=ctx.inv_temp)
        return (dz,) + (None,) * 10


class DartLmHeadPolicyLoss(torch.autograd.Function):
    """Scalar DART loss (float64) of hidden [T, d] and weight [V, d] (bfloat16)
    through logits h W^T that are never written to memory."""

    @staticmethod
    def forward(ctx, hidden, weight, target, logp_old, logp_rollout, adv, step_offsets, rho,
                eps_low, eps_high, C, chunk_rows, chunk_cols, flags, inv_temp):
        hidden, weight = hidden.detach(), weight.detach()
        logp, ent, lse = dart_lmhead_tok_stats_ex(hidden, weight, target, inv_temp)
        loss, coef = _loss(logp, ent, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                           eps_high, C)
        ctx.plan = lmhead_grad_plan(hidden.shape[0], weight.shape[0], chunk_rows, chunk_cols,
                                    flags)
        ctx.inv_temp = inv_temp
        ctx.save_for_backward(hidden, weight, target, logp, lse, coef)
        return loss

    @staticmethod
    def backward(ctx, grad):
        hidden, weight, target, logp, lse, coef = ctx.saved_tensors
        rows, cols, flags = ctx.plan
        dh, dw = dart_lmhead_backward_ex(hidden, weight, target, lse, logp, _scaled(coef, grad),
                                         chunk_rows=rows, chunk_cols=cols, flags=flags,
                                         inv_temp=ctx.inv_temp)
        return (dh, dw) + (None,) * 13


def lmhead_grad_plan(T, V, chunk_rows=None, chunk_cols=None, flags=None):
    """(chunk_rows, chunk_cols, flags) the LM-head autograd backward passes to
    dart_lmhead_backward_ex: the caller's block, else lmhead_backward_plan's;
    the caller's flags (default none), always with bfloat16 gradients."""
    if chunk_rows is None and chunk_cols is None:
        chunk_rows, chunk_cols = lmhead_backward_plan(T, V)
    elif chunk_rows is None or chunk_cols is None:
        raise ValueError("give both chunk_rows and chunk_cols, or neither")
    return int(chunk_rows), int(chunk_cols), int(flags or 0) | DART_LMHEAD_BF16_GRADS


def dart_policy_loss(logits, target, logp_old, logp_rollout, adv, step_offsets, rho, eps_low,
                     eps_high, C, inv_temp=1.0):
    """Differentiable DART loss of the logits (see the module docstring)."""
    return DartPolicyLoss.apply(logits, target, logp_old, logp_rollout, adv, step_offsets, rho,
                                eps_low, eps_high, C, float(inv_temp))


def dart_lmhead_policy_loss(hidden, weight, target, logp_old, logp_rollout, adv, step_offsets,
                            rho, eps_low, eps_high, C, chunk_rows=None, chunk_cols=None,
                            flags=None, inv_temp=1.0):
    """Differentiable DART loss of the LM head's inputs (see the module
    docstring); chunk_rows, chunk_cols and flags as for dart_lmhead_backward_ex
    (no block: the default plan)."""
    return DartLmHeadPolicyLoss.apply(hidden, weight, target, logp_old, logp_rollout, adv,
                                      step_offsets, rho, eps_low, eps_high, C, chunk_rows,
                                      chunk_cols, flags, float(inv_temp))
