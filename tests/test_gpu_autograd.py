"""The autograd wrappers run the same kernels as the direct calls: the loss
and the gradients they produce are bit-identical to those of the C-ABI
entry points called in sequence, and an incoming gradient scales the
per-token coefficient."""

import math

import numpy as np
import pytest

import synth
import synth.native as sn
from synth.gen import STREAM_HIDDEN, STREAM_WEIGHT

pytestmark = pytest.mark.gpu


def _cuda(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _workload(T=700, V=3000, S=12, seed=3):
    import torch

    rng = np.random.default_rng(seed)
    lens = np.full(S, T // S)
    lens[: T - lens.sum()] += 1
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    target = rng.integers(0, V, T).astype(np.int32)
    logits = torch.from_numpy(rng.normal(0, 3, (T, V)).astype(np.float32)).cuda().to(torch.bfloat16)
    adv = rng.choice([-1.0, 1.0], S)[np.repeat(np.arange(S), lens)].astype(np.float32)
    return logits, _cuda(target), _cuda(off), _cuda(adv), rng


def test_policy_loss_autograd_matches_direct():
    import torch

    import paper_2509_23866_amd as dart
    from paper_2509_23866_amd.autograd import dart_policy_loss

    logits, target, off, adv, rng = _workload()
    logp, _, _ = dart.dart_tok_stats(logits, target)
    lp_old = logp + _cuda(rng.normal(0, 0.05, logp.numel()).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, logp.numel()).astype(np.float32))
    ref = dart.policy_update(logits, target, lp_old, lp_roll, adv, off, 0.8, 0.2, 0.28, 2.0)
    x = logits.clone().requires_grad_(True)
    loss = dart_policy_loss(x, target, lp_old, lp_roll, adv, off, 0.8, 0.2, 0.28, 2.0)
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == ref["loss"].item()
    assert torch.equal(x.grad.view(torch.int16), ref["dlogits"].view(torch.int16))

    # an incoming gradient of 2.5 scales the coefficient before the second pass
    x.grad = None
    loss = dart_policy_loss(x, target, lp_old, lp_roll, adv, off, 0.8, 0.2, 0.28, 2.0)
    (2.5 * loss).backward()
    logp2, _, lse2 = dart.dart_tok_stats(logits, target)
    dz = dart.dart_tis_grad(logits, target, logp2, lse2, ref["tok_coef"] * 2.5)
    torch.cuda.synchronize()
    assert torch.equal(x.grad.view(torch.int16), dz.view(torch.int16))


@pytest.mark.parametrize("rows,cols,flags", [(None, None, None), (256, 5000, 0), (600, 1000, 0),
                                             (256, 1000, 0), (300, 5000, 1)])
def test_lmhead_policy_loss_autograd_matches_direct(rows, cols, flags):
    """The autograd gradients are the bits of the direct bf16-gradient call
    with the same blocking (the default plan: one block here; row chunks,
    vocabulary chunks, both, rows skipped); with row chunks over the whole
    vocabulary, dweight is the fp32 sum rounded once, so it equals the fp32
    call's dweight rounded to bf16."""
    import torch

    import paper_2509_23866_amd as dart
    from paper_2509_23866_amd.autograd import dart_lmhead_policy_loss, lmhead_grad_plan

    T, d, V, S = 600, 256, 5000, 10
    rng = np.random.default_rng(9)
    h = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    w = torch.empty((V, d), dtype=torch.bfloat16, device="cuda")
    sn.fill_gaussian_device(h, 9, STREAM_HIDDEN, 1.0)
    sn.fill_gaussian_device(w, 9, STREAM_WEIGHT, 3.0 / math.sqrt(d))
    y = _cuda(rng.integers(0, V, T).astype(np.int32))
    off = _cuda(np.linspace(0, T, S + 1).astype(np.int32))
    adv = _cuda(rng.normal(0, 1, T).astype(np.float32))
    logp, ent, lse = dart.dart_lmhead_tok_stats(h, w, y)
    lp_old = logp + _cuda(rng.normal(0, 0.05, T).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, T).astype(np.float32))
    # direct sequence
    _, mask, _ = dart.dart_step_select(ent, off, 0.7)
    loss_ref, coef, _ = dart.dart_tis_loss_fwd(logp, lp_old, lp_roll, adv, off, mask, 0.2, 0.28,
                                               2.0)
    r, c, f = lmhead_grad_plan(T, V, rows, cols, flags)
    assert f & dart.DART_LMHEAD_BF16_GRADS
    dh_ref, dw_ref = dart.dart_lmhead_backward_ex(h, w, y, lse, logp, coef, chunk_rows=r,
                                                  chunk_cols=c, flags=f)
    # autograd
    hx = h.clone().requires_grad_(True)
    wx = w.clone().requires_grad_(True)
    loss = dart_lmhead_policy_loss(hx, wx, y, lp_old, lp_roll, adv, off, 0.7, 0.2, 0.28, 2.0,
                                   chunk_rows=rows, chunk_cols=cols, flags=flags)
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == loss_ref.item()
    assert hx.grad.dtype == torch.bfloat16 and wx.grad.dtype == torch.bfloat16
    assert torch.equal(hx.grad.view(torch.int16), dh_ref.view(torch.int16))
    assert torch.equal(wx.grad.view(torch.int16), dw_ref.view(torch.int16))
    if (rows, cols, flags) == (256, 5000, 0):
        _, dw32 = dart.dart_lmhead_backward(h, w, y, lse, logp, coef, chunk_rows=256)
        torch.cuda.synchronize()
        assert torch.equal(wx.grad.view(torch.int16), dw32.to(torch.bfloat16).view(torch.int16))


def test_autograd_inverse_temperature_matches_direct():
    """At an inverse temperature both wrappers give the bits of the direct
    calls at that temperature (whose parity with the oracle is tested on its
    own): the loss and the gradient of the logits, and the loss and the bf16
    gradients of the LM head's inputs."""
    import torch

    import paper_2509_23866_amd as dart
    from paper_2509_23866_amd.autograd import (dart_lmhead_policy_loss, dart_policy_loss,
                                               lmhead_grad_plan)

    it = 1.4
    logits, target, off, adv, rng = _workload()
    logp, ent, lse = dart.dart_tok_stats(logits, target, inv_temp=it)
    lp_old = logp + _cuda(rng.normal(0, 0.05, logp.numel()).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, logp.numel()).astype(np.float32))
    _, mask, _ = dart.dart_step_select(ent, off, 0.8)
    loss_ref, coef, _ = dart.dart_tis_loss_fwd(logp, lp_old, lp_roll, adv, off, mask, 0.2, 0.28,
                                               2.0)
    dz_ref = dart.dart_tis_grad(logits, target, logp, lse, coef, inv_temp=it)
    x = logits.clone().requires_grad_(True)
    loss = dart_policy_loss(x, target, lp_old, lp_roll, adv, off, 0.8, 0.2, 0.28, 2.0, inv_temp=it)
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == loss_ref.item()
    assert torch.equal(x.grad.view(torch.int16), dz_ref.view(torch.int16))

    T, d, V, S = 600, 256, 5000, 10
    h = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    w = torch.empty((V, d), dtype=torch.bfloat16, device="cuda")
    sn.fill_gaussian_device(h, 11, STREAM_HIDDEN, 1.0)
    sn.fill_gaussian_device(w, 11, STREAM_WEIGHT, 3.0 / math.sqrt(d))
    y = _cuda(rng.integers(0, V, T).astype(np.int32))
    off = _cuda(np.linspace(0, T, S + 1).astype(np.int32))
    adv = _cuda(rng.normal(0, 1, T).astype(np.float32))
    logp, ent, lse = dart.dart_lmhead_tok_stats_ex(h, w, y, it)
    lp_old = logp + _cuda(rng.normal(0, 0.05, T).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, T).astype(np.float32))
    _, mask, _ = dart.dart_step_select(ent, off, 0.7)
    loss_ref, coef, _ = dart.dart_tis_loss_fwd(logp, lp_old, lp_roll, adv, off, mask, 0.2, 0.28,
                                               2.0)
    r, c, f = lmhead_grad_plan(T, V)
    dh_ref, dw_ref = dart.dart_lmhead_backward_ex(h, w, y, lse, logp, coef, chunk_rows=r,
                                                  chunk_cols=c, flags=f, inv_temp=it)
    hx = h.clone().requires_grad_(True)
    wx = w.clone().requires_grad_(True)
    loss = dart_lmhead_policy_loss(hx, wx, y, lp_old, lp_roll, adv, off, 0.7, 0.2, 0.28, 2.0,
                                   inv_temp=it)
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == loss_ref.item()
    assert torch.equal(hx.grad.view(torch.int16), dh_ref.view(torch.int16))
    assert torch.equal(wx.grad.view(torch.int16), dw_ref.view(torch.int16))
