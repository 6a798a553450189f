"""GPU parity of the objective variants (KL term of Eq. 2 with each estimator,
aggregation weights, step-level ratios, inverse temperature) and of the
zero-row read skipping of the gradient pass, through the C ABI, against the
float64 oracle. Same tolerances as the base path."""

import itertools

import numpy as np
import pytest

import oracle
import synth
import synth.native as sn
from tests import _harness as H

pytestmark = pytest.mark.gpu

CASES = list(itertools.product(["k1", "k2", "k3", "none"], ["token_mean", "token_mean_all", "step_mean"],
                               ["token", "step_geomean", "step_product"]))


def _setup(lens, V, dtype, seed, inv_temp, **kw):
    import torch

    wl = synth.custom_workload(lens=lens, V=V, dtype=dtype, seed=seed, **kw)
    z = sn.logits_rows_host(wl, np.arange(wl.T))
    logp, Hh, lse = oracle.token_stats(z, wl.target, inv_temp=inv_temp)
    lp_old, lp_roll = synth.perturbed_logprobs(wl, logp)
    lp_ref = synth.reference_logprobs(wl, logp)
    Hs, Hs32 = oracle.step_entropy(Hh, wl.off)
    mask, k = oracle.step_mask(Hs32, wl.rho)
    dev = torch.device("cuda")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    logits = torch.empty((wl.T, wl.V), dtype=tdt, device=dev)
    sn.fill_logits_device(sn.DeviceRecipe(wl), logits)
    cuda = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    gpu = dict(logits=logits, target=cuda(wl.target), lp_old=cuda(lp_old), lp_roll=cuda(lp_roll),
               lp_ref=cuda(lp_ref), adv=cuda(wl.adv), off=cuda(wl.off), mask=cuda(mask))
    host = dict(z=z, logp=logp, H=Hh, lse=lse, lp_old=lp_old, lp_roll=lp_roll, lp_ref=lp_ref,
                mask=mask)
    return wl, host, gpu


@pytest.mark.parametrize("case", range(len(CASES)))
def test_objective_variant(case):
    """(1) The loss kernel alone, fed the oracle's log-probs rounded to float32
    on both sides: loss 1e-4 relative, coefficients 1e-4 relative. (2) The whole
    chain from the GPU's own log-probs: token statistics at 2e-4; the loss and
    coefficients within 1e-4 relative plus the first-order propagation of the
    measured log-prob differences (through the ratio, summed over the step for
    step ratios, and through the KL derivative). (3) The gradient kernel alone,
    fed the oracle's coefficients: within 1 bf16 ulp everywhere."""
    import torch

    import paper_2509_23866_amd as dart

    kl, agg, ratio = CASES[case]
    inv_temp = [1.0, 0.75, 1.5][case % 3]
    lens = [5, 1, 9, 3, 70, 2]
    wl, host, g = _setup(lens, 8192 + 13, "bf16", 300 + case, inv_temp, rho=0.67, mix_kinds=case % 2 == 0,
                         ratio_spread=case % 4 == 1)
    eps_low, eps_high, C = H.f32(wl.eps_low), H.f32(wl.eps_high), H.f32(wl.C)
    beta = 0.1
    kw = dict(kl=kl, beta=beta, agg=agg, ratio=ratio)

    # (1) identical inputs
    lp32 = host["logp"].astype(np.float32)
    ref1 = oracle.tis_loss_ex(lp32.astype(np.float64), host["lp_old"], host["lp_roll"], wl.adv,
                              wl.off, host["mask"], eps_low, eps_high, C, lp_ref=host["lp_ref"], **kw)
    loss1, coef1, stats1 = dart.dart_tis_loss_fwd_ex(
        torch.from_numpy(lp32).cuda(), g["lp_old"], g["lp_roll"], g["adv"], g["off"], g["mask"],
        eps_low, eps_high, C, logp_ref=g["lp_ref"], kl=kl, beta=beta, aggregation=agg, ratio=ratio)
    torch.cuda.synchronize()
    ok1 = ~ref1["boundary"]
    assert ref1["boundary"].mean() <= 0.05
    assert abs(float(loss1.cpu().item()) - ref1["L"]) <= H.LOSS_RTOL * max(abs(ref1["L"]), 1e-30)
    g1 = coef1.cpu().numpy()
    floor = 1e-6 * np.abs(ref1["g"]).max()  # coefficients where the KL and policy terms cancel
    assert np.all(np.abs(g1 - ref1["g"])[ok1] <= 1e-4 * np.abs(ref1["g"][ok1]) + floor)
    st = stats1.cpu().numpy()
    N = ref1["stats"][3]
    assert st[3] == N and st[5] == ref1["stats"][5]
    if N > 0:
        assert abs(st[4] - ref1["stats"][4]) <= 1e-4 * max(1e-3, abs(ref1["stats"][4]))
        assert abs(st[1] - ref1["stats"][1]) <= 1e-5 * max(1.0, ref1["stats"][1])

    # (2) the chain from the GPU's own log-probs
    ref = oracle.tis_loss_ex(host["logp"], host["lp_old"], host["lp_roll"], wl.adv, wl.off,
                             host["mask"], eps_low, eps_high, C, lp_ref=host["lp_ref"], **kw)
    logp, ent, lse = dart.dart_tok_stats(g["logits"], g["target"], inv_temp=inv_temp)
    loss, coef, _ = dart.dart_tis_loss_fwd_ex(
        logp, g["lp_old"], g["lp_roll"], g["adv"], g["off"], g["mask"], eps_low, eps_high, C,
        logp_ref=g["lp_ref"], kl=kl, beta=beta, aggregation=agg, ratio=ratio)
    torch.cuda.synchronize()
    lp_gpu = logp.cpu().numpy()
    assert np.abs(lp_gpu - host["logp"]).max() <= H.LOGP_TOL
    assert np.abs(ent.cpu().numpy() - host["H"]).max() <= H.H_TOL
    d_lp = np.abs(lp_gpu.astype(np.float64) - host["logp"])
    step = wl.step_of_token()
    spread = d_lp if ratio == "token" else np.bincount(step, weights=d_lp, minlength=wl.S)[step]
    # first-order sensitivity of each coefficient to the log-prob differences:
    # through the ratio (relative, summed over the step for step ratios) and
    # through the KL derivative (om_t beta e^delta |d logp_t|)
    lens = np.diff(wl.off.astype(np.int64))[step]
    kept = host["mask"][step] == 1
    N, K = kept.sum(), host["mask"].sum()
    om = {"token_mean": 1.0 / max(N, 1), "token_mean_all": 1.0 / wl.T}.get(agg)
    om = np.full(wl.T, om) if om is not None else 1.0 / (max(K, 1) * lens)
    delta = host["lp_ref"].astype(np.float64) - host["logp"]
    kl_sens = om * beta * np.exp(np.minimum(delta, 50)) * d_lp if kl != "none" else 0.0
    ok = ~ref["boundary"]
    L_tol = H.LOSS_RTOL * abs(ref["L"]) + 2.0 * float(np.sum(np.abs(ref["g"]) * spread)) \
        + 2.0 * float(np.sum(kl_sens))
    assert abs(float(loss.cpu().item()) - ref["L"]) <= L_tol
    gg = coef.cpu().numpy()
    g_tol = (1e-4 + 2 * spread) * np.abs(ref["g"]) + 2 * kl_sens + floor
    assert np.all((np.abs(gg - ref["g"]) <= g_tol)[ok])

    # (3) the gradient kernel alone, fed the oracle's coefficients (float32)
    g32 = torch.from_numpy(ref["g"].astype(np.float32)).cuda()
    dz = dart.dart_tis_grad(g["logits"], g["target"], logp, lse, g32, inv_temp=inv_temp)
    torch.cuda.synchronize()
    dz_ref = oracle.dlogits(host["z"], wl.target, host["lse"], host["logp"],
                            ref["g"].astype(np.float32).astype(np.float64), inv_temp=inv_temp)
    bits = dz.view(torch.int16).cpu().numpy().view(np.uint16)
    H.check_dz(bits, dz_ref, "bf16")


@pytest.mark.parametrize("dtype,inplace", [("bf16", False), ("bf16", True), ("f32", False)])
def test_skip_zero_rows_same_gradient(dtype, inplace):
    """DART_GRAD_SKIP_ZERO_ROWS gives the same gradient (+0 for -0) and zero
    rows where the coefficient is zero (dropped steps)."""
    import torch

    import paper_2509_23866_amd as dart

    wl, host, g = _setup([7, 40, 3, 16, 9], 20000 + 3, dtype, 77, 1.0, rho=0.4)
    logp, ent, lse = dart.dart_tok_stats(g["logits"], g["target"])
    loss, dz_full, coef, _ = dart.dart_tis_loss_fwd_bwd(
        g["logits"], g["target"], logp, lse, g["lp_old"], g["lp_roll"], g["adv"], g["off"],
        g["mask"], wl.eps_low, wl.eps_high, wl.C)
    full = dz_full.float().cpu().numpy()
    src = g["logits"]
    out = src if inplace else None
    dz = dart.dart_tis_grad(src, g["target"], logp, lse, coef, dlogits=out, skip_zero_rows=True)
    torch.cuda.synchronize()
    got = dz.float().cpu().numpy()
    assert np.array_equal(got, full)  # float compare: +0 == -0
    zero_rows = coef.cpu().numpy() == 0
    assert zero_rows.sum() > 0 and np.all(got[zero_rows] == 0)
