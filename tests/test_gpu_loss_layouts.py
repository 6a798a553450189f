"""GPU parity of the loss kernel alone on step layouts that reach every branch
of its token walk: steps of one token, more steps than the offsets and mask
kept in on-chip memory (8192), token counts that are not multiples of the
wave width, fewer tokens than lanes; and of the step selection on both sides
of its direct-rank and on-chip-key limits. Inputs are float32 on both sides;
the oracle computes in float64."""

import zlib

import numpy as np
import pytest

import oracle
from tests import _harness as H

pytestmark = pytest.mark.gpu


def _cuda(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _inputs(rng, lens, keep=0.5):
    T = int(np.sum(lens))
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    logp = (-rng.random(T) * 5.0).astype(np.float32)
    lp_old = (logp + rng.uniform(-0.4, 0.4, T)).astype(np.float32)
    lp_roll = (lp_old + rng.uniform(-3.0, 3.0, T)).astype(np.float32)
    lp_ref = (logp + rng.uniform(-0.5, 0.5, T)).astype(np.float32)
    adv = rng.choice([-1.0, 1.0, 0.5], T).astype(np.float32) * (rng.random(T) < 0.9)
    mask = (rng.random(len(lens)) < keep).astype(np.uint8)
    return dict(logp=logp, lp_old=lp_old, lp_roll=lp_roll, lp_ref=lp_ref,
                adv=adv.astype(np.float32), off=off, mask=mask)


LAYOUTS = [
    # (name, lens generator)
    ("single_token", lambda r: np.ones(1, np.int64)),
    ("under_one_wave", lambda r: r.integers(1, 6, 9)),
    ("ones_9000", lambda r: np.ones(9000, np.int64)),
    ("mixed_8192", lambda r: r.choice([1, 2, 3, 70], 8192)),
    ("mixed_8193", lambda r: r.choice([1, 2, 3, 70], 8193)),
    ("long_steps", lambda r: r.integers(500, 3000, 17)),
    ("ragged_20000", lambda r: r.choice([1, 7, 64, 65, 200], 20000)),
]


def _seed(*parts):
    return zlib.crc32(repr(parts).encode())


def _check(ref, loss, coef, stats, nstats, exact_zeros=False):
    ok = ~ref["boundary"]
    assert ref["boundary"].mean() <= 0.05
    L = ref["L"]
    assert abs(float(loss.cpu().item()) - L) <= H.LOSS_RTOL * max(abs(L), 1e-30)
    g = coef.cpu().numpy().astype(np.float64)
    floor = 1e-6 * max(np.abs(ref["g"]).max(), 1e-300)
    assert np.all((np.abs(g - ref["g"]) <= 1e-4 * np.abs(ref["g"]) + floor)[ok])
    if exact_zeros:
        # tokens of dropped steps, clipped tokens and zero advantages
        assert np.all(g[ref["g"] == 0.0] == 0.0)
    st = stats.cpu().numpy()
    assert st[3] == ref["stats"][3]
    if nstats == 6:
        assert st[5] == ref["stats"][5]


@pytest.mark.parametrize("ws", ["auto", None], ids=["workspace", "one_workgroup"])
@pytest.mark.parametrize("name", [n for n, _ in LAYOUTS])
def test_default_loss_on_layouts(name, ws):
    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(_seed(name))
    lens = dict(LAYOUTS)[name](rng)
    x = _inputs(rng, lens, keep=1.0 if len(lens) == 1 else 0.5)
    eps_low, eps_high, C = H.f32(0.2), H.f32(0.28), H.f32(2.0)
    ref = oracle.tis_loss(x["logp"].astype(np.float64), x["lp_old"], x["lp_roll"], x["adv"],
                          x["off"], x["mask"], eps_low, eps_high, C)
    loss, coef, stats = dart.dart_tis_loss_fwd(
        _cuda(x["logp"]), _cuda(x["lp_old"]), _cuda(x["lp_roll"]), _cuda(x["adv"]),
        _cuda(x["off"]), _cuda(x["mask"]), eps_low, eps_high, C, workspace=ws)
    _check(ref, loss, coef, stats, 4, exact_zeros=True)


@pytest.mark.parametrize("ws", ["auto", None], ids=["workspace", "one_workgroup"])
@pytest.mark.parametrize("name", ["ones_9000", "mixed_8193", "ragged_20000"])
@pytest.mark.parametrize("kl,agg,ratio", [("k3", "step_mean", "token"),
                                          ("k2", "token_mean_all", "token"),
                                          ("none", "step_mean", "step_geomean")])
def test_general_loss_on_layouts(name, kl, agg, ratio, ws):
    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(_seed(name, kl, agg, ratio))
    lens = dict(LAYOUTS)[name](rng)
    x = _inputs(rng, lens)
    eps_low, eps_high, C = H.f32(0.2), H.f32(0.28), H.f32(2.0)
    kw = dict(kl=kl, beta=0.05, agg=agg, ratio=ratio)
    ref = oracle.tis_loss_ex(x["logp"].astype(np.float64), x["lp_old"], x["lp_roll"], x["adv"],
                             x["off"], x["mask"], eps_low, eps_high, C, lp_ref=x["lp_ref"], **kw)
    loss, coef, stats = dart.dart_tis_loss_fwd_ex(
        _cuda(x["logp"]), _cuda(x["lp_old"]), _cuda(x["lp_roll"]), _cuda(x["adv"]),
        _cuda(x["off"]), _cuda(x["mask"]), eps_low, eps_high, C, logp_ref=_cuda(x["lp_ref"]),
        kl=kl, beta=0.05, aggregation=agg, ratio=ratio, workspace=ws)
    _check(ref, loss, coef, stats, 6)


@pytest.mark.parametrize("name", ["under_one_wave", "mixed_8193", "ragged_20000"])
def test_workspace_and_one_workgroup_agree(name):
    """The two launch shapes compute each coefficient by the same arithmetic
    (bit-identical) and differ only in the order the loss is summed."""
    import torch

    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(_seed(name, "paths"))
    x = _inputs(rng, dict(LAYOUTS)[name](rng))
    args = [_cuda(x[k]) for k in ("logp", "lp_old", "lp_roll", "adv", "off", "mask")]
    ws = torch.full((dart.dart_tis_loss_workspace_bytes(x["logp"].size),), 0xA5, dtype=torch.uint8,
                    device="cuda")  # contents on entry do not matter
    la, ca, sa = dart.dart_tis_loss_fwd(*args, 0.2, 0.28, 2.0, workspace=ws)
    lb, cb, sb = dart.dart_tis_loss_fwd(*args, 0.2, 0.28, 2.0, workspace=None)
    assert np.array_equal(ca.cpu().numpy().view(np.uint32), cb.cpu().numpy().view(np.uint32))
    assert sa[3].item() == sb[3].item()
    La, Lb = la.item(), lb.item()
    assert abs(La - Lb) <= 1e-12 * max(abs(La), 1e-300)


@pytest.mark.parametrize("S,rho", [(255, 0.5), (256, 0.3), (257, 0.3), (8192, 0.5),
                                   (8193, 0.5), (12000, 0.7)])
def test_step_select_on_limits(S, rho):
    """Exact step means and mask on both sides of the direct-rank limit (256
    steps) and of the on-chip key limit (8192 steps), with tied steps."""
    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(7 * S)
    lens = rng.choice([1, 2, 5], S)
    T = int(lens.sum())
    Hv = rng.choice([0.0, 0.5, 1.25, 3.0], T).astype(np.float32)
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    Hs, Hs32 = oracle.step_entropy(Hv.astype(np.float64), off)
    mask, k = oracle.step_mask(Hs32, rho)
    sh, m, nk = dart.dart_step_select(_cuda(Hv), _cuda(off), rho)
    assert np.array_equal(sh.cpu().numpy().view(np.uint32) & 0x7FFFFFFF,
                          Hs32.view(np.uint32) & 0x7FFFFFFF)
    assert np.array_equal(m.cpu().numpy(), mask) and int(nk.cpu().item()) == k
