"""GPU parity of the fused selection and loss call (dart_select_tis_loss_fwd:
the step means and top-rho selection of Sec. 4.3, then the coefficients and
loss of Eq. (2)). On every layout it gives what dart_step_select followed by
dart_tis_loss_fwd gives: the step means, mask, kept count and coefficients bit
for bit; the loss bit for bit against the one-workgroup loss and within 1e-12
of the many-workgroup one; and it matches the oracle's selection (exactly, on
the same float32 entropies) and loss. The layouts reach both sides of the
one-workgroup limits (4096 tokens, 8192 steps) and of the selection's
direct-rank limit (256 steps), ties between step means, rho 0 and 1, and
steps of one token."""

import zlib

import numpy as np
import pytest

import oracle
from tests import _harness as H

pytestmark = pytest.mark.gpu

EPS_LOW, EPS_HIGH, C = 0.2, 0.28, 2.0


def _cuda(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _inputs(rng, lens, tie_frac=0.3):
    """Token entropies with exact ties between whole steps (copied steps),
    repeated values and signed zeros; log-probs and advantages of the loss."""
    T = int(np.sum(lens))
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    ent = rng.choice([0.0, -0.0, 0.5, 1.25, 3.0], T).astype(np.float32) + \
        ((rng.random(T) < 0.5) * rng.random(T)).astype(np.float32)
    for s in range(1, len(lens)):
        if rng.random() < tie_frac and lens[s] == lens[s - 1]:
            ent[off[s]:off[s + 1]] = ent[off[s - 1]:off[s]]
    logp = (-rng.random(T) * 5.0).astype(np.float32)
    lp_old = (logp + rng.uniform(-0.4, 0.4, T)).astype(np.float32)
    lp_roll = (lp_old + rng.uniform(-3.0, 3.0, T)).astype(np.float32)
    adv = (rng.choice([-1.0, 1.0, 0.5], T) * (rng.random(T) < 0.9)).astype(np.float32)
    return dict(ent=ent.astype(np.float32), logp=logp, lp_old=lp_old, lp_roll=lp_roll, adv=adv,
                off=off)


CASES = [
    # (name, step lengths, rho); T <= 4096 and S <= 8192 run in one workgroup
    ("one_token", lambda r: np.ones(1, np.int64), 0.5),
    ("vlm7b_steps", lambda r: r.integers(16, 33, 64), 0.8),
    ("rank_limit_256", lambda r: r.integers(1, 17, 256), 0.5),
    ("radix_257", lambda r: r.integers(1, 16, 257), 0.5),
    ("rho_zero", lambda r: r.integers(1, 40, 37), 0.0),
    ("rho_one", lambda r: r.integers(1, 40, 37), 1.0),
    ("max_tokens", lambda r: np.r_[np.full(63, 64, np.int64), [4096 - 63 * 64]], 0.8),
    ("steps_of_one_4096", lambda r: np.ones(4096, np.int64), 0.8),
    # past the limits: the two calls in turn
    ("tokens_4097", lambda r: np.r_[np.full(63, 64, np.int64), [4097 - 63 * 64]], 0.8),
    ("vlm7b_4600", lambda r: r.integers(16, 129, 64), 0.8),
    ("steps_8193", lambda r: np.ones(8193, np.int64), 0.3),
    ("microbatch_steps", lambda r: r.integers(64, 129, 128), 0.8),
]


@pytest.mark.parametrize("ws", ["auto", None])
@pytest.mark.parametrize("name,gen,rho", CASES, ids=[c[0] for c in CASES])
def test_fused_equals_the_two_calls_and_the_oracle(name, gen, rho, ws):
    import torch

    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(zlib.crc32(name.encode()))
    lens = gen(rng)
    x = _inputs(rng, lens)
    T, S = int(lens.sum()), len(lens)
    H.log(f"select+loss: {name} T={T} S={S} rho={rho} workspace={ws}")
    d = {k: _cuda(v) for k, v in x.items()}
    sh, mask, nk, loss, coef, st = dart.dart_select_tis_loss_fwd(
        d["ent"], d["logp"], d["lp_old"], d["lp_roll"], d["adv"], d["off"], rho, EPS_LOW,
        EPS_HIGH, C, workspace=ws)
    sh2, mask2, nk2 = dart.dart_step_select(d["ent"], d["off"], rho)
    loss2, coef2, st2 = dart.dart_tis_loss_fwd(d["logp"], d["lp_old"], d["lp_roll"], d["adv"],
                                               d["off"], mask2, EPS_LOW, EPS_HIGH, C,
                                               workspace=ws)
    torch.cuda.synchronize()
    bits = lambda t: t.cpu().numpy().view(np.uint8)  # noqa: E731
    assert np.array_equal(bits(sh), bits(sh2))
    assert np.array_equal(bits(mask), bits(mask2))
    assert int(nk.item()) == int(nk2.item())
    assert np.array_equal(bits(coef), bits(coef2))
    one_wg = T <= 4096 and S <= 8192
    if ws is None or not one_wg or T <= 2048:
        # the same summation order on both sides
        assert np.array_equal(bits(loss), bits(loss2)) and np.array_equal(bits(st), bits(st2))
    else:
        L, L2 = float(loss.item()), float(loss2.item())
        assert abs(L - L2) <= 1e-12 * max(abs(L2), 1e-300)
        assert np.array_equal(bits(st[3:]), bits(st2[3:]))  # N is a count
        assert np.allclose(st.cpu().numpy(), st2.cpu().numpy(), rtol=1e-6, atol=0)

    # the oracle, on the same float32 entropies
    Hs, Hs32 = oracle.step_entropy(x["ent"].astype(np.float64), x["off"])
    mask_o, k = oracle.step_mask(Hs32, rho)
    gsh = sh.cpu().numpy()
    assert np.array_equal(gsh.view(np.uint32) & 0x7FFFFFFF, Hs32.view(np.uint32) & 0x7FFFFFFF)
    assert np.array_equal(mask.cpu().numpy(), mask_o) and int(nk.item()) == k
    res = oracle.tis_loss(x["logp"], x["lp_old"], x["lp_roll"], x["adv"], x["off"], mask_o,
                          EPS_LOW, EPS_HIGH, C)
    gpu = dict(L=float(loss.item()), g=coef.cpu().numpy().astype(np.float64),
               stats=st.cpu().numpy().astype(np.float64))
    H.check_loss(gpu, res, res["boundary"])
    if k == 0:
        assert float(loss.item()) == 0.0 and not coef.any().item()


def test_fused_call_overwrites_stale_outputs():
    """Every output is written: buffers holding NaN and ones beforehand end
    with the values of a fresh call (n_kept optional, stats optional)."""
    import torch

    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(3)
    lens = rng.integers(16, 129, 64)
    x = _inputs(rng, lens)
    d = {k: _cuda(v) for k, v in x.items()}
    T, S = int(lens.sum()), len(lens)
    ref = dart.dart_select_tis_loss_fwd(d["ent"], d["logp"], d["lp_old"], d["lp_roll"], d["adv"],
                                        d["off"], 0.8, EPS_LOW, EPS_HIGH, C)
    nan = lambda n: torch.full((n,), float("nan"), device="cuda")  # noqa: E731
    sh, coef = nan(S), nan(T)
    mask = torch.full((S,), 7, dtype=torch.uint8, device="cuda")
    loss = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
    out = dart.dart_select_tis_loss_fwd(d["ent"], d["logp"], d["lp_old"], d["lp_roll"], d["adv"],
                                        d["off"], 0.8, EPS_LOW, EPS_HIGH, C, step_entropy=sh,
                                        step_mask=mask, loss=loss, tok_coef=coef,
                                        with_stats=False)
    torch.cuda.synchronize()
    assert out[5] is None
    for i in (0, 1, 3, 4):
        assert torch.equal(out[i].view(torch.uint8), ref[i].view(torch.uint8)), i
