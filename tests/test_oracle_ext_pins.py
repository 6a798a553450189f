"""Pins of the oracle's objective variants: the KL term of Eq. (2) with
selectable estimator, the aggregation weights, the step-level ratio (Eq. 1
written for the whole action) and an inverse sampling temperature."""

import math

import numpy as np
import pytest
import scipy.special

import oracle
from oracle import mini

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ----------------------------------------------------------------- temperature

@pytest.mark.parametrize("it", [0.5, 2.0, 4.0])
def test_temperature_is_a_logit_scale(it):
    """softmax(it * z) at temperature 1/it equals the statistics of the
    (exactly) scaled logits it * z at temperature 1 (powers of two scale
    float32 exactly)."""
    rng = np.random.default_rng(1)
    z = rng.normal(0, 3, (5, 301)).astype(np.float32)
    y = rng.integers(0, 301, 5).astype(np.int32)
    a = oracle.token_stats(z, y, inv_temp=it)
    b = oracle.token_stats((z * np.float32(it)).astype(np.float32), y)
    for u, v in zip(a, b):
        assert np.allclose(u, v, rtol=1e-13, atol=1e-12)


def test_temperature_two_level_closed_form():
    """Spike Delta at inverse temperature it: the two-level closed form with
    Delta * it."""
    V, delta, it = 777, 4.0, 0.75
    z = np.zeros((1, V), np.float32)
    z[0, 5] = delta
    logp, H, _ = oracle.token_stats(z, [5], inv_temp=it)
    d = delta * it
    a = (V - 1) * math.exp(-d)
    assert abs(H[0] - (math.log1p(a) + a * d / (1 + a))) < 1e-12
    assert abs(logp[0] + math.log1p(a)) < 1e-12


# ----------------------------------------------------------------- KL term

def _kl_per_token(kind, logp, lp_ref):
    """The oracle's per-token KL value, read through the loss with A = 0,
    beta = 1 and one kept step under the all-token mean (l_t = kl_t / T)."""
    T = len(logp)
    res = oracle.tis_loss_ex(np.asarray(logp, np.float64), np.asarray(logp, np.float32),
                             np.asarray(logp, np.float32), np.zeros(T, np.float32),
                             np.array([0, T], np.int32), np.array([1], np.uint8), 0.2, 0.2, 2.0,
                             lp_ref=np.asarray(lp_ref, np.float32), kl=kind, beta=1.0,
                             agg="token_mean_all")
    return res["ell"] * T, res


@pytest.mark.parametrize("kind", ["k1", "k3"])
def test_kl_estimators_are_unbiased(kind):
    """With the sampled token drawn from pi_theta, k1 and k3 are unbiased for
    KL(pi_theta || pi_ref): the pi_theta-weighted average over every possible
    target equals scipy's relative entropy of the two distributions."""
    rng = np.random.default_rng(3)
    V = 9
    zt = rng.normal(0, 1.5, V)
    zr = rng.normal(0, 1.5, V)
    lp_t = scipy.special.log_softmax(zt)
    lp_r = scipy.special.log_softmax(zr)
    # lp_ref must be float32 at the boundary: make both exactly float32
    lp_t = lp_t.astype(np.float32).astype(np.float64)
    lp_r = lp_r.astype(np.float32).astype(np.float64)
    kl_tok, _ = _kl_per_token(kind, lp_t, lp_r)
    p = np.exp(lp_t)
    expect = float(np.sum(p * kl_tok))
    q = np.exp(lp_r)
    truth = float(np.sum(p * (lp_t - lp_r)))  # KL of the (float32-rounded) log-probs
    if kind == "k3":
        # E_p[q/p - 1] = sum q - sum p, which is 0 only for exactly normalised p, q
        truth += float(q.sum() - p.sum())
    assert abs(expect - truth) < 1e-12
    assert abs(truth - scipy.special.rel_entr(p / p.sum(), np.exp(lp_r) / np.exp(lp_r).sum()).sum()) < 1e-6


def test_kl_zero_at_reference_and_nonnegative():
    """Every estimator is 0 when pi_theta == pi_ref on the token; k2 and k3
    are never negative; for small differences k2 and k3 agree to second
    order."""
    lp = np.array([-1.0, -2.5, -0.25], np.float64)
    for kind in ("k1", "k2", "k3"):
        v, _ = _kl_per_token(kind, lp, lp)
        assert np.all(v == 0.0)
    rng = np.random.default_rng(4)
    lp = rng.normal(-3, 1, 200).astype(np.float32).astype(np.float64)
    ref = (lp + rng.normal(0, 2, 200)).astype(np.float32)
    assert np.all(_kl_per_token("k2", lp, ref)[0] >= 0)
    assert np.all(_kl_per_token("k3", lp, ref)[0] >= 0)
    small = (lp + 1e-3 * rng.normal(0, 1, 200)).astype(np.float32)
    v2, _ = _kl_per_token("k2", lp, small)
    v3, _ = _kl_per_token("k3", lp, small)
    d = np.abs(small.astype(np.float64) - lp)
    assert np.all(np.abs(v2 - v3) <= d ** 3)


def test_kl_outside_tis_weight_inside_indicator():
    """Eq. (2): the KL term is not multiplied by the TIS weight and vanishes
    for dropped steps."""
    logp = np.array([-1.0, -2.0], np.float64)
    lp_old = logp.astype(np.float32)
    lp_roll = (logp - 5.0).astype(np.float32)  # w = C = 2 on both tokens
    ref = np.array([-1.5, -1.0], np.float32)
    A = np.zeros(2, np.float32)
    off = np.array([0, 1, 2], np.int32)
    res = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, np.array([1, 0], np.uint8), 0.2, 0.2,
                             2.0, lp_ref=ref, kl="k1", beta=0.1)
    # kept token: N = 1, l = beta * kl = 0.1 * (logp - ref); dropped: 0
    assert abs(res["ell"][0] - 0.1 * (-1.0 + 1.5)) < 1e-15 and res["ell"][1] == 0.0
    assert abs(res["g"][0] - 0.1) < 1e-15 and res["g"][1] == 0.0
    assert res["stats"][1] == 2.0  # the mean TIS weight is the cap


# ----------------------------------------------------------------- aggregation

def _random_problem(seed, lens):
    rng = np.random.default_rng(seed)
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    T = int(off[-1])
    logp = rng.normal(-3, 1, T)
    lp_old = (logp + rng.normal(0, 0.2, T)).astype(np.float32)
    lp_roll = (lp_old + rng.normal(0, 0.3, T)).astype(np.float32)
    A = np.repeat(rng.normal(0, 1, len(lens)), lens).astype(np.float32)
    ref = (logp + rng.normal(0, 0.3, T)).astype(np.float32)
    mask = (rng.random(len(lens)) < 0.7).astype(np.uint8)
    mask[0] = 1
    return logp, lp_old, lp_roll, A, off, mask, ref


def test_step_mean_equals_token_mean_for_equal_lengths():
    args = _random_problem(5, [4] * 6)
    logp, lp_old, lp_roll, A, off, mask, ref = args
    a = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                           kl="k3", beta=0.1, agg="token_mean")
    b = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                           kl="k3", beta=0.1, agg="step_mean")
    assert abs(a["L"] - b["L"]) < 1e-14 and np.allclose(a["g"], b["g"], rtol=1e-13, atol=1e-16)


def test_token_mean_all_rescales_by_kept_fraction():
    logp, lp_old, lp_roll, A, off, mask, ref = _random_problem(6, [3, 5, 2, 7, 4])
    a = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0)
    b = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0,
                           agg="token_mean_all")
    N, T = a["stats"][3], off[-1]
    assert abs(b["L"] - a["L"] * N / T) < 1e-14
    assert np.allclose(b["g"], a["g"] * N / T, rtol=1e-13, atol=1e-18)


def test_step_mean_is_mean_of_per_step_losses():
    """The step mean decomposes: the mean over kept steps of each step's own
    token-mean loss (each step solved alone)."""
    logp, lp_old, lp_roll, A, off, mask, ref = _random_problem(7, [3, 5, 2, 7, 4])
    full = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                              kl="k2", beta=0.05, agg="step_mean")
    per = []
    for s in np.flatnonzero(mask):
        b, e = off[s], off[s + 1]
        r = oracle.tis_loss_ex(logp[b:e], lp_old[b:e], lp_roll[b:e], A[b:e],
                               np.array([0, e - b], np.int32), np.array([1], np.uint8), 0.2, 0.28,
                               2.0, lp_ref=ref[b:e], kl="k2", beta=0.05)
        per.append(r["L"])
    assert abs(full["L"] - np.mean(per)) < 1e-14


# ----------------------------------------------------------------- step-level ratio

def test_step_ratio_reduces_to_token_ratio_for_single_token_steps():
    logp, lp_old, lp_roll, A, off, mask, ref = _random_problem(8, [1] * 9)
    t = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                           kl="k3", beta=0.1)
    for ratio in ("step_geomean", "step_product"):
        s = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                               kl="k3", beta=0.1, ratio=ratio)
        assert abs(s["L"] - t["L"]) < 1e-14 and np.allclose(s["g"], t["g"], rtol=1e-13, atol=1e-18)


def test_two_token_step_ratio_closed_form():
    """Token ratios 1.1 and 1.3, A = 2, no truncation: the product ratio 1.43
    is clipped at 1 + eps_high = 1.28 (no gradient); the geometric mean
    sqrt(1.43) = 1.1958 is not (gradient r A / 2 on each token)."""
    logp = np.log(np.array([1.1, 1.3])) - 2.0
    lp_old = np.full(2, -2.0, np.float32)
    A = np.full(2, 2.0, np.float32)
    off = np.array([0, 2], np.int32)
    m = np.array([1], np.uint8)
    prod = oracle.tis_loss_ex(logp, lp_old, lp_old, A, off, m, 0.2, 0.28, 2.0,
                              agg="step_mean", ratio="step_product")
    geo = oracle.tis_loss_ex(logp, lp_old, lp_old, A, off, m, 0.2, 0.28, 2.0,
                             agg="step_mean", ratio="step_geomean")
    assert abs(prod["L"] - (-1.28 * 2.0)) < 1e-12 and np.all(prod["g"] == 0)
    rg = math.sqrt(1.1 * 1.3)
    assert abs(geo["L"] - (-rg * 2.0)) < 1e-12
    assert np.allclose(geo["g"], -rg * 2.0 / 2, rtol=1e-12)


# ----------------------------------------------------------------- gradients of every variant

@pytest.mark.parametrize("kl,agg,ratio,it", [
    ("k3", "token_mean", "token", 1.0), ("k1", "step_mean", "token", 0.5),
    ("k2", "token_mean_all", "step_geomean", 2.0), ("k3", "step_mean", "step_product", 1.0),
    ("none", "token_mean", "step_geomean", 0.7),
])
def test_variant_gradients_finite_differences(kl, agg, ratio, it):
    """Central differences of the loss (mini oracle, float64 logits) w.r.t.
    every logit match the C oracle's coefficient times the softmax derivative
    at inverse temperature it, for the KL term, each aggregation and each
    ratio level; every ratio is kept at least 5e-3 from the clip bounds."""
    rng = np.random.default_rng(hash((kl, agg, ratio)) % 2**31)
    lens = [2, 3, 1, 2]
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    T, V = int(off[-1]), 11
    z32 = rng.normal(0, 2, (T, V)).astype(np.float32)
    y = rng.integers(0, V, T).astype(np.int32)
    logp0, _, lse0 = oracle.token_stats(z32, y, inv_temp=it)
    A = np.repeat(rng.normal(0, 1, len(lens)), lens).astype(np.float32)
    mask = np.array([1, 0, 1, 1], np.uint8)
    eps_low, eps_high, C = 0.2, 0.28, 1.5
    # choose old log-probs so that every token and step ratio avoids the bounds
    for _ in range(200):
        lp_old = (logp0 - np.log(rng.choice([0.6, 0.95, 1.05, 1.5], T))).astype(np.float32)
        lr = logp0 - lp_old.astype(np.float64)
        ratios = list(np.exp(lr))
        for s in range(len(lens)):
            seg = lr[off[s]:off[s + 1]]
            ratios += [math.exp(seg.sum()), math.exp(seg.mean())]
        if all(min(abs(r - (1 - eps_low)), abs(r - (1 + eps_high))) > 5e-3 for r in ratios):
            break
    lp_roll = (lp_old + rng.normal(0, 0.5, T)).astype(np.float32)
    ref = (logp0 + rng.normal(0, 0.3, T)).astype(np.float32)
    beta = 0.1
    res = oracle.tis_loss_ex(logp0, lp_old, lp_roll, A, off, mask, eps_low, eps_high, C,
                             lp_ref=ref, kl=kl, beta=beta, agg=agg, ratio=ratio)
    dz = oracle.dlogits(z32, y, lse0, logp0, res["g"], inv_temp=it)
    rows = z32.astype(np.float64).tolist()

    def L_of(rows_):
        st = mini.token_stats(rows_, y.tolist(), inv_temp=it)
        L, _ = mini.loss_ex([s[0] for s in st], lp_old.astype(np.float64).tolist(),
                            lp_roll.astype(np.float64).tolist(), ref.astype(np.float64).tolist(),
                            A.astype(np.float64).tolist(), off.tolist(), mask.tolist(), eps_low,
                            eps_high, C, kl=kl, beta=beta, agg=agg, ratio=ratio)
        return L

    assert abs(L_of(rows) - res["L"]) < 1e-12
    h = 1e-5
    fd = np.zeros((T, V))
    for t in range(T):
        for v in range(V):
            zp = [row[:] for row in rows]
            zm = [row[:] for row in rows]
            zp[t][v] += h
            zm[t][v] -= h
            fd[t, v] = (L_of(zp) - L_of(zm)) / (2 * h)
    assert np.allclose(fd, dz, rtol=1e-6, atol=1e-8 * np.abs(dz).max())


@pytest.mark.parametrize("seed", range(5))
def test_c_oracle_matches_mini_oracle_variants(seed):
    rng = np.random.default_rng(500 + seed)
    lens = list(rng.integers(1, 5, int(rng.integers(1, 6))))
    logp, lp_old, lp_roll, A, off, mask, ref = _random_problem(600 + seed, lens)
    kl = ["none", "k1", "k2", "k3"][seed % 4]
    agg = ["token_mean", "token_mean_all", "step_mean"][seed % 3]
    ratio = ["token", "step_geomean", "step_product"][(seed // 2) % 3]
    a = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0, lp_ref=ref,
                           kl=kl, beta=0.1, agg=agg, ratio=ratio)
    L, g = mini.loss_ex(list(logp), list(lp_old.astype(np.float64)), list(lp_roll.astype(np.float64)),
                        list(ref.astype(np.float64)), list(A.astype(np.float64)), list(off),
                        list(mask), 0.2, 0.28, 2.0, kl=kl, beta=0.1, agg=agg, ratio=ratio)
    assert abs(a["L"] - L) < 1e-12 and np.allclose(a["g"], g, rtol=0, atol=1e-12)


def test_default_configuration_is_the_base_loss():
    logp, lp_old, lp_roll, A, off, mask, ref = _random_problem(9, [3, 5, 2])
    a = oracle.tis_loss(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0)
    b = oracle.tis_loss_ex(logp, lp_old, lp_roll, A, off, mask, 0.2, 0.28, 2.0)
    assert a["L"] == b["L"] and np.array_equal(a["g"], b["g"])
    assert np.array_equal(a["stats"], b["stats"][:4])
