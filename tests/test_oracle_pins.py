"""Pins of the float64 oracle against what the paper and mathematics fix.

The paper (DART, arXiv 2509.23866) prints no worked numeric example for this
path, so each oracle function is pinned by closed forms, invariants, special
cases that reduce to a textbook or library routine, brute force on tiny inputs,
and central finite differences. Each test names the mistake it would catch.
"""

import itertools
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
from oracle import mini
from synth import f32_to_bf16_bits

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rows_f32(rows):
    return np.ascontiguousarray(np.asarray(rows, dtype=np.float32))


# --------------------------------------------------------------------------
# token entropy and log-prob (Sec. 4.3 definition of H and p; Eq. 1 numerator)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("V", [1, 2, 3, 7, 4096, 151936])
@pytest.mark.parametrize("c", [0.0, -7.25, 13.5])
def test_uniform_row_entropy_is_log_v(V, c):
    """A flat row has H = ln V and logp = -ln V (catches log2 vs ln, a missing
    normaliser, an off-by-one in V)."""
    z = np.full((2, V), c, dtype=np.float32)
    logp, H, lse = oracle.token_stats(z, [0, V - 1])
    tol = (1e-12 + V * 2.0 ** -52) * max(1.0, math.log(V))  # sequential sum of V terms
    assert np.allclose(H, math.log(V), rtol=0, atol=tol)
    assert np.allclose(logp, -math.log(V), rtol=0, atol=tol)
    assert np.allclose(lse, c + math.log(V), rtol=0, atol=tol + 1e-14 * abs(c))


def test_uniform_row_bf16_v151936_value():
    """The flat edge-workload row (V = 151936, bf16 zeros) gives
    H = ln 151936 = 11.931214658529285."""
    z = np.zeros((1, 151936), dtype=np.uint16)
    _, H, _ = oracle.token_stats(z, [5])
    # sequential float64 summation of V equal terms: error below V * 2^-53 * H
    assert abs(H[0] - 11.931214658529285) < 151936 * 2.0 ** -53 * 12


@pytest.mark.parametrize("V", [2, 33, 151936])
@pytest.mark.parametrize("delta", [0.5, 4.0, 30.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_two_level_row_closed_form(V, delta, dtype):
    """One logit raised by delta over a flat row: with a = (V-1) e^-delta,
    p_spike = 1/(1+a), H = ln(1+a) + a delta/(1+a),
    logp_spike = -ln(1+a), logp_other = -delta - ln(1+a)
    (catches a dropped entropy term, a wrong sign, the target index)."""
    z = np.zeros((2, V), dtype=np.float32)
    z[:, 3 % V] = delta
    if dtype == "bf16":
        z = f32_to_bf16_bits(z)
    logp, H, _ = oracle.token_stats(z, [3 % V, (3 % V + 1) % V])
    a = (V - 1) * math.exp(-delta)
    H_ref = math.log1p(a) + a * delta / (1 + a)
    tol = (1e-12 + V * 2.0 ** -52) * max(1.0, H_ref)  # sequential sum of V terms
    assert abs(H[0] - H_ref) <= tol
    assert abs(H[1] - H_ref) <= tol
    assert abs(logp[0] + math.log1p(a)) < tol
    assert abs(logp[1] - (-delta - math.log1p(a))) < tol


def test_near_one_hot_entropy_value():
    """Delta = 30 over V = 151936 zeros: H = 4.407e-7 (close to 0)."""
    V = 151936
    z = np.zeros((1, V), dtype=np.float32)
    z[0, 17] = 30.0
    _, H, _ = oracle.token_stats(z, [17])
    a = (V - 1) * math.exp(-30.0)
    # lse ~ 30 carries an absolute rounding of ulp(30)/2 = 1.8e-15
    assert abs(H[0] - (math.log1p(a) + 30 * a / (1 + a))) < 1e-14
    assert 4.40e-7 < H[0] < 4.41e-7


def test_binary_row_is_sigmoid_entropy():
    """V = 2 reduces to the Bernoulli entropy of sigma(z0 - z1) and
    logp = log sigma (textbook closed form)."""
    rng = np.random.default_rng(0)
    z = rng.normal(0, 3, size=(50, 2)).astype(np.float32)
    logp, H, _ = oracle.token_stats(z, np.zeros(50, np.int32))
    d = z[:, 0].astype(np.float64) - z[:, 1]
    p = 1 / (1 + np.exp(-d))
    ref = -(p * np.log(p) + (1 - p) * np.log(1 - p))
    assert np.allclose(H, ref, rtol=1e-11, atol=1e-14)
    assert np.allclose(logp, -np.log1p(np.exp(-d)), rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("V", [5, 64, 1000, 4099])
def test_matches_scipy(V):
    """Independent library routines: scipy's log_softmax and entropy."""
    rng = np.random.default_rng(V)
    z = (rng.normal(0, 3, size=(6, V))).astype(np.float32)
    y = rng.integers(0, V, size=6).astype(np.int32)
    logp, H, lse = oracle.token_stats(z, y)
    z64 = z.astype(np.float64)
    ls = scipy.special.log_softmax(z64, axis=1)
    assert np.allclose(logp, ls[np.arange(6), y], rtol=0, atol=1e-12)
    assert np.allclose(H, scipy.stats.entropy(np.exp(ls), axis=1), rtol=1e-12, atol=1e-12)
    assert np.allclose(lse, scipy.special.logsumexp(z64, axis=1), rtol=1e-14, atol=1e-12)


def test_shift_invariance():
    """Adding a constant to a row leaves H and logp unchanged (values are
    multiples of 2^-10 below 64, so the shift is exact in float32)."""
    rng = np.random.default_rng(1)
    z = np.round(rng.normal(0, 3, size=(4, 777)) * 1024) / 1024
    y = rng.integers(0, 777, 4).astype(np.int32)
    a = oracle.token_stats(z.astype(np.float32), y)
    b = oracle.token_stats((z + 8.0).astype(np.float32), y)
    assert np.allclose(a[0], b[0], atol=1e-12) and np.allclose(a[1], b[1], atol=1e-12)
    assert np.allclose(b[2] - a[2], 8.0, atol=1e-12)


def test_permutation_invariance():
    """Permuting the vocabulary (with the target remapped) leaves H and logp
    unchanged (catches reading a wrong column or a row stride bug)."""
    rng = np.random.default_rng(2)
    V = 513
    z = rng.normal(0, 2, size=(5, V)).astype(np.float32)
    y = rng.integers(0, V, 5).astype(np.int32)
    perm = rng.permutation(V)
    inv = np.argsort(perm)
    a = oracle.token_stats(z, y)
    b = oracle.token_stats(np.ascontiguousarray(z[:, perm]), inv[y].astype(np.int32))
    assert np.allclose(a[0], b[0], atol=1e-12) and np.allclose(a[1], b[1], atol=1e-12)


def test_entropy_bounds_and_neg_inf():
    """0 <= H <= ln V; a row that is -inf except at one logit has H = 0 and
    logp = 0 for that logit (0 log 0 := 0)."""
    rng = np.random.default_rng(3)
    z = rng.normal(0, 5, size=(20, 300)).astype(np.float32)
    _, H, _ = oracle.token_stats(z, np.zeros(20, np.int32))
    assert np.all(H >= 0) and np.all(H <= math.log(300) + 1e-12)
    w = np.full((1, 10), -np.inf, dtype=np.float32)
    w[0, 4] = 1.5
    logp, H, _ = oracle.token_stats(w, [4])
    assert H[0] == 0.0 and logp[0] == 0.0


def test_row_stride_is_respected():
    """A padded row stride reads only the first V columns."""
    rng = np.random.default_rng(4)
    full = rng.normal(0, 3, size=(3, 40)).astype(np.float32)
    full[:, 33:] = np.nan
    y = np.array([0, 10, 32], np.int32)
    a = oracle.token_stats(full[:, :33], y)
    b = oracle.token_stats(np.ascontiguousarray(full[:, :33]), y)
    assert np.array_equal(a[1], b[1]) and np.all(np.isfinite(a[1]))


# --------------------------------------------------------------------------
# step entropy (Sec. 4.3 mean over the step's tokens)
# --------------------------------------------------------------------------

def test_step_entropy_special_cases():
    """Constant H inside a step gives that constant; singleton steps give H
    itself; ragged steps agree with numpy's mean of each slice."""
    off = np.array([0, 3, 4, 9, 10], np.int32)
    H = np.array([2.0, 2.0, 2.0, 7.5, 1, 2, 3, 4, 5, 0.25])
    Hs, Hs32 = oracle.step_entropy(H, off)
    assert Hs[0] == 2.0 and Hs[1] == 7.5 and Hs[3] == 0.25
    assert Hs[2] == np.mean(H[4:9])
    assert np.array_equal(Hs32, Hs.astype(np.float32))


def test_step_entropy_of_closed_form_rows():
    """Steps built from flat rows of width V and from two-level rows have the
    closed-form entropies averaged over the step."""
    V = 257
    flat = np.zeros((3, V), np.float32)
    spike = np.zeros((2, V), np.float32)
    spike[:, 0] = 4.0
    z = np.concatenate([flat, spike, flat[:1]])
    _, H, _ = oracle.token_stats(z, np.zeros(6, np.int32))
    Hs, _ = oracle.step_entropy(H, np.array([0, 4, 6], np.int32))
    a = (V - 1) * math.exp(-4.0)
    h2 = math.log1p(a) + 4 * a / (1 + a)
    assert abs(Hs[0] - (3 * math.log(V) + h2) / 4) < 1e-12
    assert abs(Hs[1] - (h2 + math.log(V)) / 2) < 1e-12


# --------------------------------------------------------------------------
# step selection (Sec. 4.3: the highest-entropy 80% of steps; indicator of Eq. 2)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rho,S,k", [(0.8, 240, 192), (0.8, 64, 52), (0.5, 16, 8),
                                     (0.5, 1600, 800), (0.25, 256, 64), (1.0, 7, 7),
                                     (0.0, 7, 0), (0.8, 10, 8), (0.8, 1, 1), (0.01, 3, 1)])
def test_kept_steps_table(rho, S, k):
    """k = ceil(rho S) with the representation guard (0.8 * 240 is
    192.00000000000003 in double and must give 192)."""
    assert oracle.kept_steps(S, rho) == k
    assert mini.kept_count(S, rho) == k


def _brute_force_mask(keys, k):
    """Among all k-subsets whose every kept key is >= every dropped key, the
    one with the lexicographically smallest index tuple (lower index wins
    ties)."""
    S = len(keys)
    best = None
    for sub in itertools.combinations(range(S), k):
        kept = set(sub)
        drop = [keys[s] for s in range(S) if s not in kept]
        if sub and drop and min(keys[s] for s in sub) < max(drop):
            continue
        if best is None or sub < best:
            best = sub
    m = np.zeros(S, np.uint8)
    m[list(best)] = 1
    return m


@pytest.mark.parametrize("seed", range(12))
def test_mask_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    S = int(rng.integers(1, 10))
    keys = rng.choice([0.5, 1.0, 1.5, 2.0, 7.25], size=S).astype(np.float32)  # many ties
    rho = float(rng.choice([0.0, 0.25, 0.5, 0.8, 1.0, rng.uniform()]))
    mask, k = oracle.step_mask(keys, rho)
    assert k == oracle.kept_steps(S, rho)
    assert np.array_equal(mask, _brute_force_mask(list(keys), k))


def test_mask_threshold_property_and_paper_fraction():
    """rho = 0.8 keeps ceil(0.8 S) steps and every kept step has higher
    entropy than every dropped one (distinct entropies)."""
    rng = np.random.default_rng(7)
    Hs = rng.permutation(np.arange(10, dtype=np.float32)) + 0.5
    mask, k = oracle.step_mask(Hs, 0.8)
    assert k == 8 and mask.sum() == 8
    assert Hs[mask == 1].min() > Hs[mask == 0].max()
    assert set(np.flatnonzero(mask == 0)) == set(np.argsort(Hs)[:2])


def test_mask_all_and_none():
    Hs = np.array([3, 1, 2, 2], np.float32)
    assert oracle.step_mask(Hs, 1.0)[0].tolist() == [1, 1, 1, 1]
    assert oracle.step_mask(Hs, 0.0)[0].tolist() == [0, 0, 0, 0]
    assert oracle.step_mask(Hs, 0.5)[0].tolist() == [1, 0, 1, 0]  # tie 2 vs 2: lower index


# --------------------------------------------------------------------------
# TIS weight, clipped surrogate, loss and coefficient (Eq. 1, Sec. 4.4, Eq. 2)
# --------------------------------------------------------------------------

def _one_step(logp, lp_old, lp_roll, adv, eps_low=0.2, eps_high=0.28, C=2.0, mask=(1,)):
    T = len(logp)
    return oracle.tis_loss(np.asarray(logp, np.float64), np.asarray(lp_old, np.float32),
                           np.asarray(lp_roll, np.float32), np.asarray(adv, np.float32),
                           np.array([0, T], np.int32), np.asarray(mask, np.uint8),
                           eps_low, eps_high, C)


def test_ratio_one_gives_minus_mean_advantage():
    """lp_old = logp and lp_roll = lp_old give r = w = 1, so the loss is minus
    the token mean of the kept advantages and g_t = -A_t / N; dropped steps
    contribute nothing (catches the sign, the denominator, the mask)."""
    rng = np.random.default_rng(8)
    T = 12
    logp = rng.normal(-2, 1, T).astype(np.float32).astype(np.float64)
    adv = rng.normal(0, 1, T).astype(np.float32)
    off = np.array([0, 5, 8, 12], np.int32)
    mask = np.array([1, 0, 1], np.uint8)
    res = oracle.tis_loss(logp, logp.astype(np.float32), logp.astype(np.float32), adv, off, mask,
                          0.2, 0.28, 2.0)
    kept = np.r_[0:5, 8:12]
    assert abs(res["L"] - (-adv[kept].astype(np.float64).mean())) < 1e-14
    g_ref = np.zeros(T)
    g_ref[kept] = -adv[kept].astype(np.float64) / 9.0
    assert np.allclose(res["g"], g_ref, rtol=1e-14, atol=1e-16)
    assert res["stats"][3] == 9 and res["stats"][1] == 1.0 and res["stats"][0] == 0.0


def test_tis_weight_cap_and_unit():
    """d = lp_old - lp_roll >= ln C gives w = C exactly; d = 0 gives w = 1;
    a d below ln C gives exp(d) (catches a dropped or inverted weight)."""
    C = 2.0
    lp = [-1.0] * 4
    lp_roll = np.array([-1.0 - math.log(C) - 0.25, -1.0 - math.log(C) - 3.0, -1.0, -1.0 - 0.5],
                       np.float32)
    res = _one_step(lp, lp, lp_roll, [1.0] * 4, C=C)
    d = np.float64(-1.0) - lp_roll.astype(np.float64)
    w_ref = np.array([C, C, 1.0, math.exp(d[3])])
    assert np.allclose(res["ell"], -w_ref / 4, rtol=1e-15, atol=0)
    assert res["stats"][2] == 0.5  # two of four at the cap


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.28), (0.1, 0.5)])
def test_clip_branches(eps_low, eps_high):
    """The four branches of min(rA, clip(r) A) with asymmetric bounds
    (catches swapped bounds, an inverted ratio, a gradient through the clip):
      A>0, r>1+eh : o = (1+eh) A, g = 0
      A<0, r<1-el : o = (1-el) A, g = 0
      A>0, r<1-el : o = r A,      g = -w A r / N
      A<0, r>1+eh : o = r A,      g = -w A r / N
      A=0         : o = 0,        g = 0"""
    lp_old = np.zeros(5, np.float32)
    r = np.array([1.9, 0.5, 0.5, 1.9, 1.3])
    A = np.array([1.5, -2.0, 0.75, -0.5, 0.0], np.float32)
    logp = np.log(r)
    res = _one_step(logp, lp_old, lp_old, A, eps_low, eps_high, C=2.0)
    N = 5.0
    r_ = np.exp(logp)
    a = A.astype(np.float64)
    o = np.array([(1 + eps_high) * a[0], (1 - eps_low) * a[1], r_[2] * a[2], r_[3] * a[3], 0.0])
    g = np.array([0.0, 0.0, -a[2] * r_[2] / N, -a[3] * r_[3] / N, 0.0])
    assert np.allclose(res["ell"], -o / N, rtol=1e-14, atol=1e-300)
    assert np.allclose(res["g"], g, rtol=1e-14, atol=1e-300)
    assert res["stats"][0] == pytest.approx(2 / 5)


def test_no_clip_no_cap_limit():
    """With eps and C unbounded the loss is -sum w r A / N over kept tokens."""
    rng = np.random.default_rng(9)
    T = 30
    logp = rng.normal(-3, 1, T)
    lp_old = (logp + rng.normal(0, 0.5, T)).astype(np.float32)
    lp_roll = (lp_old + rng.normal(0, 0.5, T)).astype(np.float32)
    A = rng.normal(0, 1, T).astype(np.float32)
    res = _one_step(logp, lp_old, lp_roll, A, eps_low=1e30, eps_high=1e30, C=math.inf)
    r = np.exp(logp - lp_old.astype(np.float64))
    w = np.exp(lp_old.astype(np.float64) - lp_roll)
    assert abs(res["L"] - (-(w * r * A).sum() / T)) < 1e-13
    assert np.allclose(res["g"], -w * r * A / T, rtol=1e-13)


def test_no_kept_tokens():
    """rho = 0 (N = 0): the loss and every coefficient are 0."""
    res = _one_step([-1.0, -2.0], [-1.1, -2.1], [-1.0, -2.0], [1.0, -1.0], mask=(0,))
    assert res["L"] == 0.0 and np.all(res["g"] == 0.0)


# --------------------------------------------------------------------------
# gradient w.r.t. the logits (chain rule through log pi_theta in Eq. 2)
# --------------------------------------------------------------------------

def test_dlogits_rows_sum_to_zero():
    """sum_v g (delta - p) = g (1 - sum p) = 0."""
    rng = np.random.default_rng(10)
    z = rng.normal(0, 3, (6, 1000)).astype(np.float32)
    y = rng.integers(0, 1000, 6).astype(np.int32)
    logp, _, lse = oracle.token_stats(z, y)
    g = rng.normal(0, 1e-3, 6)
    dz = oracle.dlogits(z, y, lse, logp, g)
    assert np.all(np.abs(dz.sum(axis=1)) <= 1e-14 * np.abs(g) * 10)
    assert np.all(np.sign(dz[np.arange(6), y]) == np.sign(g))


@pytest.mark.parametrize("seed", range(4))
def test_dlogits_finite_differences(seed):
    """Central differences of the oracle's loss w.r.t. every logit, with the
    mask (hence N) and the TIS weights fixed, match g (delta - p). Inputs keep
    every ratio at least 1e-3 away from the clip bounds."""
    rng = np.random.default_rng(100 + seed)
    T, V = 7, int(rng.integers(3, 33))
    z = rng.normal(0, 2, (T, V))
    y = rng.integers(0, V, T).astype(np.int32)
    off = np.array([0, 2, 5, 7], np.int32)
    mask = np.array([1, 0, 1], np.uint8) if seed % 2 else np.array([1, 1, 1], np.uint8)
    A = rng.normal(0, 1, T).astype(np.float32)
    eps_low, eps_high, C = 0.2, 0.28, 1.5

    def loss_of(zz):
        logp, _, _ = oracle.token_stats(zz, y)
        return oracle.tis_loss(logp, lp_old, lp_roll, A, off, mask, eps_low, eps_high, C)["L"]

    z64 = z  # float64 logits are passed through float32 storage below
    # make the logits exactly float32 and pick lp_old so that ratios avoid the bounds
    z32 = z64.astype(np.float32)
    logp0, _, lse0 = oracle.token_stats(z32, y)
    r_target = rng.choice([0.6, 0.95, 1.1, 1.5], T)
    lp_old = (logp0 - np.log(r_target)).astype(np.float32)
    lp_roll = (lp_old + rng.normal(0, 0.5, T)).astype(np.float32)
    res = oracle.tis_loss(logp0, lp_old, lp_roll, A, off, mask, eps_low, eps_high, C)
    dz = oracle.dlogits(z32, y, lse0, logp0, res["g"])

    # finite differences in float64: evaluate the same definitions on float64
    # logits through the pure-Python oracle (the C oracle reads float32 storage)
    rows = z32.astype(np.float64).tolist()

    def L_of(rows_):
        st = mini.token_stats(rows_, y.tolist())
        L, _ = mini.loss_and_coef([s[0] for s in st], lp_old.astype(np.float64).tolist(),
                                  lp_roll.astype(np.float64).tolist(),
                                  A.astype(np.float64).tolist(), off.tolist(), mask.tolist(),
                                  eps_low, eps_high, C)
        return L

    h = 1e-5
    fd = np.zeros((T, V))
    for t in range(T):
        for v in range(V):
            zp = [row[:] for row in rows]
            zm = [row[:] for row in rows]
            zp[t][v] += h
            zm[t][v] -= h
            fd[t, v] = (L_of(zp) - L_of(zm)) / (2 * h)
    scale = np.abs(dz).max()
    assert np.allclose(fd, dz, rtol=1e-6, atol=1e-8 * scale)


# --------------------------------------------------------------------------
# the two oracles agree
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_c_oracle_matches_mini_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    S = int(rng.integers(1, 5))
    lens = rng.integers(1, 4, S)
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    T = int(off[-1])
    V = int(rng.integers(1, 40))
    z = rng.normal(0, 3, (T, V)).astype(np.float32)
    y = rng.integers(0, V, T).astype(np.int32)
    lp_old = rng.normal(-3, 1, T).astype(np.float32)
    lp_roll = (lp_old + rng.normal(0, 1, T)).astype(np.float32)
    A = rng.normal(0, 1, T).astype(np.float32)
    rho = float(rng.choice([0.0, 0.5, 0.8, 1.0]))
    a = oracle.forward_backward(z, y, lp_old, lp_roll, A, off, rho, 0.2, 0.28, 2.0)
    b = mini.forward_backward(z.astype(np.float64).tolist(), y.tolist(),
                              lp_old.astype(np.float64).tolist(), lp_roll.astype(np.float64).tolist(),
                              A.astype(np.float64).tolist(), off.tolist(), rho, 0.2, 0.28, 2.0)
    assert np.allclose(a["logp"], b["logp"], rtol=0, atol=1e-12)
    assert np.allclose(a["H"], b["H"], rtol=0, atol=1e-12)
    assert np.allclose(a["Hs"], b["Hs"], rtol=0, atol=1e-12)
    assert a["mask"].tolist() == b["mask"] and a["k"] == b["k"]
    assert abs(a["L"] - b["L"]) < 1e-12
    assert np.allclose(a["g"], b["g"], rtol=0, atol=1e-12)
    assert np.allclose(a["dz"], np.array(b["dz"]), rtol=0, atol=1e-12)


def test_bf16_rounding_helper():
    """f64 -> bf16 rounding is nearest-even and agrees with float32 rounding
    where the double is exactly a float32."""
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5e-20, 3e-39, 0.0, -0.0])
    bits = oracle.f64_to_bf16_bits(x)
    assert bits[0] == 0x3F80 and bits[1] == 0x3F80 and bits[2] == 0x3F82
    assert np.array_equal(oracle.f64_to_bf16_bits(x[:5].astype(np.float32).astype(np.float64)),
                          f32_to_bf16_bits(x[:5].astype(np.float32)))


def test_boundary_flag_marks_only_ratios_at_a_clip_bound():
    """The gate of the gradient can differ between precisions only where the
    ratio sits at a clip bound; ratios strictly inside or outside the range,
    and zero advantages, are not excused from element-wise checks."""
    r = np.array([1.0, 0.9, 1.1, 0.5, 1.9, 0.8 * (1 + 5e-5), 1.28 * (1 - 5e-5), 0.8, 1.28])
    A = np.array([1.0, -1.0, 2.0, 1.0, -1.0, 1.0, -2.0, 0.0, 1.0], np.float32)
    logp = np.log(r)
    res = _one_step(logp, np.zeros(9, np.float32), np.zeros(9, np.float32), A, 0.2, 0.28, 2.0)
    assert res["boundary"].tolist() == [False] * 5 + [True, True, False, True]


@pytest.mark.parametrize("V,delta", [(777, 30.0), (151936, 30.0), (33, 20.0)])
def test_near_one_hot_logp_and_gradient_relative_accuracy(V, delta):
    """Spike at the target: log p_y = -log1p(a) and 1 - p_y = a / (1 + a),
    a = (V-1) e^-delta, to 1e-10 *relative* accuracy (both are ~1e-11 here,
    far below the resolution of lse ~ delta) - the gradient's row scale."""
    z = np.zeros((1, V), np.float32)
    z[0, 3] = delta
    logp, H, lse = oracle.token_stats(z, [3])
    a = (V - 1) * math.exp(-delta)
    assert abs(logp[0] / -math.log1p(a) - 1) < 1e-10
    g = np.array([0.25])
    dz = oracle.dlogits(z, [3], lse, logp, g)
    assert abs(dz[0, 3] / (0.25 * a / (1 + a)) - 1) < 1e-10
    assert abs(dz[0, 0] / (-0.25 * math.exp(-delta) / (1 + a)) - 1) < 1e-12
