"""Pins of the oracle's LM-head functions: the statistics of softmax(h W^T)
(Sec. 4.3 on the logits of the LM head) and the gradients of the loss with
respect to the hidden states and the weight. The logits are formed in float64
by one matrix product of the exact bf16 inputs; these tests fix that product's
orientation and the backward formulas against closed forms, a second path to
the same logits, the pure-Python oracle and finite differences."""

import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
from oracle import mini
from synth import f32_to_bf16_bits, gaussian_bits


def _bits(x):
    """float array -> bf16 bits; the tests only pass values exact in bf16."""
    b = f32_to_bf16_bits(np.asarray(x, np.float32))
    assert np.array_equal(oracle.bf16_bits_to_f64(b), np.asarray(x, np.float64))
    return b


def test_zero_weight_gives_uniform_rows():
    """W = 0 makes every logit 0: H = ln V, logp = -ln V, lse = ln V."""
    T, d, V = 5, 16, 37
    h = gaussian_bits(1, 9, T, d, 1.0)
    w = np.zeros((V, d), np.uint16)
    y = np.arange(T, dtype=np.int32) % V
    logp, H, lse = oracle.lmhead_token_stats(h, w, y)
    assert np.allclose(H, math.log(V), atol=1e-13)
    assert np.allclose(logp, -math.log(V), atol=1e-13)
    assert np.allclose(lse, math.log(V), atol=1e-13)


def test_one_hot_weight_rows_select_hidden_features():
    """W_v = e_{k(v)} gives z_{t,v} = h_{t,k(v)}: the statistics equal those of
    the logits built by indexing h directly (the float32 reader of the oracle).
    A transposed product or a wrong operand would pick other features."""
    rng = np.random.default_rng(3)
    T, d, V = 6, 24, 50
    h = gaussian_bits(2, 9, T, d, 2.0)
    k = rng.integers(0, d, V)
    w = np.zeros((V, d), np.uint16)
    w[np.arange(V), k] = _bits(np.ones(1))[0]
    y = rng.integers(0, V, T).astype(np.int32)
    got = oracle.lmhead_token_stats(h, w, y)
    direct = oracle.bf16_bits_to_f64(h)[:, k].astype(np.float32)
    want = oracle.token_stats(np.ascontiguousarray(direct), y)
    for a, b in zip(got, want):
        assert np.allclose(a, b, rtol=0, atol=1e-13)


def test_rank_one_closed_form():
    """h_t = a_t u, W_v = b_v u: z_{t,v} = a_t b_v |u|^2 exactly; lse, H and
    logp from scipy's logsumexp and entropy on that outer product."""
    rng = np.random.default_rng(5)
    T, d, V = 4, 32, 300
    u = rng.choice([-1.0, 1.0], d)
    a = rng.choice([0.25, 0.5, 1.0, -0.75], T)
    b = rng.integers(-8, 9, V) / 8.0
    h = _bits(np.outer(a, u))
    w = _bits(np.outer(b, u))
    y = rng.integers(0, V, T).astype(np.int32)
    z = np.outer(a, b) * d
    logp, H, lse = oracle.lmhead_token_stats(h, w, y)
    want_lse = scipy.special.logsumexp(z, axis=1)
    p = scipy.special.softmax(z, axis=1)
    assert np.allclose(lse, want_lse, rtol=0, atol=1e-12)
    assert np.allclose(H, scipy.stats.entropy(p, axis=1), rtol=0, atol=1e-12)
    assert np.allclose(logp, z[np.arange(T), y] - want_lse, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_matches_mini_oracle_dot_products(seed):
    """The C oracle on h W^T agrees with the pure-Python oracle on logits
    summed term by term (math.fsum of h_tk W_vk)."""
    rng = np.random.default_rng(40 + seed)
    T, d, V = 3, int(rng.integers(8, 40)), int(rng.integers(2, 30))
    h = gaussian_bits(seed, 9, T, d, 1.0)
    w = gaussian_bits(seed, 10, V, d, 3.0 / math.sqrt(d))
    y = rng.integers(0, V, T).astype(np.int32)
    hf, wf = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    rows = [[math.fsum(hf[t, k] * wf[v, k] for k in range(d)) for v in range(V)] for t in range(T)]
    mini_stats = mini.token_stats(rows, y.tolist())
    logp, H, lse = oracle.lmhead_token_stats(h, w, y)
    for t in range(T):
        assert abs(logp[t] - mini_stats[t][0]) <= 1e-12
        assert abs(H[t] - mini_stats[t][1]) <= 1e-12
        assert abs(lse[t] - mini_stats[t][2]) <= 1e-12


@pytest.mark.parametrize("seed,inv_temp", [(0, 1.0), (1, 1.0), (2, 1.0), (3, 0.7), (4, 1.6)])
def test_grads_finite_differences(seed, inv_temp):
    """Central differences of the loss (through the LM head, the statistics and
    the clipped TIS surrogate, with the mask and TIS weights fixed) with
    respect to every hidden-state and weight entry match dh = dz W and
    dW = dz^T h; ratios are kept away from the clip bounds. At an inverse
    temperature the differenced loss takes softmax(inv_temp h W^T), formed in
    the pure-Python statistics, so the factor the chain rule adds is pinned."""
    rng = np.random.default_rng(70 + seed)
    T, d, V = 5, 6, 9
    h = gaussian_bits(seed, 9, T, d, 1.0)
    w = gaussian_bits(seed, 10, V, d, 1.0)
    y = rng.integers(0, V, T).astype(np.int32)
    off = np.array([0, 2, 5], np.int32)
    mask = np.array([1, 1], np.uint8) if seed % 2 == 0 else np.array([0, 1], np.uint8)
    A = rng.normal(0, 1, T).astype(np.float32)
    eps_low, eps_high, C = 0.2, 0.28, 1.5
    logp0, _, lse0 = oracle.lmhead_token_stats(h, w, y, inv_temp=inv_temp)
    r_target = rng.choice([0.6, 0.95, 1.1, 1.5], T)
    lp_old = (logp0 - np.log(r_target)).astype(np.float32)
    lp_roll = (lp_old + rng.normal(0, 0.5, T)).astype(np.float32)
    res = oracle.tis_loss(logp0, lp_old, lp_roll, A, off, mask, eps_low, eps_high, C)
    _, dh, dW = oracle.lmhead_grads(h, w, y, lse0, logp0, res["g"], inv_temp=inv_temp)

    hf, wf = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)

    def L_of(hh, ww):
        rows = (inv_temp * (hh @ ww.T)).tolist()
        st = mini.token_stats(rows, y.tolist())
        L, _ = mini.loss_and_coef([s[0] for s in st], lp_old.astype(np.float64).tolist(),
                                  lp_roll.astype(np.float64).tolist(), A.astype(np.float64).tolist(),
                                  off.tolist(), mask.tolist(), eps_low, eps_high, C)
        return L

    eps = 1e-6
    fd_h = np.zeros_like(hf)
    for t in range(T):
        for k in range(d):
            hp, hm = hf.copy(), hf.copy()
            hp[t, k] += eps
            hm[t, k] -= eps
            fd_h[t, k] = (L_of(hp, wf) - L_of(hm, wf)) / (2 * eps)
    fd_w = np.zeros_like(wf)
    for v in range(V):
        for k in range(d):
            wp, wm = wf.copy(), wf.copy()
            wp[v, k] += eps
            wm[v, k] -= eps
            fd_w[v, k] = (L_of(hf, wp) - L_of(hf, wm)) / (2 * eps)
    assert dh.shape == (T, d) and dW.shape == (V, d)
    assert np.allclose(fd_h, dh, rtol=1e-5, atol=1e-8 * max(np.abs(dh).max(), 1e-30))
    assert np.allclose(fd_w, dW, rtol=1e-5, atol=1e-8 * max(np.abs(dW).max(), 1e-30))


def test_float64_logits_reader_matches_float32_reader():
    """The oracle's float64 logits path gives the same statistics as its
    float32 path on logits that are exactly float32."""
    rng = np.random.default_rng(9)
    z32 = rng.normal(0, 3, (4, 333)).astype(np.float32)
    y = rng.integers(0, 333, 4).astype(np.int32)
    a = oracle.token_stats(z32, y)
    b = oracle.token_stats(z32.astype(np.float64), y)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
