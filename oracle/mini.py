"""Pure-Python mini oracle (lists and ``math`` only) for tiny shapes.

TEST INFRASTRUCTURE ONLY. A second, independently written reading of the same
definitions as ``dart_oracle.c`` (DART, arXiv 2509.23866: Sec. 4.3 for the
token and step entropy and the step selection, Sec. 4.4 for the truncated
importance weight, Eq. (1)/(2) for the clipped surrogate). The two are required
to agree to 1e-12 on random tiny inputs. Logits are given as Python floats
(already the exact float32/bfloat16 values).
"""

from __future__ import annotations

import math


def token_stats(rows, targets, inv_temp=1.0):
    """Sec. 4.3: per row, log-prob of the target, entropy and log-normaliser of
    softmax(inv_temp * z)."""
    out = []
    for z0, y in zip(rows, targets):
        z = [inv_temp * x for x in z0]
        top = max(z)
        norm = top + math.log(math.fsum(math.exp(x - top) for x in z))
        probs = [math.exp(x - norm) for x in z]
        ent = -math.fsum(p * math.log(p) for p in probs if p > 0.0)
        out.append((z[y] - norm, ent, norm))
    return out


def step_means(H, off):
    """Sec. 4.3: mean token entropy per step; float32 rounding of the mean is
    applied by the caller through ``_to_f32`` (the decision precision)."""
    return [math.fsum(H[off[s]:off[s + 1]]) / (off[s + 1] - off[s]) for s in range(len(off) - 1)]


def _to_f32(x):
    import struct

    return struct.unpack("f", struct.pack("f", x))[0]


def kept_count(S, rho):
    return min(S, max(0, math.ceil(rho * S - 1e-6)))


def select(Hs, rho):
    """Top-k by float32 step entropy, ties to the lower index: sort by
    (-entropy, index) and keep the first k."""
    keys = [_to_f32(h) for h in Hs]
    k = kept_count(len(keys), rho)
    order = sorted(range(len(keys)), key=lambda s: (-keys[s], s))
    keep = set(order[:k])
    return [1 if s in keep else 0 for s in range(len(keys))], k


def loss_and_coef(logp, lp_old, lp_roll, adv, off, mask, eps_low, eps_high, C):
    """Eq. (2) without the KL term, token mean over kept tokens; returns
    (L, g) with g_t = dL/dlogp_t."""
    step_of = []
    for s in range(len(off) - 1):
        step_of += [s] * (off[s + 1] - off[s])
    kept = [t for t in range(len(logp)) if mask[step_of[t]]]
    N = len(kept)
    terms, coef = [], [0.0] * len(logp)
    if N == 0:
        return 0.0, coef
    for t in kept:
        ratio = math.exp(logp[t] - lp_old[t])
        weight = min(math.exp(lp_old[t] - lp_roll[t]), C)
        clipped = min(max(ratio, 1.0 - eps_low), 1.0 + eps_high)
        a = adv[t]
        unclipped_term, clipped_term = ratio * a, clipped * a
        terms.append(-weight * min(unclipped_term, clipped_term) / N)
        if unclipped_term <= clipped_term:
            coef[t] = -weight * a * ratio / N
    return math.fsum(terms), coef


def grad_rows(rows, targets, norms, coef, inv_temp=1.0):
    """dL/dz_{t,v} = inv_temp g_t (delta_{v,y} - p_v)."""
    out = []
    for z, y, norm, gt in zip(rows, targets, norms, coef):
        out.append([inv_temp * gt * ((1.0 if v == y else 0.0) - math.exp(inv_temp * x - norm))
                    for v, x in enumerate(z)])
    return out


def _kl(kind, delta):
    """(value, d value / d logp) of the KL estimator; delta = lp_ref - logp."""
    if kind == "k1":
        return -delta, 1.0
    if kind == "k2":
        return 0.5 * delta * delta, -delta
    if kind == "k3":
        return math.exp(delta) - delta - 1.0, 1.0 - math.exp(delta)
    return 0.0, 0.0


def loss_ex(logp, lp_old, lp_roll, lp_ref, adv, off, mask, eps_low, eps_high, C, kl="none",
            beta=0.0, agg="token_mean", ratio="token"):
    """Eq. (2) with the KL term, an aggregation weight per token and a token- or
    step-level ratio; returns (L, g)."""
    T = len(logp)
    steps = [(off[s], off[s + 1]) for s in range(len(off) - 1)]
    kept = [s for s in range(len(steps)) if mask[s]]
    N = sum(steps[s][1] - steps[s][0] for s in kept)
    K = len(kept)
    terms, coef = [], [0.0] * T
    for s in kept:
        b, e = steps[s]
        n = e - b
        om = {"token_mean": 1.0 / N if N else 0.0, "token_mean_all": 1.0 / T,
              "step_mean": 1.0 / (K * n) if K else 0.0}[agg]
        if ratio == "token":
            units = [([t], om, 1.0) for t in range(b, e)]
        else:
            units = [(list(range(b, e)), om * n, 1.0 / n if ratio == "step_geomean" else 1.0)]
        for toks, weight, dlog in units:
            lr = math.fsum(logp[t] - lp_old[t] for t in toks)
            lw = math.fsum(lp_old[t] - lp_roll[t] for t in toks)
            if ratio == "step_geomean":
                lr, lw = lr / len(toks), lw / len(toks)
            a = math.fsum(adv[t] for t in toks) / len(toks)
            r, w = math.exp(lr), min(math.exp(lw), C)
            clipped = min(max(r, 1.0 - eps_low), 1.0 + eps_high)
            unclipped_term, clipped_term = r * a, clipped * a
            terms.append(-weight * w * min(unclipped_term, clipped_term))
            for t in toks:
                if unclipped_term <= clipped_term:
                    coef[t] -= weight * w * r * a * dlog
        for t in range(b, e):
            if kl != "none":
                val, dval = _kl(kl, lp_ref[t] - logp[t])
                terms.append(om * beta * val)
                coef[t] += om * beta * dval
    return math.fsum(terms), coef


def forward_backward(rows, targets, lp_old, lp_roll, adv, off, rho, eps_low, eps_high, C):
    st = token_stats(rows, targets)
    logp = [s[0] for s in st]
    H = [s[1] for s in st]
    lse = [s[2] for s in st]
    Hs = step_means(H, off)
    mask, k = select(Hs, rho)
    L, g = loss_and_coef(logp, lp_old, lp_roll, adv, off, mask, eps_low, eps_high, C)
    dz = grad_rows(rows, targets, lse, g)
    return dict(logp=logp, H=H, lse=lse, Hs=Hs, mask=mask, k=k, L=L, g=g, dz=dz)
