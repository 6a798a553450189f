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


def token_stats(rows, targets):
    """Sec. 4.3: per row, log-prob of the target, entropy and log-normaliser."""
    out = []
    for z, y in zip(rows, targets):
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


def grad_rows(rows, targets, norms, coef):
    """dL/dz_{t,v} = g_t (delta_{v,y} - p_v)."""
    out = []
    for z, y, norm, gt in zip(rows, targets, norms, coef):
        out.append([gt * ((1.0 if v == y else 0.0) - math.exp(x - norm)) for v, x in enumerate(z)])
    return out


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
