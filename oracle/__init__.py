"""Float64 CPU oracle of the DART policy-update hot path.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the product package.
It shares no code with the HIP path.

Two independent implementations live here:

* ``liboracle.so`` built from ``dart_oracle.c`` (float64, OpenMP over rows),
  wrapped by the functions of this module;
* ``oracle.mini``, pure Python with ``math`` only, for tiny shapes.

Both follow the paper's definitions (DART, arXiv 2509.23866): token entropy and
log-prob (Sec. 4.3, Eq. 1), the step mean entropy and the top-rho step mask
(Sec. 4.3, the indicator of Eq. 2), the truncated importance-sampling weight
(Sec. 4.4) and the clipped surrogate of Eq. (2), and the gradient of the loss
with respect to the logits. Every function is pinned by the ``-m "not gpu"``
tests in ``tests/test_oracle_*.py`` against closed forms, invariants, brute
force, a library routine and finite differences.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB lets the mutation tests load a deliberately broken build
LIB = os.environ.get("ORACLE_LIB") or os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "dart_oracle.c")


def build(verbose: bool = False, src: str = SRC, out: str = os.path.join(HERE, "liboracle.so")) -> None:
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", src, "-o", out, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_D = ctypes.c_double


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"{LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB)
        lib.oracle_token_stats_ex.restype = None
        lib.oracle_token_stats_ex.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _D, _P, _P,
                                              _P, ctypes.c_int]
        lib.oracle_tis_loss_ex.restype = _D
        lib.oracle_tis_loss_ex.argtypes = [_I64, _P, _P, _P, _P, _P, _P, _I64, _P, _D, _D, _D,
                                           ctypes.c_int, _D, ctypes.c_int, ctypes.c_int, _P, _P,
                                           _P, _P]
        lib.oracle_dlogits_ex.restype = None
        lib.oracle_dlogits_ex.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _D,
                                          _P, ctypes.c_int]
        lib.oracle_grpo_advantage.restype = None
        lib.oracle_grpo_advantage.argtypes = [_P, _P, _I64, _P, _I64, _P, _P, _P, _P]
        lib.oracle_token_stats.restype = None
        lib.oracle_token_stats.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P,
                                           ctypes.c_int]
        lib.oracle_step_entropy.restype = None
        lib.oracle_step_entropy.argtypes = [_P, _P, _I64, _P, _P]
        lib.oracle_kept_steps.restype = _I64
        lib.oracle_kept_steps.argtypes = [_I64, _D]
        lib.oracle_step_mask.restype = _I64
        lib.oracle_step_mask.argtypes = [_P, _I64, _D, _P]
        lib.oracle_tis_loss.restype = _D
        lib.oracle_tis_loss.argtypes = [_I64, _P, _P, _P, _P, _P, _I64, _P, _D, _D, _D, _P, _P,
                                        _P, _P]
        lib.oracle_dlogits.restype = None
        lib.oracle_dlogits.argtypes = [_P, ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P,
                                       ctypes.c_int]
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _logits_arg(z):
    """float32 array -> dtype 0; uint16 (bfloat16 bit patterns) -> dtype 1;
    float64 -> dtype 2."""
    z = np.asarray(z)
    if z.ndim != 2 or z.strides[1] != z.itemsize:
        raise ValueError("logits must be a 2-D array with contiguous rows")
    if z.dtype == np.float32:
        return z, 0
    if z.dtype == np.uint16:
        return z, 1
    if z.dtype == np.float64:
        return z, 2
    raise TypeError("logits must be float32, float64 or bfloat16 bit patterns (uint16)")


def token_stats(z, target, nthreads=None, inv_temp=1.0):
    """Per-row (logp, H, lse) in float64 for logits rows ``z`` [n, V], of the
    distribution softmax(inv_temp * z)."""
    lib = _load()
    z, dt = _logits_arg(z)
    n, V = z.shape
    ld = z.strides[0] // z.itemsize
    target = _c(target, np.int32)
    assert target.shape == (n,)
    logp = np.empty(n, np.float64)
    H = np.empty(n, np.float64)
    lse = np.empty(n, np.float64)
    if inv_temp == 1.0:
        lib.oracle_token_stats(z.ctypes.data, dt, n, V, ld, target.ctypes.data, logp.ctypes.data,
                               H.ctypes.data, lse.ctypes.data, nthreads or default_threads())
    else:
        lib.oracle_token_stats_ex(z.ctypes.data, dt, n, V, ld, target.ctypes.data,
                                  float(inv_temp), logp.ctypes.data, H.ctypes.data,
                                  lse.ctypes.data, nthreads or default_threads())
    return logp, H, lse


def step_entropy(H, off):
    """(Hs float64 [S], Hs32 float32 [S]) for token entropies H and offsets off."""
    lib = _load()
    H = _c(H, np.float64)
    off = _c(off, np.int32)
    S = off.size - 1
    Hs = np.empty(S, np.float64)
    Hs32 = np.empty(S, np.float32)
    lib.oracle_step_entropy(H.ctypes.data, off.ctypes.data, S, Hs.ctypes.data, Hs32.ctypes.data)
    return Hs, Hs32


def kept_steps(S, rho):
    return int(_load().oracle_kept_steps(int(S), float(rho)))


def step_mask(Hs32, rho):
    """(mask uint8 [S], k) decided on the float32 step entropies."""
    lib = _load()
    Hs32 = _c(Hs32, np.float32)
    mask = np.empty(Hs32.size, np.uint8)
    k = lib.oracle_step_mask(Hs32.ctypes.data, Hs32.size, float(rho), mask.ctypes.data)
    return mask, int(k)


def tis_loss(logp, lp_old, lp_roll, adv, off, mask, eps_low, eps_high, C):
    """Returns dict(L, g, ell, boundary, stats)."""
    lib = _load()
    logp = _c(logp, np.float64)
    T = logp.size
    lp_old = _c(lp_old, np.float32)
    lp_roll = _c(lp_roll, np.float32)
    adv = _c(adv, np.float32)
    off = _c(off, np.int32)
    mask = _c(mask, np.uint8)
    S = off.size - 1
    assert lp_old.size == T and lp_roll.size == T and adv.size == T and mask.size == S
    assert off[0] == 0 and off[-1] == T
    g = np.empty(T, np.float64)
    ell = np.empty(T, np.float64)
    boundary = np.empty(T, np.uint8)
    stats = np.empty(4, np.float64)
    L = lib.oracle_tis_loss(T, logp.ctypes.data, lp_old.ctypes.data, lp_roll.ctypes.data,
                            adv.ctypes.data, off.ctypes.data, S, mask.ctypes.data,
                            float(eps_low), float(eps_high), float(C), g.ctypes.data,
                            ell.ctypes.data, boundary.ctypes.data, stats.ctypes.data)
    return dict(L=float(L), g=g, ell=ell, boundary=boundary.astype(bool), stats=stats)


KL = {"none": 0, "k1": 1, "k2": 2, "k3": 3}
AGG = {"token_mean": 0, "token_mean_all": 1, "step_mean": 2}
RATIO = {"token": 0, "step_geomean": 1, "step_product": 2}


def tis_loss_ex(logp, lp_old, lp_roll, adv, off, mask, eps_low, eps_high, C, lp_ref=None,
                kl="none", beta=0.0, agg="token_mean", ratio="token"):
    """The loss with the KL term, aggregation and ratio level selectable.
    Returns dict(L, g, ell, boundary, stats[6])."""
    lib = _load()
    logp = _c(logp, np.float64)
    T = logp.size
    lp_old = _c(lp_old, np.float32)
    lp_roll = _c(lp_roll, np.float32)
    adv = _c(adv, np.float32)
    off = _c(off, np.int32)
    mask = _c(mask, np.uint8)
    S = off.size - 1
    if KL[kl] != 0:
        lp_ref = _c(lp_ref, np.float32)
        assert lp_ref.size == T
    assert lp_old.size == T and lp_roll.size == T and adv.size == T and mask.size == S
    assert off[0] == 0 and off[-1] == T
    g = np.empty(T, np.float64)
    ell = np.empty(T, np.float64)
    boundary = np.empty(T, np.uint8)
    stats = np.empty(6, np.float64)
    L = lib.oracle_tis_loss_ex(T, logp.ctypes.data, lp_old.ctypes.data, lp_roll.ctypes.data,
                               None if KL[kl] == 0 else lp_ref.ctypes.data, adv.ctypes.data,
                               off.ctypes.data, S, mask.ctypes.data, float(eps_low),
                               float(eps_high), float(C), KL[kl], float(beta), AGG[agg],
                               RATIO[ratio], g.ctypes.data, ell.ctypes.data, boundary.ctypes.data,
                               stats.ctypes.data)
    return dict(L=float(L), g=g, ell=ell, boundary=boundary.astype(bool), stats=stats)


def dlogits(z, target, lse, logp, g, nthreads=None, inv_temp=1.0):
    """float64 [n, V] gradient rows for logits rows ``z`` (``lse`` and ``logp``
    of the same rows from token_stats)."""
    lib = _load()
    z, dt = _logits_arg(z)
    n, V = z.shape
    ld = z.strides[0] // z.itemsize
    target = _c(target, np.int32)
    lse = _c(lse, np.float64)
    logp = _c(logp, np.float64)
    g = _c(g, np.float64)
    assert lse.shape == (n,) and logp.shape == (n,) and g.shape == (n,)
    out = np.empty((n, V), np.float64)
    if inv_temp == 1.0:
        lib.oracle_dlogits(z.ctypes.data, dt, n, V, ld, target.ctypes.data, lse.ctypes.data,
                           logp.ctypes.data, g.ctypes.data, out.ctypes.data,
                           nthreads or default_threads())
    else:
        lib.oracle_dlogits_ex(z.ctypes.data, dt, n, V, ld, target.ctypes.data, lse.ctypes.data,
                              logp.ctypes.data, g.ctypes.data, float(inv_temp), out.ctypes.data,
                              nthreads or default_threads())
    return out


def forward_backward(z, target, lp_old, lp_roll, adv, off, rho, eps_low, eps_high, C,
                     nthreads=None, mask=None):
    """The whole path on full logits: stats -> step entropy -> mask -> loss -> dlogits.
    ``mask`` may be given to skip the selection (it is then an input)."""
    logp, H, lse = token_stats(z, target, nthreads)
    Hs, Hs32 = step_entropy(H, off)
    if mask is None:
        mask, k = step_mask(Hs32, rho)
    else:
        k = int(np.sum(mask))
    res = tis_loss(logp, lp_old, lp_roll, adv, off, mask, eps_low, eps_high, C)
    dz = dlogits(z, target, lse, logp, res["g"], nthreads)
    res.update(logp=logp, H=H, lse=lse, Hs=Hs, Hs32=Hs32, mask=mask, k=k, dz=dz)
    return res


def grpo_advantage(reward, traj_off, grp_off, off):
    """Step-wise GRPO advantage per token (Sec. 3.3); returns (adv [T] float64,
    group_mean [G], group_std [G])."""
    lib = _load()
    reward = _c(reward, np.float32)
    traj_off = _c(traj_off, np.int32)
    grp_off = _c(grp_off, np.int32)
    off = _c(off, np.int32)
    n_traj, G = reward.size, grp_off.size - 1
    assert traj_off.size == n_traj + 1 and grp_off[-1] == n_traj
    assert traj_off[-1] == off.size - 1
    T = int(off[-1])
    adv = np.zeros(T, np.float64)
    mean = np.empty(G, np.float64)
    std = np.empty(G, np.float64)
    lib.oracle_grpo_advantage(reward.ctypes.data, traj_off.ctypes.data, n_traj, grp_off.ctypes.data,
                              G, off.ctypes.data, adv.ctypes.data, mean.ctypes.data, std.ctypes.data)
    return adv, mean, std


def step_mask_groups(Hs32, group_step_off, rho):
    """Top-k selection within each group of steps [group_step_off[g],
    group_step_off[g+1]) (Sec. 4.3 applied per task group): (mask, k per group)."""
    Hs32 = np.asarray(Hs32, np.float32)
    mask = np.zeros(Hs32.size, np.uint8)
    ks = []
    for g in range(len(group_step_off) - 1):
        a, b = int(group_step_off[g]), int(group_step_off[g + 1])
        m, k = step_mask(Hs32[a:b], rho)
        mask[a:b] = m
        ks.append(k)
    return mask, np.array(ks, np.int64)


def bf16_bits_to_f64(bits):
    """bfloat16 bit patterns (uint16) widened exactly to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def lmhead_logits(h_bits, w_bits):
    """z = h W^T in float64 from the bf16 hidden states h [T, d] and the LM-head
    weight W [V, d] (torch.nn.Linear's layout): the logits the LM head produces
    before any rounding, as one library matrix product of the exact inputs."""
    return np.ascontiguousarray(bf16_bits_to_f64(h_bits) @ bf16_bits_to_f64(w_bits).T)


def lmhead_token_stats(h_bits, w_bits, target, nthreads=None, inv_temp=1.0):
    """(logp, H, lse) of softmax(inv_temp h W^T) per row, in float64 (Sec. 4.3,
    Eq. 1 on the logits of the LM head; inv_temp is an inverse sampling
    temperature, 1 in the paper, App. A.4)."""
    return token_stats(lmhead_logits(h_bits, w_bits), target, nthreads=nthreads,
                       inv_temp=inv_temp)


def lmhead_grads(h_bits, w_bits, target, lse, logp, g, nthreads=None, inv_temp=1.0):
    """Gradients of the loss through the LM head, given the per-token
    coefficient g = dL/dlogp: dz = inv_temp g (onehot - p) [T, V] (the gradient
    of the logits h W^T, p = softmax(inv_temp h W^T)), dh = dz W [T, d] and
    dW = dz^T h [V, d], all in float64."""
    z = lmhead_logits(h_bits, w_bits)
    dz = dlogits(z, target, lse, logp, g, nthreads=nthreads, inv_temp=inv_temp)
    h = bf16_bits_to_f64(h_bits)
    w = bf16_bits_to_f64(w_bits)
    return dz, dz @ w, dz.T @ h


def f64_to_bf16_bits(x):
    """Correctly rounded (nearest-even) float64 -> bfloat16 bit patterns,
    including bfloat16 subnormals; used only to compare with bf16 outputs."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    ax = np.abs(x)
    sub = ax < 2.0 ** -126
    # normal range: round the double's 52-bit fraction to 7 bits
    u = x.view(np.uint64)
    half = np.uint64((1 << 44) - 1)
    r = (u + half + ((u >> np.uint64(45)) & np.uint64(1))) & ~np.uint64((1 << 45) - 1)
    f = r.view(np.float64).astype(np.float32)
    out[...] = (f.view(np.uint32) >> 16).astype(np.uint16)
    if np.any(sub):
        q = np.rint(x[sub] / 2.0 ** -133) * 2.0 ** -133  # rint is round-half-even
        out[sub] = (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return out


def bf16_ulp(bits):
    """Spacing of bfloat16 numbers at the magnitude of ``bits`` (float64)."""
    f = (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    a = np.abs(f.astype(np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.where(a < 2.0 ** -126, 2.0 ** -133, 2.0 ** (e - 7))
