"""Counter-based generator and workload recipes (numpy reference definition).

Nothing here computes any part of the method: the generator only draws random
numbers and arranges them into the inputs of one policy-update call.

Generator
---------
Every random number is a pure function of ``(seed, stream, row, col)``::

    x = (seed * PHI64 mod 2^64) XOR (stream << 56 | row << 28 | col)
    h = splitmix64(x)
    normal  = Q[h >> 48],   Q[i] = inverse standard-normal CDF of (i + 0.5) / 65536
    uniform = ((h >> 40) + 0.5) / 2^24          (strictly inside (0, 1))

``splitmix64`` is Steele, Lea and Flood's SplitMix64 finaliser (OOPSLA 2014).
``Q`` is built once with ``statistics.NormalDist().inv_cdf`` (pure-Python
IEEE double arithmetic, so the same table on every machine); its tails end at
+-4.3249.

Streams: 0 logits, 1 target id, 2 target spike, 3 step lengths, 4 advantages,
5 old-policy offset, 6 rollout-policy offset, 7 row type / one-hot column,
8 reference-policy offset.

Logits
------
Row ``t`` draws its random numbers from row ``src_row[t]`` (rows that must be
identical share a source row).  Element ``v`` is, in IEEE double::

    base  = sigma * Q[h(seed, 0, src_row[t], v) >> 48]   for Gaussian rows, else 0.0
    value = base + (spike_val[t] if v == spike_col[t] else 0.0)

then rounded to float32 (round-to-nearest-even) and, for bf16 workloads, from
float32 to bfloat16 (round-to-nearest-even).  The C and HIP twins evaluate the
same two double operations with contraction disabled.
"""

from __future__ import annotations

import math
import statistics
from dataclasses import dataclass, field
from functools import lru_cache

import numpy as np

MASK64 = (1 << 64) - 1
PHI64 = 0x9E3779B97F4A7C15

STREAM_LOGITS = 0
STREAM_TARGET = 1
STREAM_SPIKE = 2
STREAM_LENGTH = 3
STREAM_ADV = 4
STREAM_OLD = 5
STREAM_ROLL = 6
STREAM_ROWTYPE = 7
STREAM_REF = 8
STREAM_HIDDEN = 9   # LM-head inputs: hidden states h [T, d]
STREAM_WEIGHT = 10  # LM-head weight W [V, d]

KIND_GAUSS = 0
KIND_FLAT = 1
KIND_ONEHOT = 2

_U64 = np.uint64


@lru_cache(maxsize=1)
def normal_table() -> np.ndarray:
    """``Q[i] = Phi^{-1}((i + 0.5) / 65536)`` as float64, 65536 entries."""
    nd = statistics.NormalDist()
    q = np.array([nd.inv_cdf((i + 0.5) / 65536.0) for i in range(65536)], dtype=np.float64)
    q.setflags(write=False)
    return q


def _splitmix64(x: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        x = x + _U64(0x9E3779B97F4A7C15)
        x = (x ^ (x >> _U64(30))) * _U64(0xBF58476D1CE4E5B9)
        x = (x ^ (x >> _U64(27))) * _U64(0x94D049BB133111EB)
        return x ^ (x >> _U64(31))


def base_key(seed: int) -> int:
    return (int(seed) * PHI64) & MASK64


def counter_hash(seed: int, stream: int, row, col) -> np.ndarray:
    """SplitMix64 of the packed counter; ``row`` and ``col`` broadcast."""
    row = np.asarray(row, dtype=np.uint64)
    col = np.asarray(col, dtype=np.uint64)
    if np.any(row >= _U64(1 << 28)) or np.any(col >= _U64(1 << 28)):
        raise ValueError("row and col must be below 2^28")
    if not 0 <= stream < 256:
        raise ValueError("stream must be below 256")
    x = _U64(base_key(seed)) ^ ((_U64(stream) << _U64(56)) | (row << _U64(28)) | col)
    return _splitmix64(x)


def draw_normal(seed: int, stream: int, row, col) -> np.ndarray:
    return normal_table()[(counter_hash(seed, stream, row, col) >> _U64(48)).astype(np.int64)]


def stream_key(seed: int, stream: int) -> int:
    """The key whose XOR with (row << 28 | col) addresses stream ``stream``:
    counter_hash(seed, stream, row, col) == splitmix64(stream_key ^ (row << 28 | col))."""
    return base_key(seed) ^ (stream << 56)


def gaussian_bits(seed: int, stream: int, rows: int, cols: int, sigma: float,
                  row0: int = 0) -> np.ndarray:
    """bf16 bit patterns [rows, cols] of the matrix whose element (r, c) is
    sigma * Q[hash(seed, stream, row0 + r, c) >> 48] in double, rounded to
    float32 and then to bf16 (nearest even): the LM-head inputs."""
    r = np.arange(row0, row0 + rows, dtype=np.uint64)[:, None]
    c = np.arange(cols, dtype=np.uint64)[None, :]
    vals = sigma * draw_normal(seed, stream, r, c)
    return f32_to_bf16_bits(vals.astype(np.float32))


def draw_uniform(seed: int, stream: int, row, col) -> np.ndarray:
    h = counter_hash(seed, stream, row, col)
    return ((h >> _U64(40)).astype(np.float64) + 0.5) / float(1 << 24)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round-to-nearest-even (finite inputs;
    NaN stays a quiet NaN)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if np.any(nan):
        rounded = np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), rounded)
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass
class Workload:
    """All inputs of one policy-update call, as a recipe (not materialised)."""

    name: str
    T: int
    V: int
    dtype: str  # "f32" or "bf16"
    off: np.ndarray  # int32 [S+1], step offsets
    rho: float
    eps_low: float
    eps_high: float
    C: float
    inplace: bool
    seed: int
    sigma: float
    kind: np.ndarray  # int32 [T]
    src_row: np.ndarray  # int32 [T]
    spike_col: np.ndarray  # int32 [T], -1 = none
    spike_val: np.ndarray  # float64 [T]
    target: np.ndarray  # int32 [T]
    adv: np.ndarray  # float32 [T]
    old_offset: np.ndarray  # float64 [T]: lp_old = logp_new + old_offset
    roll_offset: np.ndarray  # float64 [T]: lp_roll = lp_old + roll_offset
    ref_offset: np.ndarray = None  # float64 [T]: lp_ref = logp_new + ref_offset
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def S(self) -> int:
        return int(self.off.shape[0] - 1)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def step_of_token(self) -> np.ndarray:
        lens = np.diff(self.off.astype(np.int64))
        return np.repeat(np.arange(self.S, dtype=np.int64), lens)


def _uniform_int(seed, stream, row, col, lo, hi):
    """Integer uniform on [lo, hi] (inclusive); the product is exact in double."""
    u = draw_uniform(seed, stream, row, col)
    return lo + np.floor(u * (hi - lo + 1)).astype(np.int64)


def _step_lengths(seed, S, lo, hi, T_exact=None):
    lens = _uniform_int(seed, STREAM_LENGTH, np.arange(S), 0, lo, hi)
    if T_exact is not None:
        total = int(lens.sum())
        it = 0
        while total != T_exact:
            j = int(_uniform_int(seed, STREAM_LENGTH, it % (1 << 28), 1 + it // (1 << 28), 0, S - 1))
            if total > T_exact and lens[j] > lo:
                lens[j] -= 1
                total -= 1
            elif total < T_exact and lens[j] < hi:
                lens[j] += 1
                total += 1
            it += 1
    return lens


def _offsets(lens) -> np.ndarray:
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    if off[-1] >= (1 << 31):
        raise ValueError("T must fit in int32")
    return off.astype(np.int32)


def _gauss_noise_offsets(seed, T, old_std=0.05, roll_std=0.1):
    t = np.arange(T)
    return old_std * draw_normal(seed, STREAM_OLD, t, 0), roll_std * draw_normal(seed, STREAM_ROLL, t, 0)


def _build(name, *, seed, V, dtype, lens, rho, eps_low, eps_high, C, inplace, sigma,
           spike, adv_mode, steps_per_traj=None, kind=None, src_row=None,
           spike_col=None, spike_val=None, offsets=None, description=""):
    off = _offsets(lens)
    T = int(off[-1])
    S = len(lens)
    t = np.arange(T, dtype=np.int64)
    if src_row is None:
        src_row = t.copy()
    if kind is None:
        kind = np.full(T, KIND_GAUSS, dtype=np.int64)
    target = np.floor(draw_uniform(seed, STREAM_TARGET, src_row, 0) * V).astype(np.int64)
    if spike_col is None:
        spike_col = target.copy()
    if spike_val is None:
        if spike == "uniform_2_8":
            spike_val = 2.0 + 6.0 * draw_uniform(seed, STREAM_SPIKE, src_row, 0)
        else:
            spike_val = np.full(T, float(spike), dtype=np.float64)
    step = np.repeat(np.arange(S, dtype=np.int64), lens)
    if adv_mode == "step":
        adv = draw_normal(seed, STREAM_ADV, step, 0)
    elif adv_mode == "trajectory":
        adv = draw_normal(seed, STREAM_ADV, step // steps_per_traj, 1)
    else:
        raise ValueError(adv_mode)
    if offsets is None:
        old_off, roll_off = _gauss_noise_offsets(seed, T)
    else:
        old_off, roll_off = offsets(seed, T)
    return Workload(
        name=name, T=T, V=V, dtype=dtype, off=off, rho=rho, eps_low=eps_low,
        eps_high=eps_high, C=C, inplace=inplace, seed=seed, sigma=sigma,
        kind=np.asarray(kind, dtype=np.int32), src_row=np.asarray(src_row, dtype=np.int32),
        spike_col=np.asarray(spike_col, dtype=np.int32),
        spike_val=np.asarray(spike_val, dtype=np.float64),
        target=target.astype(np.int32), adv=adv.astype(np.float32),
        old_offset=np.asarray(old_off, dtype=np.float64),
        roll_offset=np.asarray(roll_off, dtype=np.float64),
        ref_offset=0.05 * draw_normal(seed, STREAM_REF, t, 0),
        description=description,
    )


def _tiny():
    return _build(
        "tiny", seed=0, V=4096, dtype="f32", lens=np.full(16, 32), rho=0.5, eps_low=0.2,
        eps_high=0.2, C=2.0, inplace=False, sigma=2.0, spike=4.0, adv_mode="step",
        description="T=512 in 16 steps of 32, V=4096 fp32, logits N(0,2^2) + 4 at target")


def _vlm7b():
    lens = _step_lengths(1, 64, 16, 128, T_exact=4096)
    return _build(
        "vlm7b", seed=1, V=152064, dtype="bf16", lens=lens, rho=0.8, eps_low=0.2, eps_high=0.2,
        C=2.0, inplace=False, sigma=3.0, spike="uniform_2_8", adv_mode="step",
        description="T=4096 in 64 steps U[16,128], V=152064 bf16, logits N(0,3^2) + U(2,8) at target")


def _microbatch():
    lens = _step_lengths(2, 8 * 30, 32, 256)
    return _build(
        "microbatch", seed=2, V=152064, dtype="bf16", lens=lens, rho=0.8, eps_low=0.2,
        eps_high=0.2, C=2.0, inplace=False, sigma=3.0, spike="uniform_2_8",
        adv_mode="trajectory", steps_per_traj=30,
        description="8 trajectories x 30 steps U[32,256], V=152064 bf16")


def _longhorizon():
    lens = _step_lengths(3, 32 * 50, 32, 160)
    return _build(
        "longhorizon", seed=3, V=152064, dtype="bf16", lens=lens, rho=0.5, eps_low=0.28,
        eps_high=0.28, C=5.0, inplace=True, sigma=3.0, spike="uniform_2_8",
        adv_mode="trajectory", steps_per_traj=50,
        description="32 trajectories x 50 steps U[32,160], V=152064 bf16, in-place gradient")


def _edge_offsets(seed, T):
    t = np.arange(T)
    ratio = 0.5 + draw_uniform(seed, STREAM_OLD, t, 0)  # r = U(0.5, 1.5)
    d = -3.0 + 6.0 * draw_uniform(seed, STREAM_ROLL, t, 0)  # lp_old - lp_roll = U(-3, 3)
    return -np.log(ratio), -d


def edge_layout(S=256, steps_per_block=4, tokens_per_step=64, V=151936, seed=4):
    """Row kinds for the edge workload: blocks of 4 steps cycle through
    Gaussian (every other Gaussian block = 4 copies of one step), flat (all
    logits 0) and near-one-hot (zeros and +30 at one column)."""
    T = S * tokens_per_step
    t = np.arange(T, dtype=np.int64)
    step = t // tokens_per_step
    block = step // steps_per_block
    btype = block % 3
    kind = np.where(btype == 0, KIND_GAUSS, np.where(btype == 1, KIND_FLAT, KIND_ONEHOT))
    copies = (btype == 0) & ((block // 3) % 2 == 1)
    first_step = block * steps_per_block
    src_row = np.where(copies, first_step * tokens_per_step + (t % tokens_per_step), t)
    target = np.floor(draw_uniform(seed, STREAM_TARGET, src_row, 0) * V).astype(np.int64)
    spike_val = np.where(kind == KIND_GAUSS, 2.0 + 6.0 * draw_uniform(seed, STREAM_SPIKE, src_row, 0),
                         np.where(kind == KIND_ONEHOT, 30.0, 0.0))
    on_target = draw_uniform(seed, STREAM_ROWTYPE, src_row, 1) < 0.5
    other_col = np.floor(draw_uniform(seed, STREAM_ROWTYPE, src_row, 2) * V).astype(np.int64)
    spike_col = np.where(kind == KIND_GAUSS, target,
                         np.where(kind == KIND_ONEHOT, np.where(on_target, target, other_col), -1))
    return kind, src_row, spike_col, spike_val


def _edge():
    S, per = 256, 64
    kind, src_row, spike_col, spike_val = edge_layout(S=S, tokens_per_step=per)
    return _build(
        "edge", seed=4, V=151936, dtype="bf16", lens=np.full(S, per), rho=0.25, eps_low=0.2,
        eps_high=0.2, C=2.0, inplace=False, sigma=3.0, spike=None, adv_mode="step",
        kind=kind, src_row=src_row, spike_col=spike_col, spike_val=spike_val,
        offsets=_edge_offsets,
        description="T=16384 in 256 steps of 64, V=151936 bf16; Gaussian, flat and "
                    "near-one-hot rows, exact-tie step blocks, ratios U(0.5,1.5), "
                    "lp_old-lp_roll U(-3,3)")


class LmHeadProblem:
    """An LM-head workload: the step structure, targets, advantages and
    log-prob offsets of a logits workload, with the logits replaced by
    h W^T: h [T, d] ~ N(0, sigma_h^2), W [V, d] ~ N(0, sigma_w^2), bf16, so
    that z ~ N(0, d sigma_h^2 sigma_w^2)."""

    def __init__(self, wl: "Workload", d: int, sigma_h: float, sigma_w: float, description: str):
        self.wl, self.d, self.sigma_h, self.sigma_w = wl, d, sigma_h, sigma_w
        self.name = "lmhead_" + wl.name
        self.description = description

    def hidden_bits(self, rows=None):
        wl = self.wl
        if rows is None:
            return gaussian_bits(wl.seed, STREAM_HIDDEN, wl.T, self.d, self.sigma_h)
        return np.concatenate([gaussian_bits(wl.seed, STREAM_HIDDEN, 1, self.d, self.sigma_h, int(r))
                               for r in rows]) if len(rows) else np.zeros((0, self.d), np.uint16)

    def weight_bits(self):
        return gaussian_bits(self.wl.seed, STREAM_WEIGHT, self.wl.V, self.d, self.sigma_w)


def lmhead_problem(name: str, d: int | None = None) -> LmHeadProblem:
    """The LM-head version of a named logits workload: d = 3584 (the 7B VLM's
    hidden size) unless given; sigma_h = 1, sigma_w = 3 / sqrt(d) so that the
    logits have the N(0, 3^2) spread of the logits workloads."""
    wl = make_workload(name)
    d = 3584 if d is None else d
    return LmHeadProblem(wl, d, 1.0, 3.0 / math.sqrt(d),
                         f"h [T={wl.T}, d={d}] N(0,1), W [V={wl.V}, d] N(0, 9/d), bf16; "
                         f"steps, targets and advantages of {wl.name}")


def lmhead_custom(lens, V, d, seed, **kw) -> LmHeadProblem:
    wl = custom_workload(lens=lens, V=V, dtype="bf16", seed=seed, **kw)
    return LmHeadProblem(wl, d, 1.0, 3.0 / math.sqrt(d), f"custom T={wl.T}, d={d}, V={V}")


WORKLOADS = {
    "tiny": _tiny,
    "vlm7b": _vlm7b,
    "microbatch": _microbatch,
    "longhorizon": _longhorizon,
    "edge": _edge,
}


@lru_cache(maxsize=None)
def make_workload(name: str) -> Workload:
    return WORKLOADS[name]()


def custom_workload(*, lens, V, dtype="bf16", seed=11, rho=0.8, eps_low=0.2, eps_high=0.28,
                    C=2.0, sigma=3.0, spike="uniform_2_8", adv_mode="step", steps_per_traj=None,
                    mix_kinds=False, ratio_spread=False, inplace=False, name="custom"):
    """A small workload of the same recipe for parity tests (ragged shapes).

    ``mix_kinds`` cycles rows through Gaussian, flat and near-one-hot kinds per
    step; ``ratio_spread`` uses the wide ratio/offset model of the edge workload.
    """
    lens = np.asarray(lens, dtype=np.int64)
    kind = src_row = spike_col = spike_val = None
    if mix_kinds:
        T = int(lens.sum())
        t = np.arange(T, dtype=np.int64)
        step = np.repeat(np.arange(len(lens)), lens)
        k = step % 3
        kind = np.where(k == 0, KIND_GAUSS, np.where(k == 1, KIND_FLAT, KIND_ONEHOT))
        src_row = t
        target = np.floor(draw_uniform(seed, STREAM_TARGET, t, 0) * V).astype(np.int64)
        on_target = draw_uniform(seed, STREAM_ROWTYPE, t, 1) < 0.5
        other_col = np.floor(draw_uniform(seed, STREAM_ROWTYPE, t, 2) * V).astype(np.int64)
        spike_col = np.where(kind == KIND_GAUSS, target,
                             np.where(kind == KIND_ONEHOT, np.where(on_target, target, other_col), -1))
        spike_val = np.where(kind == KIND_GAUSS, 2.0 + 6.0 * draw_uniform(seed, STREAM_SPIKE, t, 0),
                             np.where(kind == KIND_ONEHOT, 30.0, 0.0))
    return _build(
        name, seed=seed, V=V, dtype=dtype, lens=lens, rho=rho, eps_low=eps_low,
        eps_high=eps_high, C=C, inplace=inplace, sigma=sigma, spike=spike, adv_mode=adv_mode,
        steps_per_traj=steps_per_traj, kind=kind, src_row=src_row, spike_col=spike_col,
        spike_val=spike_val, offsets=_edge_offsets if ratio_spread else None)


def logits_rows_numpy(wl: Workload, rows) -> np.ndarray:
    """Logits of the given rows, shape [len(rows), V]: float32 values for f32
    workloads, bfloat16 bit patterns (uint16) for bf16 workloads."""
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    V = wl.V
    cols = np.arange(V, dtype=np.int64)
    out = np.empty((rows.size, V), dtype=np.float32)
    q = normal_table()
    for i, t in enumerate(rows):
        kind = int(wl.kind[t])
        if kind == KIND_GAUSS:
            h = counter_hash(wl.seed, STREAM_LOGITS, int(wl.src_row[t]), cols)
            base = wl.sigma * q[(h >> _U64(48)).astype(np.int64)]
        else:
            base = np.zeros(V, dtype=np.float64)
        spike = np.zeros(V, dtype=np.float64)
        sc = int(wl.spike_col[t])
        if sc >= 0:
            spike[sc] = wl.spike_val[t]
        out[i] = (base + spike).astype(np.float32)
    if wl.dtype == "bf16":
        return f32_to_bf16_bits(out)
    return out


def reference_logprobs(wl: Workload, logp_new: np.ndarray):
    """Reference-policy log-probs of the targets, float32:
    ``lp_ref = fl32(logp_new + ref_offset)`` (offsets 0.05 N(0,1))."""
    return (np.asarray(logp_new, dtype=np.float64) + wl.ref_offset).astype(np.float32)


def perturbed_logprobs(wl: Workload, logp_new: np.ndarray):
    """Old-policy and rollout-policy log-probs of the targets, as float32:
    ``lp_old = fl32(logp_new + old_offset)``, ``lp_roll = fl32(lp_old + roll_offset)``.

    ``logp_new`` is the caller's float64 log-prob of each target under the
    generated logits (the perturbation model of the workload description)."""
    logp_new = np.asarray(logp_new, dtype=np.float64)
    lp_old = (logp_new + wl.old_offset).astype(np.float32)
    lp_roll = (lp_old.astype(np.float64) + wl.roll_offset).astype(np.float32)
    return lp_old, lp_roll
