"""Shared machinery of the parity tests: inputs, the oracle's side, the GPU's
side, and the comparisons at the tolerances of the specification:

* logp, entropy (and lse, step entropy): 2e-4 absolute;
* loss: 1e-4 relative;
* dlogits: at most 1 bfloat16 ulp of the oracle value (and 1e-2 absolute)
  per element, rows of clip-boundary tokens (ratio within 1e-4 of a clip
  bound, where the gate may legitimately differ) excluded;
* step mask: exactly k kept; identical to the oracle wherever the oracle's step
  entropy is more than 1e-5 away from the k-th largest; a valid top-k of the
  GPU's own step entropies with ties towards the lower index everywhere.

The oracle's inputs come from the generator only (host twin), never from the
GPU path. Old/rollout log-probs are the oracle's float64 logp of the generated
logits perturbed by the workload's offsets.
"""

from __future__ import annotations

import sys
import time

import numpy as np

import oracle
import synth
import synth.native as sn

LOGP_TOL = 2e-4
H_TOL = 2e-4
LOSS_RTOL = 1e-4
BAND = 1e-5


def log(msg):
    print(f"[parity] {msg}", file=sys.stderr, flush=True)


def f32(x):
    return float(np.float32(x))


# ---------------------------------------------------------------- oracle side

class OracleSide:
    """The oracle's view of a workload: token stats for every row (streamed
    in chunks from the host generator), inputs, selection and loss."""

    def __init__(self, wl: synth.Workload, chunk_rows: int = 1024, need_rows=True):
        t0 = time.time()
        self.wl = wl
        T = wl.T
        self.logp = np.empty(T)
        self.H = np.empty(T)
        self.lse = np.empty(T)
        dt = np.float32 if wl.dtype == "f32" else np.uint16
        buf = np.empty((min(chunk_rows, T), wl.V), dtype=dt)
        for r0 in range(0, T, chunk_rows):
            rows = np.arange(r0, min(T, r0 + chunk_rows))
            z = sn.logits_rows_host(wl, rows, out=buf[: rows.size])
            lp, h, ls = oracle.token_stats(z, wl.target[rows])
            self.logp[rows], self.H[rows], self.lse[rows] = lp, h, ls
        self.lp_old, self.lp_roll = synth.perturbed_logprobs(wl, self.logp)
        self.eps_low, self.eps_high, self.C = f32(wl.eps_low), f32(wl.eps_high), f32(wl.C)
        self.Hs, self.Hs32 = oracle.step_entropy(self.H, wl.off)
        self.mask, self.k = oracle.step_mask(self.Hs32, wl.rho)
        self.res = self.loss_with_mask(self.mask)
        log(f"oracle {wl.name}: T={T} V={wl.V} k={self.k} L={self.res['L']:.6g} "
            f"({time.time() - t0:.1f}s)")

    def loss_with_mask(self, mask):
        wl = self.wl
        return oracle.tis_loss(self.logp, self.lp_old, self.lp_roll, wl.adv, wl.off, mask,
                               self.eps_low, self.eps_high, self.C)

    def dz_rows(self, rows, g=None):
        wl = self.wl
        rows = np.asarray(rows, dtype=np.int64)
        z = sn.logits_rows_host(wl, rows)
        g = self.res["g"] if g is None else g
        return oracle.dlogits(z, wl.target[rows], self.lse[rows], self.logp[rows], g[rows])


# ---------------------------------------------------------------- GPU side

class GpuSide:
    """Device buffers of a workload (logits from the device twin of the
    generator) and one pass of the path through the C ABI."""

    def __init__(self, wl: synth.Workload, ors: OracleSide, ld=None, misalign=0, inplace=None):
        import torch

        import paper_2509_23866_amd as dart

        self.torch, self.dart, self.wl = torch, dart, wl
        dev = torch.device("cuda")
        tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
        ld = wl.V if ld is None else ld
        self.inplace = wl.inplace if inplace is None else inplace
        recipe = sn.DeviceRecipe(wl)
        if misalign:
            flat = torch.full((wl.T * ld + misalign,), float("nan"), dtype=tdt, device=dev)
            self.logits = flat[misalign:].view(wl.T, ld)
        else:
            self.logits = torch.full((wl.T, ld), float("nan"), dtype=tdt, device=dev)
        sn.fill_logits_device(recipe, self.logits)
        self.logits = self.logits[:, : wl.V] if ld != wl.V else self.logits
        self.target = torch.from_numpy(wl.target).to(dev)
        self.lp_old = torch.from_numpy(ors.lp_old).to(dev)
        self.lp_roll = torch.from_numpy(ors.lp_roll).to(dev)
        self.adv = torch.from_numpy(wl.adv).to(dev)
        self.off = torch.from_numpy(wl.off).to(dev)
        self.eps_low, self.eps_high, self.C = ors.eps_low, ors.eps_high, ors.C
        del recipe

    def run(self, mask=None, keep_rows=None, fused=True):
        """One pass; ``mask`` (numpy) replaces the GPU's own selection as the
        input of the loss call. With the GPU's own selection and ``fused`` the
        pass is the benchmark's: dart_tok_stats -> dart_select_tis_loss_fwd ->
        dart_tis_grad; else dart_tok_stats -> dart_step_select ->
        dart_tis_loss_fwd_bwd. Returns numpy outputs; dlogits only for
        ``keep_rows`` (all rows if None)."""
        torch, dart = self.torch, self.dart
        logp, ent, lse = dart.dart_tok_stats(self.logits, self.target)
        dl = self.logits if self.inplace else None
        if mask is None and fused:
            step_H, step_mask, n_kept, loss, coef, stats = dart.dart_select_tis_loss_fwd(
                ent, logp, self.lp_old, self.lp_roll, self.adv, self.off, self.wl.rho,
                self.eps_low, self.eps_high, self.C)
            dz = dart.dart_tis_grad(self.logits, self.target, logp, lse, coef, dlogits=dl)
        else:
            step_H, step_mask, n_kept = dart.dart_step_select(ent, self.off, self.wl.rho)
            use_mask = step_mask if mask is None else torch.from_numpy(
                np.ascontiguousarray(mask, dtype=np.uint8)).to(self.logits.device)
            loss, dz, coef, stats = dart.dart_tis_loss_fwd_bwd(
                self.logits, self.target, logp, lse, self.lp_old, self.lp_roll, self.adv,
                self.off, use_mask, self.eps_low, self.eps_high, self.C, dlogits=dl)
        torch.cuda.synchronize()
        rows = slice(None) if keep_rows is None else torch.from_numpy(
            np.asarray(keep_rows, dtype=np.int64)).to(self.logits.device)
        dz_sel = dz[rows]
        if dz_sel.dtype == torch.bfloat16:
            dz_np = dz_sel.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            dz_np = dz_sel.contiguous().cpu().numpy()
        out = dict(logp=logp.cpu().numpy(), H=ent.cpu().numpy(), lse=lse.cpu().numpy(),
                   Hs=step_H.cpu().numpy(), mask=step_mask.cpu().numpy(),
                   k=int(n_kept.cpu().item()), L=float(loss.cpu().item()),
                   g=coef.cpu().numpy(), stats=stats.cpu().numpy(), dz=dz_np)
        return out


# ---------------------------------------------------------------- checks

def rne_bf16_bits(x):
    """fp32 -> bf16 bits, round to nearest even on the bit pattern (a NaN
    stays a quiet NaN with its upper payload): the rounding the header states
    for every bf16 output."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r[nan] = ((u[nan] >> 16) | 0x40) & 0xFFFF
    return r.astype(np.uint16)


def rounding_coefs():
    """Coefficients g on and beside bf16 rounding ties, in the fp32 denormal
    range and at the top of the range, of both signs."""
    import math

    e = lambda k: math.ldexp(1.0, k)  # noqa: E731
    return np.array([1.0 + e(-8), 1.0 + 3 * e(-8), 1.0 + e(-8) + e(-23), 1.0 + e(-8) - e(-23),
                     -(1.0 + e(-8)), -(1.0 + 3 * e(-8)), 1.5, 0.3, -0.7, 1e-3, 65504.0, 1e10,
                     e(-126), e(-127), e(-133) + e(-149), 3 * e(-134), e(-134), e(-149),
                     -e(-130), 1e-30, 3.0e38, 3.4028235e38, -3.4028235e38, 0.0, -0.0],
                    dtype=np.float32)


def check_token_stats(gpu, ors, rows=None):
    sl = slice(None) if rows is None else rows
    dl = np.abs(gpu["logp"][sl] - ors.logp[sl])
    dh = np.abs(gpu["H"][sl] - ors.H[sl])
    ds = np.abs(gpu["lse"][sl] - ors.lse[sl])
    assert dl.max() <= LOGP_TOL, f"logp max err {dl.max():.3g} at {np.argmax(dl)}"
    assert dh.max() <= H_TOL, f"entropy max err {dh.max():.3g} at {np.argmax(dh)}"
    assert ds.max() <= 2e-4 + 1e-6 * np.abs(ors.lse[sl]).max(), f"lse max err {ds.max():.3g}"
    assert np.all(gpu["H"][sl] >= 0)
    return dict(logp=float(dl.max()), H=float(dh.max()))


def valid_topk(mask, vals, k):
    """mask keeps exactly k values, none smaller than a dropped one, and among
    values equal to the smallest kept one the kept indices precede the dropped."""
    mask = np.asarray(mask).astype(bool)
    if mask.sum() != k:
        return False
    if k == 0 or k == len(vals):
        return True
    kept_min = vals[mask].min()
    if kept_min < vals[~mask].max():
        return False
    eq = np.flatnonzero(vals == kept_min)
    kept_eq = mask[eq]
    return bool(np.all(kept_eq[:kept_eq.sum()]))


def check_mask(gpu, ors):
    wl = ors.wl
    k = ors.k
    assert gpu["k"] == k
    assert int(gpu["mask"].sum()) == k
    assert np.abs(gpu["Hs"] - ors.Hs).max() <= H_TOL
    assert valid_topk(gpu["mask"], gpu["Hs"], k), "GPU mask is not a top-k of its step entropies"
    if 0 < k < wl.S:
        thr = np.sort(ors.Hs)[::-1][k - 1]
        sep = np.abs(ors.Hs - thr) > BAND
        bad = np.flatnonzero(sep & (gpu["mask"] != ors.mask))
        assert bad.size == 0, f"mask differs on well-separated steps {bad[:10]}"
    return bool(np.array_equal(gpu["mask"], ors.mask))


def check_loss(gpu, res, boundary):
    L, Lg = res["L"], gpu["L"]
    scale = max(abs(L), 1e-30)
    assert abs(Lg - L) <= LOSS_RTOL * scale, f"loss {Lg!r} vs {L!r} (|L|={abs(L):.3g})"
    ok = ~boundary
    g, gg = res["g"][ok], gpu["g"][ok]
    err = np.abs(gg - g)
    floor = 1e-6 * np.abs(res["g"]).max() + 1e-30
    assert np.all(err <= 1e-4 * np.abs(g) + floor), f"tok_coef max rel err {np.max(err / np.maximum(np.abs(g), 1e-30)):.3g}"
    N = res["stats"][3]
    assert gpu["stats"][3] == N
    if N > 0:
        assert abs(gpu["stats"][0] - res["stats"][0]) <= (boundary.sum() + 0.5) / N
        assert abs(gpu["stats"][1] - res["stats"][1]) <= 1e-5 * max(1.0, res["stats"][1])
        assert abs(gpu["stats"][2] - res["stats"][2]) <= 1.5 / N
    return abs(Lg - L) / scale


def check_dz(gpu_dz, ref64, dtype, row_ok=None):
    """Element-wise: at most 1 bf16 ulp of the correctly rounded oracle value
    (and 1e-2 absolute); float32 logits: 1e-5 relative to the row's scale."""
    if row_ok is not None:
        gpu_dz, ref64 = gpu_dz[row_ok], ref64[row_ok]
    if gpu_dz.size == 0:
        return 0.0
    if dtype == "bf16":
        ref_bits = oracle.f64_to_bf16_bits(ref64)
        ref = synth.bf16_bits_to_f32(ref_bits).astype(np.float64)
        got = synth.bf16_bits_to_f32(gpu_dz).astype(np.float64)
        ulp = oracle.bf16_ulp(ref_bits)
        diff = np.abs(got - ref)
        bad = (diff > ulp) | (diff > 1e-2)
        if np.any(bad):
            i = np.argwhere(bad)[0]
            raise AssertionError(f"dlogits {bad.sum()} elements beyond 1 bf16 ulp; first at {tuple(i)}: "
                                 f"got {got[tuple(i)]!r} ref {ref64[tuple(i)]!r}")
        return float((diff / ulp).max())
    scale = np.abs(ref64).max(axis=1, keepdims=True) + 1e-30
    err = np.abs(gpu_dz.astype(np.float64) - ref64)
    rel = err / scale
    if not np.all(rel <= 1e-5):
        i, j = np.unravel_index(np.argmax(rel), rel.shape)
        raise AssertionError(f"dlogits f32 max scaled err {rel.max():.3g} at row {i} col {j}: "
                             f"got {gpu_dz[i, j]!r} ref {ref64[i, j]!r} row scale {scale[i, 0]!r}")
    return float(rel.max())


def sample_rows(wl, res, n_random=48, seed=0):
    """Rows for element-wise gradient checks: the first and last rows, the
    first and last token of a spread of steps, rows of every row kind, rows
    whose target sits in the first or last 16 columns, the largest |g|, and
    random rows."""
    rng = np.random.default_rng(seed)
    T = wl.T
    rows = {0, T - 1}
    steps = np.unique(np.linspace(0, wl.S - 1, min(wl.S, 12)).astype(int))
    for s in steps:
        rows.add(int(wl.off[s]))
        rows.add(int(wl.off[s + 1] - 1))
    for kind in np.unique(wl.kind):
        idx = np.flatnonzero(wl.kind == kind)
        rows.update(int(i) for i in rng.choice(idx, min(4, idx.size), replace=False))
    edge = np.flatnonzero((wl.target < 16) | (wl.target >= wl.V - 16))
    rows.update(int(i) for i in edge[:4])
    g = np.abs(res["g"])
    rows.update(int(i) for i in np.argsort(g)[-4:])
    rows.update(int(i) for i in rng.integers(0, T, n_random))
    return np.array(sorted(rows), dtype=np.int64)
