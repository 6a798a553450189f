"""GPU parity of the gradient pass through the LM head with the float64 oracle,
through the C ABI: dlogits of the recomputed logits z = h W^T (bfloat16,
within 1 bf16 ulp of the correctly rounded oracle value, as on the logits
path), and dhidden = dlogits W, dweight = dlogits^T h.

The GPU side runs its own chain (fused statistics, then the gradient entry
points); the oracle side computes its float64 statistics and gradients from
the same bf16 inputs. The per-token coefficient g = dL/dlogp is an input of
both (seeded float32, with zeros as dropped tokens have).

dhidden and dweight, each element two ways, with B = |dz| |W| (resp.
|dz|^T |h|) the sum of the absolute terms:
- against the oracle's exact product: the GPU's bf16 dlogits are within one
  bf16 ulp of the correctly rounded value (checked element by element above),
  so within 1.5 ulp <= 3 U of the exact value (U = 2^-8, the unit roundoff of
  bf16's 8-bit significand, and an ulp is at most 2 U relative), and the
  library sums in fp32: tolerance 3 U B + A B, with A = 2^-13 for the fp32
  sums;
- a consistency property of the GEMM stage, not a parity reference: against
  the exact product of the GPU's own bf16 dlogits (the same kernel's output,
  bit for bit the values the backward multiplies) only the fp32 sums differ,
  tolerance A B; a block left out or added twice, or a wrong offset, moves an
  element by far more than A B. Parity rests on the oracle comparison above.
A bf16 gradient adds its own rounding, U |value| (round to nearest even)."""

import math
import zlib

import numpy as np
import pytest

import oracle
import synth
import synth.native as sn
from synth import gaussian_bits
from synth.gen import STREAM_HIDDEN, STREAM_WEIGHT
from tests import _harness as H

pytestmark = pytest.mark.gpu

U = 2.0 ** -8   # unit roundoff of bf16
A = 2.0 ** -13  # fp32 summation in the GEMMs, relative to the sum of |terms|


def _dev_bf16(bits, pad=0):
    import torch

    bits = np.ascontiguousarray(bits)
    rows, cols = bits.shape
    t = torch.zeros((rows, cols + pad), dtype=torch.int16, device="cuda")
    t[:, :cols] = torch.from_numpy(bits.view(np.int16)).cuda()
    return t.view(torch.bfloat16)[:, :cols]


def _cuda(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _coef(rng, T):
    g = rng.uniform(-1.0, 1.0, T) * 1e-2
    g[rng.random(T) < 0.25] = 0.0
    return g.astype(np.float32)


def _problem(T, d, V):
    seed = zlib.crc32(repr(("grad", T, d, V)).encode()) % 1000
    rng = np.random.default_rng(seed)
    h = gaussian_bits(seed, STREAM_HIDDEN, T, d, 1.0)
    w = gaussian_bits(seed, STREAM_WEIGHT, V, d, 3.0 / math.sqrt(d))
    y = rng.integers(0, V, T).astype(np.int32)
    return h, w, y, _coef(rng, T)


def _bits(t):
    import torch

    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _as_f64(x):
    import torch

    if isinstance(x, torch.Tensor):
        x = x.float().cpu().numpy()
    return np.asarray(x, dtype=np.float64)


def _check_grad(got, ref, own, bound, name, bf16=False):
    """got against the oracle's exact product ref (3 U B + A B) and, unless own
    is None, against the exact product own of the GPU's own bf16 dlogits (A B);
    a bf16 output adds U |value| to both. Returns the largest error against ref
    in units of B."""
    got = _as_f64(got)
    checks = [("oracle", ref, (3 * U + A) * bound)]
    if own is not None:
        checks.append(("own dlogits", own, A * bound))
    for what, target, tol in checks:
        if bf16:
            tol = tol + U * np.abs(target)
        err = np.abs(got - target)
        bad = err > tol + 1e-30
        if np.any(bad):
            i = tuple(np.argwhere(bad)[0])
            raise AssertionError(f"{name} vs {what}: {bad.sum()} elements out of tolerance; first "
                                 f"at {i}: got {got[i]!r} ref {target[i]!r} B {bound[i]!r}")
    return float((np.abs(got - ref) / np.maximum(bound, 1e-300)).max())


def _own_dz(hd, wd, yd, lse, logp, gd):
    """The GPU's own bf16 dlogits (the kernel every backward runs), as float64."""
    import torch

    import paper_2509_23866_amd as dart

    T, V = hd.shape[0], wd.shape[0]
    buf = torch.empty((T, (V + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")
    dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd, dlogits=buf[:, :V])
    return buf[:, :V].double().cpu().numpy()


SHAPES = [
    # (T, d, V, pad of the hidden / weight rows)
    (1, 8, 1, 0),
    (3, 8, 5, 0),
    (127, 136, 129, 0),
    (129, 72, 127, 8),
    (200, 200, 1000, 0),
    (64, 256, 4099, 16),
    (300, 512, 16384, 0),
]


@pytest.mark.parametrize("T,d,V,pad", SHAPES)
def test_lmhead_dlogits_shapes(T, d, V, pad):
    import torch

    import paper_2509_23866_amd as dart

    h, w, y, g = _problem(T, d, V)
    rlogp, _, rlse = oracle.lmhead_token_stats(h, w, y)
    dz64, _, _ = oracle.lmhead_grads(h, w, y, rlse, rlogp, g)
    hd, wd, yd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    ld = (V + 7) // 8 * 8 + 8
    out = torch.full((T, ld), -7.0, dtype=torch.bfloat16, device="cuda")
    dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, _cuda(g), dlogits=out[:, :V])
    torch.cuda.synchronize()
    ulps = H.check_dz(_bits(out[:, :V]), dz64, "bf16")
    assert torch.all(out[:, V:] == -7.0), "columns past V were written"
    # rows with g = 0 are exact zeros
    zero = g == 0.0
    assert np.all(_bits(out[:, :V])[zero] & 0x7FFF == 0)
    H.log(f"lmhead dlogits T={T} d={d} V={V}: max {ulps:.2f} ulp")


@pytest.mark.parametrize("T,d,V,pad,chunk", [
    (1, 8, 1, 0, 1),
    (3, 8, 5, 0, 2),
    (129, 72, 127, 8, 1024),
    (200, 200, 1000, 0, 64),
    (300, 512, 16384, 0, 257),
    (257, 3584, 2000, 0, 100),
])
def test_lmhead_backward_shapes(T, d, V, pad, chunk):
    import torch

    import paper_2509_23866_amd as dart

    h, w, y, g = _problem(T, d, V)
    rlogp, _, rlse = oracle.lmhead_token_stats(h, w, y)
    dz64, dh64, dw64 = oracle.lmhead_grads(h, w, y, rlse, rlogp, g)
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    hd, wd, yd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    dh = torch.full((T, d + 4), 3.0, dtype=torch.float32, device="cuda")
    dw = torch.full((V, d), 12345.0, dtype=torch.float32, device="cuda")  # overwritten
    dart.dart_lmhead_backward(hd, wd, yd, lse, logp, _cuda(g), chunk_rows=chunk,
                              dhidden=dh[:, :d], dweight=dw)
    dzo = _own_dz(hd, wd, yd, lse, logp, _cuda(g))
    torch.cuda.synchronize()
    adz = np.abs(dz64)
    rh = _check_grad(dh[:, :d], dh64, dzo @ w64, adz @ np.abs(w64), "dhidden")
    rw = _check_grad(dw, dw64, dzo.T @ h64, adz.T @ np.abs(h64), "dweight")
    assert torch.all(dh[:, d:] == 3.0), "dhidden padding was written"
    H.log(f"lmhead backward T={T} d={d} V={V} chunk={chunk}: dh {rh:.2e} dW {rw:.2e} of |dz||.|")


def test_lmhead_backward_chunking_consistent():
    """The chunk size changes only the order dweight's terms are summed in;
    dhidden rows are computed identically."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 300, 256, 3000
    h, w, y, g = _problem(T, d, V)
    hd, wd, yd, gd = _dev_bf16(h), _dev_bf16(w), _cuda(y), _cuda(g)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    dha, dwa = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=300)
    dhb, dwb = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=77)
    dz = _own_dz(hd, wd, yd, lse, logp, gd)
    torch.cuda.synchronize()
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    # against the exact products of the GPU's own bf16 dlogits: only the fp32
    # summation differs between chunkings
    for x, ref, bound in ((dwa, dz.T @ h64, np.abs(dz).T @ np.abs(h64)),
                          (dwb, dz.T @ h64, np.abs(dz).T @ np.abs(h64)),
                          (dha, dz @ w64, np.abs(dz) @ np.abs(w64)),
                          (dhb, dz @ w64, np.abs(dz) @ np.abs(w64))):
        assert np.all(np.abs(x.cpu().numpy() - ref) <= A * bound + 1e-30)


def test_lmhead_backward_vlm7b_shape():
    """T = 4096, d = 3584, V = 152064 with chunks of 1024 rows (four dweight
    accumulations). g is non-zero on a sampled row set R (first and last rows,
    chunk and tile edges, random rows), so that dweight is the oracle's product
    over R alone and is compared whole; dhidden rows outside R are exact
    zeros."""
    import torch

    import paper_2509_23866_amd as dart

    prob = synth.lmhead_problem("vlm7b")
    wl, d = prob.wl, prob.d
    T, V = wl.T, wl.V
    rng = np.random.default_rng(17)
    R = np.unique(np.r_[0, 1, 255, 256, 1023, 1024, 2047, 2048, T - 1, rng.integers(0, T, 23)])
    g = np.zeros(T, np.float32)
    g[R] = (rng.uniform(-1.0, 1.0, R.size) * 1e-3).astype(np.float32)
    hd = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    wd = torch.empty((V, d), dtype=torch.bfloat16, device="cuda")
    sn.fill_gaussian_device(hd, wl.seed, STREAM_HIDDEN, prob.sigma_h)
    sn.fill_gaussian_device(wd, wl.seed, STREAM_WEIGHT, prob.sigma_w)
    yd = _cuda(wl.target.astype(np.int32))
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    gd = _cuda(g)
    dh, dw = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=1024)
    # the row-skipping backward: the GEMMs over the rows of R only
    dhs, dws = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=1024,
                                            chunk_cols=V, flags=dart.DART_LMHEAD_SKIP_ZERO_ROWS)
    # the default plan's blocks with bf16 gradients, as the autograd function runs them
    pr, pc = dart.lmhead_backward_plan(T, V)
    assert pc < V
    dhb, dwb = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=pr, chunk_cols=pc,
                                            flags=dart.DART_LMHEAD_BF16_GRADS)
    torch.cuda.synchronize()
    dh, dhs = dh.cpu().numpy(), dhs.cpu().numpy()
    outside = np.ones(T, bool)
    outside[R] = False
    assert np.all(dh[outside] == 0.0) and np.all(dhs[outside] == 0.0)
    assert torch.all(dhb[torch.from_numpy(outside).cuda()] == 0.0)

    hb = prob.hidden_bits(R)
    wb = sn.gaussian_bits_host(wl.seed, STREAM_WEIGHT, V, d, prob.sigma_w)
    y = wl.target[R].astype(np.int32)
    rlogp, _, rlse = oracle.lmhead_token_stats(hb, wb, y)
    z = oracle.lmhead_logits(hb, wb)
    dz64 = oracle.dlogits(z, y, rlse, rlogp, g[R])
    del z
    w64, h64 = oracle.bf16_bits_to_f64(wb), oracle.bf16_bits_to_f64(hb)
    # the GPU's own dlogits of the rows of R
    Rd = torch.from_numpy(R).cuda()
    dzo = _own_dz(hd[Rd].contiguous(), wd, yd[Rd].contiguous(), lse[Rd].contiguous(),
                  logp[Rd].contiguous(), gd[Rd].contiguous())
    adz = np.abs(dz64)
    ref_h, own_h, bound_h = dz64 @ w64, dzo @ w64, adz @ np.abs(w64)
    rh = _check_grad(dh[R], ref_h, own_h, bound_h, "dhidden")
    rhs = _check_grad(dhs[R], ref_h, own_h, bound_h, "dhidden (rows skipped)")
    rhb = _check_grad(dhb[Rd], ref_h, own_h, bound_h, "dhidden (plan, bf16)", bf16=True)
    del w64
    rw = rws = rwb = 0.0
    for v0 in range(0, V, 16384):
        sl = slice(v0, min(V, v0 + 16384))
        ref, own = dz64[:, sl].T @ h64, dzo[:, sl].T @ h64
        bound = adz[:, sl].T @ np.abs(h64)
        rw = max(rw, _check_grad(dw[sl], ref, own, bound, f"dweight rows {v0}+"))
        rws = max(rws, _check_grad(dws[sl], ref, own, bound, f"dweight rows {v0}+ (rows skipped)"))
        rwb = max(rwb, _check_grad(dwb[sl], ref, own, bound, f"dweight rows {v0}+ (plan, bf16)",
                                   bf16=True))
    H.log(f"lmhead backward vlm7b: dh {rh:.2e} dW {rw:.2e} of |dz||.|; "
          f"rows skipped: dh {rhs:.2e} dW {rws:.2e}; plan {pr}x{pc} bf16: dh {rhb:.2e} "
          f"dW {rwb:.2e}")


def test_lmhead_caller_workspaces_contents_do_not_matter():
    """Caller-provided workspaces filled with garbage give the same bits as
    freshly allocated ones (statistics and backward)."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 300, 136, 2100
    h, w, y, g = _problem(T, d, V)
    hd, wd, yd, gd = _dev_bf16(h), _dev_bf16(w), _cuda(y), _cuda(g)
    a = dart.dart_lmhead_tok_stats(hd, wd, yd)
    ws = torch.full((dart.dart_lmhead_stats_workspace_bytes(T, V),), 0xC3, dtype=torch.uint8,
                    device="cuda")
    b = dart.dart_lmhead_tok_stats(hd, wd, yd, workspace=ws)
    for u, v in zip(a, b):
        assert torch.equal(u.view(torch.int32), v.view(torch.int32))
    logp, _, lse = a
    dha, dwa = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=128)
    wsb = torch.full((dart.dart_lmhead_backward_workspace_bytes(128, V),), 0x7F, dtype=torch.uint8,
                     device="cuda")
    dhb, dwb = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=128, workspace=wsb)
    torch.cuda.synchronize()
    assert torch.equal(dha, dhb) and torch.equal(dwa, dwb)


def _ones_zeros(kind, rng, T):
    g = (rng.uniform(-1.0, 1.0, T) * 1e-2).astype(np.float32)
    if kind == "all_zero":
        g[:] = 0.0
    elif kind == "one_row":
        g[np.arange(T) != T // 2] = 0.0
    elif kind == "steps":
        # whole runs of rows dropped, as the step mask drops whole steps
        for a in range(0, T, 37):
            if (a // 37) % 3 == 1:
                g[a:a + 37] = 0.0
    return g


@pytest.mark.parametrize("T,d,V,pad,chunk,kind", [
    (1, 8, 1, 0, 1, "dense"),
    (1, 8, 5, 0, 1, "all_zero"),
    (3, 8, 5, 0, 2, "one_row"),
    (129, 72, 127, 8, 1024, "steps"),
    (200, 200, 1000, 0, 64, "quarter"),
    (300, 512, 16384, 0, 257, "steps"),
    (1100, 136, 2000, 8, 100, "quarter"),
    (257, 3584, 2000, 0, 100, "all_zero"),
])
def test_lmhead_backward_skip_zero_rows(T, d, V, pad, chunk, kind):
    """dart_lmhead_backward_ex with DART_LMHEAD_SKIP_ZERO_ROWS against the
    oracle at the bound of the dense backward, rows with g = 0 exactly 0, the
    padding of dhidden untouched, and dweight 0 when every row is dropped. The
    row compaction walks 1024 rows at a time, so T = 1100 spans two passes."""
    import torch

    import paper_2509_23866_amd as dart

    h, w, y, _ = _problem(T, d, V)
    rng = np.random.default_rng(T * 7 + d)
    g = _ones_zeros(kind, rng, T) if kind != "quarter" else _coef(rng, T)
    rlogp, _, rlse = oracle.lmhead_token_stats(h, w, y)
    dz64, dh64, dw64 = oracle.lmhead_grads(h, w, y, rlse, rlogp, g)
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    hd, wd, yd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    dh = torch.full((T, d + 4), 3.0, dtype=torch.float32, device="cuda")
    dw = torch.full((V, d), 12345.0, dtype=torch.float32, device="cuda")  # overwritten
    flags = dart.DART_LMHEAD_SKIP_ZERO_ROWS
    ws = torch.full((dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, chunk, V, flags),),
                    0xA5, dtype=torch.uint8, device="cuda")
    dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, _cuda(g), chunk_rows=chunk, chunk_cols=V,
                                 flags=flags, dhidden=dh[:, :d], dweight=dw, workspace=ws)
    torch.cuda.synchronize()
    got_h = dh[:, :d].cpu().numpy()
    assert torch.all(dh[:, d:] == 3.0), "dhidden padding was written"
    assert np.all(got_h[g == 0.0] == 0.0), "a dropped row of dhidden is not 0"
    if not np.any(g):
        assert torch.all(dw == 0.0)
    dzo = _own_dz(hd, wd, yd, lse, logp, _cuda(g))
    adz = np.abs(dz64)
    rh = _check_grad(got_h, dh64, dzo @ w64, adz @ np.abs(w64), "dhidden")
    rw = _check_grad(dw, dw64, dzo.T @ h64, adz.T @ np.abs(h64), "dweight")
    H.log(f"lmhead backward rows skipped T={T} d={d} V={V} chunk={chunk} {kind} "
          f"({int(np.count_nonzero(g))} rows kept): dh {rh:.2e} dW {rw:.2e} of |dz||.|")


def test_lmhead_backward_skip_zero_rows_reused_workspace():
    """Two calls in a row on one workspace, the second keeping fewer rows: the
    row map and count left by the first call do not leak into the second, and
    flags = 0 of the _ex entry point gives dart_lmhead_backward's bits."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 600, 136, 2100
    h, w, y, g = _problem(T, d, V)
    hd, wd, yd = _dev_bf16(h), _dev_bf16(w), _cuda(y)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    flags = dart.DART_LMHEAD_SKIP_ZERO_ROWS
    ws = torch.empty((dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, 128, V, flags),),
                     dtype=torch.uint8, device="cuda")
    g2 = g.copy()
    g2[T // 3:] = 0.0
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    for gx in (g, g2):
        gd = _cuda(gx)
        dha, dwa = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=128)
        dhs, dws = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=128,
                                                chunk_cols=V, flags=flags, workspace=ws)
        dh0, dw0 = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=128,
                                                chunk_cols=V)
        zbuf = torch.empty((T, (V + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")
        dz = dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd, dlogits=zbuf[:, :V])
        dz = dz.double().cpu().numpy()
        torch.cuda.synchronize()
        assert torch.equal(dha, dh0) and torch.equal(dwa, dw0)
        assert np.all(dhs.cpu().numpy()[gx == 0.0] == 0.0)
        # both are products of the same bf16 dlogits, summed by the library in
        # fp32 in different orders: each is within fp32 summation error of the
        # exact product of those dlogits
        adz = np.abs(dz)
        for got, ref, bound in ((dhs, dz @ w64, adz @ np.abs(w64)),
                                (dha, dz @ w64, adz @ np.abs(w64)),
                                (dws, dz.T @ h64, adz.T @ np.abs(h64)),
                                (dwa, dz.T @ h64, adz.T @ np.abs(h64))):
            assert np.all(np.abs(got.cpu().numpy() - ref) <= A * bound + 1e-30)


_SKIP, _BF = 1, 4


@pytest.mark.parametrize("T,d,V,pad,rows,cols,flags", [
    (1, 8, 5, 0, 1, 2, 0),
    (129, 72, 127, 8, 129, 64, 0),
    (129, 72, 127, 8, 129, 64, _BF),
    (300, 512, 16384, 0, 300, 4096, _BF),
    (300, 512, 16384, 0, 300, 1000, 0),
    (257, 3584, 2000, 0, 257, 777, _BF),
    (257, 3584, 2000, 0, 100, 2000, _BF),
    (257, 3584, 2000, 0, 1024, 2000, _BF),
    (1100, 136, 2000, 8, 300, 700, 0),
    (1100, 136, 2000, 8, 300, 700, _BF),
    (1100, 136, 2000, 8, 1100, 256, _SKIP),
    (1100, 136, 2000, 8, 1100, 256, _SKIP | _BF),
    (1100, 136, 2000, 8, 300, 2000, _SKIP | _BF),
    (1100, 136, 2000, 8, 256, 512, _SKIP | _BF),
    (200, 200, 1000, 0, 5000, 5000, _SKIP | _BF),
])
def test_lmhead_backward_ex_modes(T, d, V, pad, rows, cols, flags):
    """dart_lmhead_backward_ex in blocks of rows x vocabulary entries (all rows
    with vocabulary chunks, row chunks over the whole vocabulary, both split;
    ragged: blocks that are not whole tiles, last blocks shorter than the
    others, one block covering everything), with bf16 gradients (summed over
    several blocks in fp32 first, or written straight from one block) and with
    zero rows skipped, each against the oracle; padding of dhidden untouched;
    skipped rows exactly 0."""
    import torch

    import paper_2509_23866_amd as dart

    h, w, y, g = _problem(T, d, V)
    rlogp, _, rlse = oracle.lmhead_token_stats(h, w, y)
    dz64, dh64, dw64 = oracle.lmhead_grads(h, w, y, rlse, rlogp, g)
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    hd, wd, yd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    gdt = torch.bfloat16 if flags & _BF else torch.float32
    dh = torch.full((T, d + 4), 3.0, dtype=gdt, device="cuda")
    dwp = torch.full((V, d + 8), 7.0, dtype=gdt, device="cuda")  # rows padded by 8
    dw = dwp[:, :d]
    dw.fill_(12345.0)  # overwritten
    nb = dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, flags)
    ws = torch.full((nb,), 0x5A, dtype=torch.uint8, device="cuda")
    dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, _cuda(g), chunk_rows=rows, chunk_cols=cols,
                                 flags=flags, dhidden=dh[:, :d], dweight=dw, workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(dh[:, d:] == 3.0), "dhidden padding was written"
    assert torch.all(dwp[:, d:] == 7.0), "dweight padding was written"
    if flags & _SKIP:
        assert torch.all(dh[:, :d][torch.from_numpy(g == 0.0).cuda()] == 0.0)
    dzo = _own_dz(hd, wd, yd, lse, logp, _cuda(g))
    adz = np.abs(dz64)
    bf = bool(flags & _BF)
    rh = _check_grad(dh[:, :d], dh64, dzo @ w64, adz @ np.abs(w64), "dhidden", bf16=bf)
    rw = _check_grad(dw, dw64, dzo.T @ h64, adz.T @ np.abs(h64), "dweight", bf16=bf)
    H.log(f"lmhead backward_ex T={T} d={d} V={V} block={rows}x{cols} flags={flags}: "
          f"dh {rh:.2e} dW {rw:.2e}")


@pytest.mark.parametrize("T,d,V,pad,rows,cols,flags,inv_temp", [
    (129, 72, 127, 8, 129, 64, _BF, 0.7),
    (300, 512, 16384, 0, 300, 4096, 0, 1.6),
    (257, 3584, 2000, 0, 100, 2000, _BF, 1.3),
    (1100, 136, 2000, 8, 300, 700, _SKIP | _BF, 0.5),
])
def test_lmhead_inverse_temperature(T, d, V, pad, rows, cols, flags, inv_temp):
    """Statistics and gradients of softmax(inv_temp h W^T) (the _ex entry
    points) against the oracle at the same inverse temperature: logp, H and lse
    to the tolerances of the logits path, dz within 1 bf16 ulp, dhidden and
    dweight to 3 U B + A B with the factor inv_temp inside dz (and to A B
    against the GPU's own dz, the consistency property of the GEMM stage)."""
    import torch

    import paper_2509_23866_amd as dart

    h, w, y, g = _problem(T, d, V)
    ref = oracle.lmhead_token_stats(h, w, y, inv_temp=inv_temp)
    _, dh64, dw64 = oracle.lmhead_grads(h, w, y, ref[2], ref[0], g, inv_temp=inv_temp)
    dz64 = oracle.dlogits(oracle.lmhead_logits(h, w), y, ref[2], ref[0], g, inv_temp=inv_temp)
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    hd, wd, yd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y)
    logp, ent, lse = dart.dart_lmhead_tok_stats_ex(hd, wd, yd, inv_temp)
    got = [x.cpu().numpy().astype(np.float64) for x in (logp, ent, lse)]
    err = [float(np.abs(a - b).max()) for a, b in zip(got, ref)]
    assert err[0] <= H.LOGP_TOL and err[1] <= H.H_TOL and err[2] <= H.LOGP_TOL, err
    buf = torch.empty((T, (V + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")
    dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, _cuda(g), dlogits=buf[:, :V],
                             inv_temp=inv_temp)
    torch.cuda.synchronize()
    ulps = H.check_dz(_bits(buf[:, :V]), dz64, "bf16")
    dzo = buf[:, :V].double().cpu().numpy()
    dh, dw = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, _cuda(g), chunk_rows=rows,
                                          chunk_cols=cols, flags=flags, inv_temp=inv_temp)
    torch.cuda.synchronize()
    adz = np.abs(dz64)
    bf = bool(flags & _BF)
    rh = _check_grad(dh, dh64, dzo @ w64, adz @ np.abs(w64), "dhidden", bf16=bf)
    rw = _check_grad(dw, dw64, dzo.T @ h64, adz.T @ np.abs(h64), "dweight", bf16=bf)
    H.log(f"lmhead inv_temp={inv_temp} T={T} d={d} V={V} block={rows}x{cols} flags={flags}: "
          f"stats {max(err):.2e} dz {ulps:.2f} ulp dh {rh:.2e} dW {rw:.2e}")


def test_lmhead_inverse_temperature_one_is_the_plain_call():
    """At inv_temp = 1 the _ex statistics and the backward give the bits of the
    calls without a temperature."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 300, 136, 2000
    h, w, y, g = _problem(T, d, V)
    hd, wd, yd, gd = _dev_bf16(h), _dev_bf16(w), _cuda(y), _cuda(g)
    plain = dart.dart_lmhead_tok_stats(hd, wd, yd)
    ex = dart.dart_lmhead_tok_stats_ex(hd, wd, yd, 1.0)
    for a, b in zip(plain, ex):
        assert torch.equal(a, b)
    logp, _, lse = plain
    z1 = dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd)
    z2 = dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd, inv_temp=1.0)
    assert torch.equal(z1.view(torch.int16), z2.view(torch.int16))
    ref = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, gd, chunk_rows=128)
    got = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=128, chunk_cols=V,
                                       inv_temp=1.0)
    for a, b in zip(ref, got):
        assert torch.equal(a, b)


def test_lmhead_backward_blockings_agree():
    """The same bf16 dlogits summed in other orders: row chunks, vocabulary
    chunks and 2-D blocks, fp32 outputs, each within fp32 summation error of
    the exact products of those dlogits; bf16 outputs equal the fp32 ones of
    the same blocking rounded, within one bf16 ulp."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 300, 256, 3000
    h, w, y, g = _problem(T, d, V)
    hd, wd, yd, gd = _dev_bf16(h), _dev_bf16(w), _cuda(y), _cuda(g)
    logp, _, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    zbuf = torch.empty((T, (V + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")
    dz = dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd, dlogits=zbuf[:, :V])
    dz = dz.double().cpu().numpy()
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    adz = np.abs(dz)
    refs = ((dz @ w64, adz @ np.abs(w64)), (dz.T @ h64, adz.T @ np.abs(h64)))
    blocks = [(77, V), (T, 700), (T, 256), (128, 1000)]
    outs = [dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=r, chunk_cols=c)
            for r, c in blocks]
    bfs = [dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=r, chunk_cols=c,
                                        flags=_BF) for r, c in blocks]
    torch.cuda.synchronize()
    for got in outs:
        for x, (ref, bound) in zip(got, refs):
            assert np.all(np.abs(x.cpu().numpy() - ref) <= A * bound + 1e-30)
    for bf, fp in zip(bfs, outs):
        for xb, xf, (_, bound) in zip(bf, fp, refs):
            # one rounding of the fp32 sum, up to the fp32 summation order of
            # the GEMM kernels for bf16 and fp32 outputs
            a = xb.float().cpu().numpy().astype(np.float64)
            b = xf.cpu().numpy().astype(np.float64)
            assert np.all(np.abs(a - b) <= U * np.abs(b) + A * bound + 1e-37)


@pytest.mark.parametrize("seed", range(16))
def test_lmhead_random_configurations(seed):
    """16 seeded random LM-head problems: T in 1..300, d a multiple of 8 up
    to 512, V in 1..5000, padded rows, random blocks of rows x vocabulary
    entries and random flags; statistics, rows skipped exactly 0, and both
    gradients against the oracle and the GPU's own dlogits."""
    import torch

    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(7000 + seed)
    T, d, V = int(rng.integers(1, 301)), 8 * int(rng.integers(1, 65)), int(rng.integers(1, 5001))
    pad = 8 * int(rng.integers(0, 3))
    rows, cols = int(rng.integers(1, T + 65)), int(rng.integers(1, V + 300))
    flags = int(rng.choice([0, _SKIP, _BF, _SKIP | _BF]))
    h, w, y, g = _problem(T, d, V)
    rlogp, rH, rlse = oracle.lmhead_token_stats(h, w, y)
    dz64, dh64, dw64 = oracle.lmhead_grads(h, w, y, rlse, rlogp, g)
    h64, w64 = oracle.bf16_bits_to_f64(h), oracle.bf16_bits_to_f64(w)
    hd, wd, yd, gd = _dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y), _cuda(g)
    logp, ent, lse = dart.dart_lmhead_tok_stats(hd, wd, yd)
    dh, dw = dart.dart_lmhead_backward_ex(hd, wd, yd, lse, logp, gd, chunk_rows=rows,
                                          chunk_cols=cols, flags=flags)
    dzo = _own_dz(hd, wd, yd, lse, logp, gd)
    torch.cuda.synchronize()
    assert np.abs(logp.cpu().numpy() - rlogp).max() <= 2e-4
    assert np.abs(ent.cpu().numpy() - rH).max() <= 2e-4
    if flags & _SKIP:
        assert np.all(_as_f64(dh)[g == 0.0] == 0.0)
    adz = np.abs(dz64)
    bf = bool(flags & _BF)
    rh = _check_grad(dh, dh64, dzo @ w64, adz @ np.abs(w64), "dhidden", bf16=bf)
    rw = _check_grad(dw, dw64, dzo.T @ h64, adz.T @ np.abs(h64), "dweight", bf16=bf)
    H.log(f"lmhead random {seed}: T={T} d={d} V={V} pad={pad} block={rows}x{cols} "
          f"flags={flags}: dh {rh:.2e} dW {rw:.2e}")
