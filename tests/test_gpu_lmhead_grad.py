"""GPU parity of the gradient pass through the LM head with the float64 oracle,
through the C ABI: dlogits of the recomputed logits z = h W^T (bfloat16,
within 1 bf16 ulp of the correctly rounded oracle value, as on the logits
path), and dhidden = dlogits W, dweight = dlogits^T h.

The GPU side runs its own chain (fused statistics, then the gradient entry
points); the oracle side computes its float64 statistics and gradients from
the same bf16 inputs. The per-token coefficient g = dL/dlogp is an input of
both (seeded float32, with zeros as dropped tokens have).

dhidden and dweight: the GPU rounds dlogits to bf16 (relative error at most
2^-9) and accumulates in fp32, so each element is compared against
2^-8 * (|dz| |W|) (resp. |dz|^T |h|), twice the rounding bound."""

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

BF16_REL = 2.0 ** -8


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


def _check_product(got, ref, bound, name):
    err = np.abs(got.astype(np.float64) - ref)
    tol = BF16_REL * bound + 1e-30
    bad = err > tol
    if np.any(bad):
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{name}: {bad.sum()} elements beyond 2^-8 |dz||.|; first at {i}: "
                             f"got {got[i]!r} ref {ref[i]!r} bound {bound[i]!r}")
    return float((err / np.maximum(bound, 1e-300)).max())


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
    torch.cuda.synchronize()
    adz = np.abs(dz64)
    rh = _check_product(dh[:, :d].cpu().numpy(), dh64, adz @ np.abs(w64), "dhidden")
    rw = _check_product(dw.cpu().numpy(), dw64, adz.T @ np.abs(h64), "dweight")
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
    dz = dart.dart_lmhead_dlogits(hd, wd, yd, lse, logp, gd).float()
    torch.cuda.synchronize()
    ref = (dz.T.cpu().double() @ torch.from_numpy(oracle.bf16_bits_to_f64(h))).numpy()
    bound = np.abs(dz.T.cpu().double().numpy()) @ np.abs(oracle.bf16_bits_to_f64(h))
    for dwx in (dwa, dwb):
        # against the bf16 dlogits themselves: only fp32 summation error remains
        err = np.abs(dwx.cpu().numpy() - ref)
        assert np.all(err <= 1e-4 * bound + 1e-30)
    assert torch.allclose(dha, dhb, rtol=1e-5, atol=1e-7)


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
    dh, dw = dart.dart_lmhead_backward(hd, wd, yd, lse, logp, _cuda(g), chunk_rows=1024)
    torch.cuda.synchronize()
    dh = dh.cpu().numpy()
    outside = np.ones(T, bool)
    outside[R] = False
    assert np.all(dh[outside] == 0.0)

    hb = prob.hidden_bits(R)
    wb = sn.gaussian_bits_host(wl.seed, STREAM_WEIGHT, V, d, prob.sigma_w)
    y = wl.target[R].astype(np.int32)
    rlogp, _, rlse = oracle.lmhead_token_stats(hb, wb, y)
    z = oracle.lmhead_logits(hb, wb)
    dz64 = oracle.dlogits(z, y, rlse, rlogp, g[R])
    del z
    w64, h64 = oracle.bf16_bits_to_f64(wb), oracle.bf16_bits_to_f64(hb)
    adz = np.abs(dz64)
    rh = _check_product(dh[R], dz64 @ w64, adz @ np.abs(w64), "dhidden")
    del w64
    rw = 0.0
    for v0 in range(0, V, 16384):
        sl = slice(v0, min(V, v0 + 16384))
        got = dw[sl].cpu().numpy()
        rw = max(rw, _check_product(got, dz64[:, sl].T @ h64, adz[:, sl].T @ np.abs(h64),
                                    f"dweight rows {v0}+"))
    H.log(f"lmhead backward vlm7b: dh {rh:.2e} dW {rw:.2e} of |dz||.|")


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
