"""GPU parity of the LM-head statistics (logits h W^T formed on the matrix
cores and never written) with the float64 oracle, through the C ABI.

Shapes cover ragged token, vocabulary and hidden-size tiles (128 x 128 x 64),
the smallest hidden size (8), one-entry vocabularies, padded rows, a real
hidden size (3584), and the 7B-VLM shape (T = 4096, d = 3584, V = 152064) on
sampled rows. Tolerances are those of the logits path (2e-4 absolute on logp,
H and lse): z is accumulated in fp32 from bf16 inputs, an error of order
1e-5 against the float64 product."""

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


def _check(got, ref, rows=None):
    logp, ent, lse = (x.cpu().numpy().astype(np.float64) for x in got)
    rlogp, rH, rlse = ref
    if rows is not None:
        logp, ent, lse = logp[rows], ent[rows], lse[rows]
    e = dict(logp=np.abs(logp - rlogp).max(), H=np.abs(ent - rH).max(), lse=np.abs(lse - rlse).max())
    H.log(f"lmhead stats max err: logp {e['logp']:.2e} H {e['H']:.2e} lse {e['lse']:.2e}")
    assert e["logp"] <= H.LOGP_TOL and e["H"] <= H.H_TOL and e["lse"] <= H.LOGP_TOL


SHAPES = [
    # (T, d, V, pad of the hidden / weight rows)
    (1, 8, 1, 0),
    (3, 8, 5, 0),
    (128, 64, 128, 0),
    (127, 136, 129, 0),
    (129, 72, 127, 8),
    (200, 200, 1000, 0),
    (64, 256, 4099, 16),
    (256, 3584, 2000, 0),
    (300, 512, 16384, 0),
]


@pytest.mark.parametrize("T,d,V,pad", SHAPES)
def test_lmhead_stats_shapes(T, d, V, pad):
    import paper_2509_23866_amd as dart

    seed = zlib.crc32(repr((T, d, V)).encode()) % 1000
    h = gaussian_bits(seed, STREAM_HIDDEN, T, d, 1.0)
    w = gaussian_bits(seed, STREAM_WEIGHT, V, d, 3.0 / math.sqrt(d))
    y = np.random.default_rng(seed).integers(0, V, T).astype(np.int32)
    ref = oracle.lmhead_token_stats(h, w, y)
    got = dart.dart_lmhead_tok_stats(_dev_bf16(h, pad), _dev_bf16(w, pad), _cuda(y))
    _check(got, ref)


def test_lmhead_stats_deterministic_and_device_inputs():
    """The device twin of the generator fills h and W bit for bit; two runs
    give bit-identical statistics."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 300, 256, 3000
    h = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    w = torch.empty((V, d), dtype=torch.bfloat16, device="cuda")
    sn.fill_gaussian_device(h, 11, STREAM_HIDDEN, 1.0)
    sn.fill_gaussian_device(w, 11, STREAM_WEIGHT, 3.0 / math.sqrt(d))
    torch.cuda.synchronize()
    hb = gaussian_bits(11, STREAM_HIDDEN, T, d, 1.0)
    wb = gaussian_bits(11, STREAM_WEIGHT, V, d, 3.0 / math.sqrt(d))
    assert np.array_equal(h.view(torch.int16).cpu().numpy().view(np.uint16), hb)
    assert np.array_equal(w.view(torch.int16).cpu().numpy().view(np.uint16), wb)
    y = _cuda(np.random.default_rng(0).integers(0, V, T).astype(np.int32))
    a = [x.clone() for x in dart.dart_lmhead_tok_stats(h, w, y)]
    b = dart.dart_lmhead_tok_stats(h, w, y)
    for u, v in zip(a, b):
        assert torch.equal(u.view(torch.int32), v.view(torch.int32))


def test_lmhead_stats_vlm7b_shape_sampled_rows():
    """T = 4096 tokens, d = 3584, V = 152064: the 7B VLM's LM head at the
    bench shape, compared on sampled rows (first, last, tile edges, random)."""
    import torch

    import paper_2509_23866_amd as dart

    prob = synth.lmhead_problem("vlm7b")
    wl, d = prob.wl, prob.d
    h = torch.empty((wl.T, d), dtype=torch.bfloat16, device="cuda")
    w = torch.empty((wl.V, d), dtype=torch.bfloat16, device="cuda")
    sn.fill_gaussian_device(h, wl.seed, STREAM_HIDDEN, prob.sigma_h)
    sn.fill_gaussian_device(w, wl.seed, STREAM_WEIGHT, prob.sigma_w)
    y = _cuda(wl.target.astype(np.int32))
    got = dart.dart_lmhead_tok_stats(h, w, y)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    rows = np.unique(np.r_[0, 1, 127, 128, 129, wl.T - 1, rng.integers(0, wl.T, 18)])
    hb = prob.hidden_bits(rows)
    wb = sn.gaussian_bits_host(wl.seed, STREAM_WEIGHT, wl.V, d, prob.sigma_w)
    ref = oracle.lmhead_token_stats(hb, wb, wl.target[rows].astype(np.int32))
    _check(got, ref, rows=rows)



@pytest.mark.parametrize("inv_temp", [None, 2.0])
def test_lmhead_dlogits_bf16_rounding(inv_temp):
    """The bf16 rounding of dz in the dlogits epilogue, bit for bit. With
    hidden rows of zeros every logit is exactly 0 and with lse = 0 every
    softmax term is exactly 1, so dz = -s g on every column but the target,
    where logp = -inf makes it s g (-expm1(-inf) = 1); s = 1 or 2 keeps s g
    exact. The coefficients sit on and beside rounding ties, in the fp32
    denormal range, and at the top of the range (rounding up to infinity);
    V = 300 ends each row with a partial 8-column chunk, and the target's
    chunk takes the epilogue's other path."""
    import torch

    import paper_2509_23866_amd as dart

    g = H.rounding_coefs()
    T, d, V = len(g), 16, 300
    h = np.zeros((T, d), dtype=np.uint16)
    w = gaussian_bits(5, STREAM_WEIGHT, V, d, 0.1)
    y = np.random.default_rng(5).integers(0, V, T).astype(np.int32)
    lse = np.zeros(T, dtype=np.float32)
    logp = np.full(T, -np.inf, dtype=np.float32)
    # the output's rows padded to a multiple of 8 elements (V = 300)
    out = torch.empty((T, V + 4), dtype=torch.bfloat16, device="cuda")[:, :V]
    dz = dart.dart_lmhead_dlogits(_dev_bf16(h), _dev_bf16(w), _cuda(y), _cuda(lse), _cuda(logp),
                                  _cuda(g), dlogits=out, inv_temp=inv_temp)
    torch.cuda.synchronize()
    got = dz.view(torch.int16).cpu().numpy().view(np.uint16)
    with np.errstate(over="ignore"):  # 2 x the fp32 maximum is inf, as on the GPU
        sg = g * np.float32(1.0 if inv_temp is None else inv_temp)
    want = np.repeat(H.rne_bf16_bits(-sg)[:, None], V, axis=1)
    want[np.arange(T), y] = H.rne_bf16_bits(sg)
    bad = np.argwhere(got != want)
    H.log(f"dlogits bf16 rounding (inv_temp={inv_temp}): {len(bad)} of {got.size} differ")
    assert len(bad) == 0, [(int(r), int(c), hex(got[r, c]), hex(want[r, c]), float(sg[r]))
                           for r, c in bad[:8]]
