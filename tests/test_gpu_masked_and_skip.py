"""GPU parity, through the C ABI, for two input classes the base parity tests
do not reach:

* masked vocabulary entries: -inf logits (probability 0, a 0 log 0 = 0 term of
  the entropy of Sec. 4.3), placed where the statistics kernel's lazy
  reference and exact-redo branch and the gradient kernel's vector and scalar
  paths meet them, in bf16 and fp32 rows, against the float64 oracle;
* the read-skipping gradient pass (DART_GRAD_SKIP_ZERO_ROWS: rows whose
  coefficient is 0 -- tokens of steps the indicator of Eq. (2) drops, tokens on
  the clipped branch of Eq. (1) -- written as zeros without reading their
  logits) at the edge workload's full size, separate and in place, against the
  oracle's gradient;
* the gradient pass's bf16 rounding, bit for bit, in the vector, head and
  tail paths of its rows.
"""

import numpy as np
import pytest

import oracle
import synth
from synth.gen import STREAM_LOGITS, gaussian_bits
from tests import _harness as H

pytestmark = pytest.mark.gpu

# tok_stats_kernel reads vector j of a row's aligned body with lane j % 768 in
# iteration j // (768 * 4); vectors hold 8 bf16 or 4 fp32 values
LANES, UNROLL = 768, 4
EPV = {"bf16": 8, "f32": 4}


def _vector_cols(v, dtype, head=0):
    return head + v * EPV[dtype] + np.arange(EPV[dtype])


def _masked_rows(dtype, V, ld, rng):
    """Logit rows (host, the dtype's bit patterns or float32) with -inf
    patterns; returns (z [T, ld], target [T], description per row). Row t of
    the device copy starts t * ld elements past a 16-byte aligned base, so
    with ld * element size not a multiple of 16 rows have unaligned heads of
    different lengths."""
    T = 12
    if dtype == "bf16":
        z = gaussian_bits(31, STREAM_LOGITS, T, ld, 3.0)
        ninf = np.uint16(0xFF80)
    else:
        z = (3.0 * rng.standard_normal((T, ld))).astype(np.float32)
        ninf = np.float32(-np.inf)
    target = rng.integers(0, V, T).astype(np.int32)
    desc = []
    per_it = LANES * UNROLL
    for t in range(T):
        esize = 2 if dtype == "bf16" else 4
        head = ((16 - (t * ld * esize) % 16) % 16) // esize
        cols = np.array([], dtype=np.int64)
        kind = t % 12
        if kind == 0:
            cols = np.flatnonzero(rng.random(V) < 0.1)
            d = "scattered 10%"
        elif kind == 1:
            cols = head + np.arange(LANES) * EPV[dtype]  # every lane's first element
            d = "first element of every lane"
        elif kind == 2:
            cols = np.concatenate([_vector_cols(v, dtype, head) for v in (5, LANES + 5, 7)])
            d = "whole 16-byte vectors"
        elif kind == 3:
            vecs = [3 + u * LANES for u in range(UNROLL)]  # lane 3, iteration 0
            cols = np.concatenate([_vector_cols(v, dtype, head) for v in vecs])
            d = "a whole iteration of one lane"
        elif kind == 4:
            cols = np.arange(V)
            d = "all but the target"
        elif kind == 5:
            target[t] = max(1, target[t])
            cols = np.setdiff1d(np.arange(V), [target[t] - 1])
            d = "all but the target and its left neighbour"
        elif kind == 6:
            nfull_cols = (V - head) // (EPV[dtype] * per_it) * EPV[dtype] * per_it
            cols = np.arange(head + nfull_cols, V)  # the vectors past the full iterations + tail
            d = "every element after the last full iteration"
        elif kind == 7:
            cols = np.array([target[t] - 1, target[t] + 1]) % V
            d = "both neighbours of the target"
        elif kind == 8:
            cols = np.array([0, V - 1, V - 2])
            d = "first and last columns"
        elif kind == 9:
            cols = np.arange(0, min(V, 8))  # the unaligned head of an odd row
            d = "the first 8 columns"
        elif kind == 10:
            cols = np.flatnonzero(rng.random(V) < 0.9)
            d = "scattered 90%"
        else:
            d = "none"
        cols = cols[(cols >= 0) & (cols < V) & (cols != target[t])]
        z[t, cols] = ninf
        desc.append(d)
    return z, target, desc


@pytest.mark.parametrize("dtype,V,ld", [("bf16", 2 * 8 * LANES * UNROLL + 8 * 100 + 5,
                                         2 * 8 * LANES * UNROLL + 8 * 100 + 5),
                                        ("bf16", 8 * LANES * UNROLL + 8 * 37 + 3,
                                         8 * LANES * UNROLL + 8 * 37 + 3 + 1),
                                        ("f32", 2 * 4 * LANES * UNROLL + 4 * 50 + 3,
                                         2 * 4 * LANES * UNROLL + 4 * 50 + 3)])
def test_masked_neg_inf_logits(dtype, V, ld):
    """Token statistics at 2e-4, the gradient within 1 bf16 ulp (fp32: 1e-5 of
    the row scale) and exactly 0 on every -inf column, for rows with -inf at
    the places listed in _masked_rows, through the statistics, the gradient and
    the whole fused call."""
    import torch

    import paper_2509_23866_amd as dart

    rng = np.random.default_rng(7 + V)
    z, target, desc = _masked_rows(dtype, V, ld, rng)
    T = z.shape[0]
    H.log(f"masked -inf rows: {dtype} V={V} ld={ld}")
    zv = z[:, :V]
    logp, Hh, lse = oracle.token_stats(np.ascontiguousarray(zv), target)
    dev = torch.device("cuda")
    if dtype == "bf16":
        zt = torch.from_numpy(z.view(np.int16)).to(dev).view(torch.bfloat16)[:, :V]
    else:
        zt = torch.from_numpy(z).to(dev)[:, :V]
    tt = torch.from_numpy(target).to(dev)
    glogp, gH, glse = dart.dart_tok_stats(zt, tt)
    torch.cuda.synchronize()
    for name, got, ref in (("logp", glogp, logp), ("entropy", gH, Hh), ("lse", glse, lse)):
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref)
        bad = np.flatnonzero(~(err <= 2e-4))
        assert bad.size == 0, f"{name} off at rows {[(int(i), desc[i]) for i in bad]}"
    assert abs(float(gH[4].item())) == 0.0 and float(glogp[4].item()) == 0.0  # one finite entry

    # the gradient kernel alone, fed coefficients of both signs
    g = ((np.arange(T) % 3) - 1.0) * 0.01 * (1 + np.arange(T))
    g32 = g.astype(np.float32)
    gd = torch.from_numpy(g32).to(dev)
    dz = dart.dart_tis_grad(zt, tt, glogp, glse, gd)
    torch.cuda.synchronize()
    ref = oracle.dlogits(np.ascontiguousarray(zv), target, lse, logp, g32.astype(np.float64))
    if dtype == "bf16":
        got = dz.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        gotf = synth.bf16_bits_to_f32(got)
        masked = zv == np.uint16(0xFF80)
    else:
        got = dz.cpu().numpy()
        gotf = got
        masked = np.isneginf(zv)
    H.check_dz(got, ref, dtype)
    assert np.all(gotf[masked] == 0.0)

    # the whole fused call: three steps, every step kept, clipping off
    off = torch.tensor([0, 4, 8, T], dtype=torch.int32, device=dev)
    mask = torch.ones(3, dtype=torch.uint8, device=dev)
    lp_old = glogp.clone()
    adv_np = rng.standard_normal(T).astype(np.float32)
    adv = torch.from_numpy(adv_np).to(dev)
    loss, dz2, coef, _ = dart.dart_tis_loss_fwd_bwd(zt, tt, glogp, glse, lp_old, lp_old, adv, off,
                                                    mask, 0.2, 0.2, 2.0)
    torch.cuda.synchronize()
    # ratio 1 and weight 1: loss = -mean(A), g = -A / T
    want = -float(adv_np.astype(np.float64).mean())
    assert abs(float(loss.item()) - want) <= 1e-12 * max(1.0, abs(want))
    gref = -adv_np.astype(np.float64) / T
    assert np.allclose(coef.cpu().numpy(), gref, rtol=1e-6, atol=0)
    ref2 = oracle.dlogits(np.ascontiguousarray(zv), target, lse, logp,
                          gref.astype(np.float32).astype(np.float64))
    if dtype == "bf16":
        got2 = dz2.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.all(synth.bf16_bits_to_f32(got2)[masked] == 0.0)
    else:
        got2 = dz2.cpu().numpy()
        assert np.all(got2[masked] == 0.0)
    H.check_dz(got2, ref2, dtype)


@pytest.mark.slow
@pytest.mark.parametrize("inplace", [False, True])
def test_skip_zero_rows_edge_against_oracle(inplace):
    """The edge workload at full size (T = 16384, V = 151936, rho = 0.25: three
    quarters of the steps dropped, plus clipped tokens): the read-skipping
    gradient is within 1 bf16 ulp of the oracle's on sampled rows (rows with a
    zero coefficient among them), every row with a zero coefficient is exactly
    zero, and the result equals the dense pass's (+0 == -0). In place, the
    logits buffer receives the gradient."""
    import torch

    import paper_2509_23866_amd as dart

    wl = synth.make_workload("edge")
    H.log(f"skip rows vs oracle: edge T={wl.T} V={wl.V} inplace={inplace}")
    ors = H.OracleSide(wl)
    gpu = H.GpuSide(wl, ors, inplace=False)
    logp, ent, lse = dart.dart_tok_stats(gpu.logits, gpu.target)
    _, mask, _ = dart.dart_step_select(ent, gpu.off, wl.rho)
    loss, coef, _ = dart.dart_tis_loss_fwd(logp, gpu.lp_old, gpu.lp_roll, gpu.adv, gpu.off, mask,
                                           gpu.eps_low, gpu.eps_high, gpu.C)
    dense = dart.dart_tis_grad(gpu.logits, gpu.target, logp, lse, coef)
    if inplace:
        out = gpu.logits
    else:
        out = torch.full_like(gpu.logits, float("nan"))  # every element must be written
    skip = dart.dart_tis_grad(gpu.logits, gpu.target, logp, lse, coef, dlogits=out,
                              skip_zero_rows=True)
    torch.cuda.synchronize()
    assert skip.data_ptr() == out.data_ptr()
    zero = coef == 0
    frac = float(zero.float().mean().item())
    H.log(f"zero-coefficient rows: {frac:.3f}")
    assert frac > 0.7
    assert bool((skip[zero] == 0).all().item())
    assert bool((skip == dense).all().item())

    # against the oracle, with the GPU's own mask (identical to the oracle's here)
    res = ors.loss_with_mask(mask.cpu().numpy())
    assert abs(float(loss.item()) - res["L"]) <= 1e-4 * abs(res["L"])
    rows = H.sample_rows(wl, res, n_random=40, seed=5)
    zero_rows = np.flatnonzero(coef.cpu().numpy() == 0)
    rows = np.union1d(rows, zero_rows[:: max(1, zero_rows.size // 16)])
    ref64 = ors.dz_rows(rows, res["g"])
    sel = skip[torch.from_numpy(rows).to(skip.device)]
    got = sel.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    H.check_dz(got, ref64, "bf16", row_ok=~res["boundary"][rows])


@pytest.mark.parametrize("V,ld,out_ld", [(1000, 1000, 1000), (1003, 1011, 1011), (1003, 1011, 1003)])
def test_tis_grad_bf16_rounding(V, ld, out_ld):
    """dlogits leave the gradient pass rounded to bf16 to nearest even, bit for
    bit: with logits of exactly 0 and lse = 0 every softmax term is exactly 1,
    so dz = -g on every column but the target, where logp = -inf makes it g
    (-expm1(-inf) = 1). The coefficients sit on and beside rounding ties, in
    the fp32 denormal range and at the top of the range. Rows ld = 1011
    elements apart start unaligned: with the output rows as far apart their
    heads and tails take the kernel's scalar paths around the vector body,
    with contiguous output rows (other heads) the whole row takes them."""
    import torch

    import paper_2509_23866_amd as dart

    g = H.rounding_coefs()
    T = len(g)
    logits = torch.zeros((T, ld), dtype=torch.bfloat16, device="cuda")[:, :V]
    y = np.random.default_rng(7).integers(0, V, T).astype(np.int32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    out = torch.empty((T, out_ld), dtype=torch.bfloat16, device="cuda")[:, :V]
    dz = dart.dart_tis_grad(logits, dev(y), dev(np.full(T, -np.inf, dtype=np.float32)),
                            dev(np.zeros(T, dtype=np.float32)), dev(g), dlogits=out)
    torch.cuda.synchronize()
    got = dz.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    want = np.repeat(H.rne_bf16_bits(-g)[:, None], V, axis=1)
    want[np.arange(T), y] = H.rne_bf16_bits(g)
    bad = np.argwhere(got != want)
    H.log(f"tis_grad bf16 rounding V={V} ld={ld} out_ld={out_ld}: {len(bad)} of {got.size} differ")
    assert len(bad) == 0, [(int(r), int(c), hex(got[r, c]), hex(want[r, c]), float(g[r]))
                           for r, c in bad[:8]]
