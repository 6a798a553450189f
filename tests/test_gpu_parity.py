"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Small shapes span several tiles of the streaming kernels (8192 bf16 elements
per workgroup iteration) plus ragged tails, odd and tiny vocabularies,
unaligned and padded rows, in-place gradients, every row kind and the
degenerate selections; the five named workloads run at their full sizes in the
launch configuration the benchmark times, with every per-token and per-step
output compared and the gradient compared element-wise on sampled rows.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import _harness as H

pytestmark = pytest.mark.gpu


def _full_check(wl, ld=None, misalign=0, inplace=None, dz_rows=None, fused=True):
    ors = H.OracleSide(wl)
    gpu_side = H.GpuSide(wl, ors, ld=ld, misalign=misalign, inplace=inplace)
    rows = dz_rows if dz_rows is not None else np.arange(wl.T)
    gpu = gpu_side.run(keep_rows=rows, fused=fused)
    stats_err = H.check_token_stats(gpu, ors)
    same_mask = H.check_mask(gpu, ors)
    res = ors.res
    if not same_mask:
        # the selections differ only inside the near-tie band: compare the loss
        # and gradient of the GPU path given the oracle's mask as input
        H.log(f"{wl.name}: masks differ inside the tie band; rerunning with the oracle mask")
        gpu_side = H.GpuSide(wl, ors, ld=ld, misalign=misalign, inplace=inplace)
        gpu = gpu_side.run(mask=ors.mask, keep_rows=rows)
    # only ratios at a clip bound may be excused from the element-wise checks
    assert res["boundary"].mean() <= 0.01, f"{res['boundary'].sum()} boundary tokens"
    loss_err = H.check_loss(gpu, res, res["boundary"])
    ref = ors.dz_rows(rows)
    ok = ~res["boundary"][rows]
    dz_err = H.check_dz(gpu["dz"], ref, wl.dtype, row_ok=ok)
    H.log(f"{wl.name}: logp {stats_err['logp']:.2e} H {stats_err['H']:.2e} "
          f"loss rel {loss_err:.2e} dz {dz_err:.2f} ulp, mask {'equal' if same_mask else 'band'}")
    return ors, gpu


SMALL = [
    # (lens, V, dtype, extra kwargs)
    ([3, 5, 1, 7], 4099, "bf16", {}),
    ([2, 2, 2], 1, "bf16", {}),
    ([4, 1, 3], 7, "bf16", {}),
    ([5, 5], 8, "f32", {}),
    ([6, 2, 9], 9, "f32", {}),
    ([3, 4, 5, 6], 63, "bf16", dict(mix_kinds=True)),
    ([8, 8, 8], 8192 * 3 + 5, "bf16", dict(mix_kinds=True, ratio_spread=True)),
    ([7, 1, 1, 9], 1000, "f32", dict(ratio_spread=True)),
    ([16] * 6, 4096 * 5 + 3, "f32", dict(mix_kinds=True)),
    ([1], 33, "bf16", {}),
    ([30, 2], 152064, "bf16", dict(ratio_spread=True, mix_kinds=True)),
    ([5, 9, 3], 151936, "bf16", dict(rho=0.25, C=float("inf"))),
    ([4, 4, 4, 4], 2048, "bf16", dict(rho=0.0)),
    ([4, 4, 4, 4], 2048, "bf16", dict(rho=1.0, eps_low=0.1, eps_high=0.5, C=1.0)),
    ([4, 6, 2], 20000, "bf16", dict(inplace=True, ratio_spread=True)),
    ([4, 6, 2], 20001, "f32", dict(inplace=True)),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_shapes(case):
    lens, V, dtype, kw = SMALL[case]
    wl = synth.custom_workload(lens=lens, V=V, dtype=dtype, seed=100 + case, **kw)
    _full_check(wl)


def _random_case(seed):
    """A seeded random configuration: 1-25 steps of 1-120 tokens, V from 1 to
    40000 (often just off a multiple of 8 or of the 2048-element chunk), fp32 or
    bf16, padded or misaligned rows, any rho, the wide or narrow ratio model,
    C finite or infinite."""
    rng = np.random.default_rng(1000 + seed)
    lens = rng.integers(1, 121, int(rng.integers(1, 26)))
    V = int(rng.choice([rng.integers(1, 64), rng.integers(64, 40001),
                        8 * rng.integers(1, 5000) + rng.integers(-1, 2),
                        2048 * rng.integers(1, 20) + rng.integers(-1, 2)]))
    V = max(V, 1)
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    kw = dict(rho=float(rng.choice([0.0, 0.25, 0.5, 0.8, 1.0, rng.random()])),
              C=float(rng.choice([1.0, 2.0, 5.0, float("inf")])),
              ratio_spread=bool(rng.random() < 0.5), mix_kinds=bool(rng.random() < 0.5))
    layout = dict(ld=None, misalign=0)
    r = rng.random()
    if r < 0.25:
        layout["ld"] = V + int(rng.integers(1, 17))
    elif r < 0.4:
        layout["misalign"] = 1
    return lens, V, dtype, kw, layout


@pytest.mark.parametrize("seed", range(24))
def test_random_shapes(seed):
    """24 seeded random configurations through the whole path against the oracle."""
    lens, V, dtype, kw, layout = _random_case(seed)
    wl = synth.custom_workload(lens=lens, V=V, dtype=dtype, seed=500 + seed, **kw)
    H.log(f"random case {seed}: S={lens.size} T={int(lens.sum())} V={V} {dtype} {kw} {layout}")
    _full_check(wl, **layout)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("V,ld,misalign", [(4099, 4107, 0), (5000, 5003, 0), (777, 777, 1),
                                           (8200, 8203, 3)])
def test_strided_and_unaligned_rows(dtype, V, ld, misalign):
    """Padded rows (the padding holds NaN and must never be read) and rows that
    do not start on a 16-byte boundary."""
    wl = synth.custom_workload(lens=[3, 4, 2], V=V, dtype=dtype, seed=7, mix_kinds=True)
    _full_check(wl, ld=ld, misalign=misalign)
    _full_check(wl, ld=ld, misalign=misalign, inplace=True)


@pytest.mark.parametrize("fused", [True, False])  # the benchmark's calls, and the separate ones
@pytest.mark.parametrize("name", ["tiny", "vlm7b", "edge"])
def test_named_workload(name, fused):
    wl = synth.make_workload(name)
    rows = None if wl.T * wl.V <= (1 << 22) else H.sample_rows(wl, _oracle_g_placeholder(wl))
    _full_check(wl, dz_rows=rows, fused=fused)


def _oracle_g_placeholder(wl):
    # sample_rows only uses |g| to pick extra rows; before the oracle has run,
    # advantages stand in for it
    return dict(g=np.abs(wl.adv).astype(np.float64))


@pytest.mark.slow
@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["microbatch", "longhorizon"])
def test_named_workload_large(name):
    wl = synth.make_workload(name)
    rows = H.sample_rows(wl, _oracle_g_placeholder(wl), n_random=32)
    _full_check(wl, dz_rows=rows)


def test_edge_ties_are_exact():
    """Identical rows give bit-identical entropies, identical steps identical
    step entropies, and the flat steps straddling the selection boundary are
    kept lowest index first (the mask equals the oracle's exactly)."""
    wl = synth.make_workload("edge")
    ors, gpu = _full_check(wl, dz_rows=np.array([0, 1, wl.T - 1]))
    copies = np.flatnonzero(wl.src_row != np.arange(wl.T))
    src = wl.src_row[copies]
    assert np.array_equal(gpu["H"][copies].view(np.uint32), gpu["H"][src].view(np.uint32))
    flat = np.flatnonzero(wl.kind == synth.gen.KIND_FLAT)
    assert np.unique(gpu["H"][flat].view(np.uint32)).size == 1
    assert np.array_equal(gpu["mask"], ors.mask)
    flat_steps = np.unique(flat // 64)
    kept_flat = flat_steps[gpu["mask"][flat_steps] == 1]
    assert kept_flat.size == ors.k and np.array_equal(kept_flat, flat_steps[: ors.k])


def test_deterministic_repeat():
    wl = synth.make_workload("vlm7b")
    ors = H.OracleSide(wl)
    side = H.GpuSide(wl, ors)
    rows = np.arange(0, wl.T, 97)
    a = side.run(keep_rows=rows)
    b = side.run(keep_rows=rows)
    for key in ("logp", "H", "lse", "Hs", "mask", "g", "dz"):
        assert np.array_equal(np.asarray(a[key]).view(np.uint8), np.asarray(b[key]).view(np.uint8)), key
    assert a["L"] == b["L"]


def test_device_generator_matches_host():
    """The device twin of the generator writes the same bits as the host twin."""
    import torch

    import synth.native as sn

    for name in ("tiny", "edge"):
        wl = synth.make_workload(name)
        rows = np.unique(np.r_[0, wl.T - 1, np.linspace(0, wl.T - 1, 9).astype(np.int64)])
        t = torch.empty((wl.T, wl.V), dtype=torch.float32 if wl.dtype == "f32" else torch.bfloat16,
                        device="cuda")
        sn.fill_logits_device(sn.DeviceRecipe(wl), t)
        got = t[torch.from_numpy(rows).cuda()].cpu()
        got = got.numpy() if wl.dtype == "f32" else got.view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(got, sn.logits_rows_host(wl, rows))


def test_tok_stats_rows_beyond_one_launch():
    """2^22 + 999 rows of V = 8 bf16 logits, more rows than one launch of the
    statistics takes: rows on both sides of row 2^22, the first and last rows
    and a random sample against the oracle (tolerances of the named workloads)."""
    import torch

    import paper_2509_23866_amd as dart

    T, V = (1 << 22) + 999, 8
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    logits = (torch.randn((T, V), device="cuda", generator=g) * 3.0).to(torch.bfloat16)
    target = torch.randint(0, V, (T,), device="cuda", generator=g, dtype=torch.int32)
    logp, ent, lse = dart.dart_tok_stats(logits, target)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    rows = np.unique(np.r_[0, 1, (1 << 22) - 2, (1 << 22) - 1, 1 << 22, (1 << 22) + 1, T - 1,
                           rng.integers(0, T, 200)])
    idx = torch.from_numpy(rows).cuda()
    z = logits[idx].view(torch.int16).cpu().numpy().view(np.uint16)
    y = target[idx].cpu().numpy()
    rlogp, rH, rlse = oracle.token_stats(z, y)
    for got, ref, name in ((logp, rlogp, "logp"), (ent, rH, "entropy"), (lse, rlse, "lse")):
        err = np.abs(got[idx].double().cpu().numpy() - ref)
        assert err.max() <= 2e-4, (name, float(err.max()), rows[int(err.argmax())])


@pytest.mark.timeout(600)
def test_whole_path_beyond_the_grid_limits():
    """T = 2^24 + 1000 rows of V = 8 bf16 logits in 1000 steps: the statistics
    run in five launches of at most 2^22 rows, and the gradient pass has more
    4 KB chunks (one per row) than its 2^24 workgroups, so it takes its
    grid-stride loop. The whole path (policy_update) against the oracle: every
    token's logp and entropy, the mask, the loss, and the gradient on rows
    sampled across both limits."""
    import torch

    import paper_2509_23866_amd as dart

    T, V, S = (1 << 24) + 1000, 8, 1000
    rng = np.random.default_rng(24)
    z32 = (rng.standard_normal((T, V), dtype=np.float32) * 3.0)
    z = synth.f32_to_bf16_bits(z32)
    del z32
    target = rng.integers(0, V, T).astype(np.int32)
    cuts = np.sort(rng.choice(np.arange(1, T), S - 1, replace=False))
    off = np.r_[0, cuts, T].astype(np.int32)
    adv = rng.standard_normal(T).astype(np.float32)
    logp0, _, _ = oracle.token_stats(z, target)
    lp_old = (logp0 + 0.05 * rng.standard_normal(T)).astype(np.float32)
    lp_roll = (lp_old + 0.1 * rng.standard_normal(T)).astype(np.float32)
    rho, eps_low, eps_high, C = 0.8, 0.2, 0.28, 2.0
    ref = oracle.forward_backward(z, target, lp_old, lp_roll, adv, off, rho, eps_low, eps_high, C)
    cuda = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    logits = cuda(z.view(np.int16)).view(torch.bfloat16)
    out = dart.policy_update(logits, cuda(target), cuda(lp_old), cuda(lp_roll), cuda(adv),
                             cuda(off), rho, eps_low, eps_high, C)
    torch.cuda.synchronize()
    assert np.abs(out["logp"].cpu().numpy() - ref["logp"]).max() <= 2e-4
    assert np.abs(out["entropy"].cpu().numpy() - ref["H"]).max() <= 2e-4
    assert np.array_equal(out["step_mask"].cpu().numpy(), ref["mask"])
    L = float(out["loss"].cpu().item())
    assert abs(L - ref["L"]) <= 1e-4 * abs(ref["L"])
    rows = np.unique(np.r_[0, (1 << 22) - 1, 1 << 22, (1 << 24) - 1, 1 << 24, T - 1,
                           rng.integers(0, T, 300)])
    rows = rows[~ref["boundary"][rows]]
    got = out["dlogits"][torch.from_numpy(rows).cuda()].view(torch.int16).cpu().numpy()
    got = synth.bf16_bits_to_f32(got.view(np.uint16)).astype(np.float64)
    want_bits = oracle.f64_to_bf16_bits(ref["dz"][rows])
    want = synth.bf16_bits_to_f32(want_bits).astype(np.float64)
    assert np.all(np.abs(got - want) <= oracle.bf16_ulp(want_bits))
