"""dart_tis_loss_fwd_bwd_noalloc (the loss and gradient with the loss
workspace in the library's fixed per-GPU scratch array) against
dart_tis_loss_fwd_bwd with a caller workspace, through the C ABI: bit for bit
on three calls in a row that share the scratch array, each smaller than the
one before (many-workgroup loss with 5 and then 3 workgroups of partial sums,
then the one-workgroup loss), and against the float64 oracle at the parity
tolerances."""

import numpy as np
import pytest

import synth
from tests import _harness as H

pytestmark = pytest.mark.gpu

# (step lengths, V, dtype, seed): T = 4600, 2600, 300 tokens
CASES = [
    ([73, 120, 255, 31, 400, 97, 64, 160] * 4 + [200] * 3 + [16], 2053, "bf16", 21),
    ([41, 90, 200, 17, 300] * 4 + [648, 264], 4099, "bf16", 22),
    ([5, 30, 64, 1, 100, 100], 777, "f32", 23),
]


def _bits(t):
    import torch

    if t.dtype == torch.bfloat16:
        return t.contiguous().view(torch.int16).cpu().numpy()
    if t.dtype == torch.float64:
        return t.contiguous().view(torch.int64).cpu().numpy()
    return t.contiguous().view(torch.int32).cpu().numpy()


def test_noalloc_matches_workspace_entry_point_on_consecutive_calls():
    import torch

    import paper_2509_23866_amd as dart

    assert sum(CASES[0][0]) > sum(CASES[1][0]) > sum(CASES[2][0])
    for lens, V, dtype, seed in CASES:
        wl = synth.custom_workload(lens=lens, V=V, dtype=dtype, seed=seed, mix_kinds=True,
                                   ratio_spread=True, rho=0.5, eps_low=0.2, eps_high=0.28)
        H.log(f"noalloc case T={wl.T} V={V} {dtype} seed={seed}")
        ors = H.OracleSide(wl)
        gpu = H.GpuSide(wl, ors)
        logp, ent, lse = dart.dart_tok_stats(gpu.logits, gpu.target)
        _, mask, _ = dart.dart_step_select(ent, gpu.off, wl.rho)
        args = (gpu.logits, gpu.target, logp, lse, gpu.lp_old, gpu.lp_roll, gpu.adv, gpu.off,
                mask, gpu.eps_low, gpu.eps_high, gpu.C)
        ref_loss, ref_dz, ref_coef, ref_stats = dart.dart_tis_loss_fwd_bwd(*args, workspace="auto")
        torch.cuda.synchronize()
        loss, dz, coef, stats = dart.dart_tis_loss_fwd_bwd_noalloc(*args)
        torch.cuda.synchronize()
        for name, a, b in (("loss", loss, ref_loss), ("dlogits", dz, ref_dz),
                           ("tok_coef", coef, ref_coef), ("stats", stats, ref_stats)):
            assert np.array_equal(_bits(a), _bits(b)), f"{name} differs (T={wl.T})"

        # and the oracle's values, at the parity tolerances
        gmask = mask.cpu().numpy()
        res = ors.loss_with_mask(gmask)
        out = dict(L=float(loss.cpu().item()), g=coef.cpu().numpy(), stats=stats.cpu().numpy())
        H.check_loss(out, res, res["boundary"])
        rows = H.sample_rows(wl, res, n_random=24, seed=seed)
        ref64 = ors.dz_rows(rows, res["g"])
        sel = dz[torch.from_numpy(rows).to(dz.device)]
        got = (sel.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
               if dtype == "bf16" else sel.cpu().numpy())
        H.check_dz(got, ref64, dtype, row_ok=~res["boundary"][rows])


def test_noalloc_bad_arguments_enqueue_nothing():
    import ctypes

    import torch

    import paper_2509_23866_amd as dart

    lib = dart.load_library()
    dev = torch.device("cuda")
    x = torch.zeros(64, dtype=torch.float32, device=dev)
    y = torch.zeros(64, dtype=torch.float32, device=dev)
    p, q = x.data_ptr(), y.data_ptr()
    # S > T and C <= 0: host rules, INVALID_ARG
    for S, C in ((5, 2.0), (2, 0.0)):
        rc = lib.dart_tis_loss_fwd_bwd_noalloc(
            p, dart.DART_F32, 4, 8, 8, p, p, p, p, p, p, p, S, p, ctypes.c_float(0.2),
            ctypes.c_float(0.2), ctypes.c_float(C), q, 8, p, p, None, None)
        assert rc == dart.DART_ERR_INVALID_ARG
