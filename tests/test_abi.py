"""The C-ABI library loads, exports every function include/dart.h declares,
and rejects bad scalar arguments on the host (no device work is enqueued for
any case here)."""

import ctypes
import math
import os
import re

import pytest

import paper_2509_23866_amd as dart

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            with open(os.path.join(ROOT, "include", fn)) as fh:
                text = fh.read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names.update(re.findall(r"\b(dart_[a-z_0-9]+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    lib = dart.load_library()
    declared = _declared_functions()
    assert {"dart_tok_stats", "dart_step_select", "dart_tis_loss_fwd_bwd"} <= declared
    for name in declared:
        assert hasattr(lib, name), f"{name} is declared in include/ but not exported"
    assert set(dart.EXPORTED) == declared


def test_kept_steps_host_helper():
    for rho, S, k in [(0.8, 240, 192), (0.8, 64, 52), (0.5, 16, 8), (0.5, 1600, 800),
                      (0.25, 256, 64), (0.0, 9, 0), (1.0, 9, 9), (0.01, 3, 1)]:
        assert dart.dart_kept_steps(S, rho) == k
    assert dart.dart_kept_steps(10, 1.5) == -1
    assert dart.dart_kept_steps(10, -0.1) == -1
    assert dart.dart_kept_steps(10, float("nan")) == -1
    assert dart.dart_kept_steps(-1, 0.5) == -1


def test_status_strings():
    assert dart.dart_status_string(0) == "DART_OK"
    assert dart.dart_status_string(1) == "DART_ERR_INVALID_ARG"
    assert dart.dart_status_string(3) == "DART_ERR_HIP"
    assert dart.dart_status_string(42) == "DART_ERR_UNKNOWN"


def _gpu_visible():
    import torch

    return torch.cuda.device_count() > 0


# Fake, never-dereferenced addresses. Every call below fails a host-side check
# before any launch; on a machine with a GPU the module skips them anyway.
P = 4096
INF = float("inf")


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("args", [
    (0, 1, 4, 8, 8, P, P, P, P),          # null logits
    (P, 1, 4, 8, 8, 0, P, P, P),          # null target
    (P, 1, 4, 8, 8, P, 0, P, P),          # null logp
    (P, 1, 0, 8, 8, P, P, P, P),          # T = 0
    (P, 1, 4, 0, 8, P, P, P, P),          # V = 0
    (P, 1, 4, 8, 7, P, P, P, P),          # ld < V
    (P, 7, 4, 8, 8, P, P, P, P),          # unknown dtype
    (P + 1, 1, 4, 8, 8, P, P, P, P),      # bf16 logits not 2-byte aligned
])
def test_tok_stats_rejects(args):
    lib = dart.load_library()
    assert lib.dart_tok_stats(*args, None) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("T,S,rho,null", [
    (10, 0, 0.5, None), (10, 11, 0.5, None), (0, 1, 0.5, None), (10, 2, 1.01, None),
    (10, 2, -0.01, None), (10, 2, float("nan"), None), (10, 2, 0.5, 0), (10, 2, 0.5, 2),
    (10, 2, 0.5, 5), (10, 2, 0.5, 6),
])
def test_step_select_rejects(T, S, rho, null):
    lib = dart.load_library()
    ptrs = [P, P, P, P, P]  # entropy, offsets, step_entropy, mask, n_kept
    idx = {0: 0, 2: 1, 5: 2, 6: 3}
    if null is not None:
        ptrs[idx[null]] = 0
    rc = lib.dart_step_select(ptrs[0], T, ptrs[1], S, rho, ptrs[2], ptrs[3], ptrs[4], None)
    assert rc == dart.DART_ERR_INVALID_ARG


def _tis_args(**kw):
    a = dict(logits=P, dtype=1, T=4, V=8, ld=8, target=P, logp=P, lse=P, lp_old=P, lp_roll=P,
             adv=P, off=P, S=2, mask=P, eps_low=0.2, eps_high=0.2, C=2.0, dlogits=1 << 20,
             ld_out=8, loss=P, coef=P, stats=0, workspace=0, workspace_bytes=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(logits=0), dict(target=0), dict(logp=0), dict(lse=0), dict(lp_old=0), dict(lp_roll=0),
    dict(adv=0), dict(off=0), dict(mask=0), dict(dlogits=0), dict(loss=0), dict(coef=0),
    dict(T=0), dict(V=0), dict(ld=7), dict(ld_out=7), dict(S=0), dict(S=5), dict(dtype=3),
    dict(eps_low=-0.1), dict(eps_high=float("nan")), dict(C=0.0), dict(C=-1.0),
    dict(C=float("nan")), dict(dlogits=P + 2),  # partial overlap with logits
    dict(dlogits=P, ld_out=9),  # same base, different stride
    dict(dlogits=(1 << 20) + 1),  # bf16 output not 2-byte aligned
    dict(workspace=1 << 24, workspace_bytes=55),  # one byte short for T = 4
    dict(workspace=(1 << 24) + 4, workspace_bytes=1 << 16),  # not 8-byte aligned
])
def test_tis_loss_rejects(kw):
    lib = dart.load_library()
    assert lib.dart_tis_loss_fwd_bwd(*_tis_args(**kw), None) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(logits=0), dict(target=0), dict(logp=0), dict(lse=0), dict(lp_old=0), dict(lp_roll=0),
    dict(adv=0), dict(off=0), dict(mask=0), dict(dlogits=0), dict(loss=0), dict(coef=0),
    dict(T=0), dict(T=1 << 31), dict(V=0), dict(ld=7), dict(ld_out=7), dict(S=0), dict(S=5),
    dict(dtype=3), dict(eps_low=-0.1), dict(eps_high=float("nan")), dict(C=0.0),
    dict(C=float("nan")), dict(dlogits=P + 2), dict(dlogits=P, ld_out=9),
    dict(dlogits=(1 << 20) + 1),
])
def test_tis_loss_noalloc_rejects_before_any_hip_call(kw):
    """The no-allocation entry point applies dart_tis_loss_fwd_bwd's host rules
    before it looks up its scratch array (no GPU here: a HIP call would fail)."""
    lib = dart.load_library()
    args = _tis_args(**kw)[:-2]  # no workspace arguments
    assert lib.dart_tis_loss_fwd_bwd_noalloc(*args, None) == dart.DART_ERR_INVALID_ARG


def _select_loss_args(**kw):
    a = dict(T=4, entropy=P, logp=P, lp_old=P, lp_roll=P, adv=P, off=P, S=2, rho=0.5,
             eps_low=0.2, eps_high=0.2, C=2.0, step_entropy=P, mask=P, n_kept=0, loss=P, coef=P,
             stats=0, workspace=0, workspace_bytes=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(entropy=0), dict(logp=0), dict(lp_old=0), dict(lp_roll=0), dict(adv=0), dict(off=0),
    dict(step_entropy=0), dict(mask=0), dict(loss=0), dict(coef=0), dict(T=0), dict(T=1 << 31),
    dict(S=0), dict(S=5), dict(rho=1.01), dict(rho=-0.01), dict(rho=float("nan")),
    dict(eps_low=-0.1), dict(eps_high=float("nan")), dict(C=0.0), dict(C=float("nan")),
    dict(workspace=1 << 24, workspace_bytes=55),  # one byte short for T = 4
    dict(workspace=(1 << 24) + 4, workspace_bytes=1 << 16),  # not 8-byte aligned
    # too large for one workgroup: still rejected before the two calls begin
    dict(T=20000, S=20001), dict(T=20000, S=3, rho=2.0), dict(T=20000, S=3, C=-1.0),
])
def test_select_tis_loss_rejects(kw):
    """The fused selection and loss call applies the rules of dart_step_select
    and dart_tis_loss_fwd on the host before anything is enqueued."""
    lib = dart.load_library()
    assert lib.dart_select_tis_loss_fwd(*_select_loss_args(**kw), None) == \
        dart.DART_ERR_INVALID_ARG


def test_workspace_bytes():
    """kParts = 5 doubles per workgroup of 1024 tokens (at most 1024
    workgroups), then N and K."""
    lib = dart.load_library()
    f = lib.dart_tis_loss_workspace_bytes
    assert f(0) == 0 and f(-3) == 0 and f(1 << 31) == 0
    assert f(1) == 56 and f(1024) == 56 and f(1025) == 96
    assert f(1024 * 1024) == (1024 * 5 + 2) * 8 and f((1 << 31) - 1) == (1024 * 5 + 2) * 8


def test_python_binding_requires_built_library(monkeypatch, tmp_path):
    """No CPU fallback: a missing library is an error, not a silent path."""
    monkeypatch.setattr(dart, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(dart, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        dart.load_library()


class _Cfg:
    pass


def _loss_ex_args(lib, **kw):
    import paper_2509_23866_amd as d

    cfg = d.dart_loss_config_t(0.2, 0.28, 2.0, kw.pop("kl", 0), kw.pop("beta", 0.0),
                               kw.pop("aggregation", 0), kw.pop("ratio", 0))
    a = dict(T=4, logp=P, lp_old=P, lp_roll=P, lp_ref=0, adv=P, off=P, S=2, mask=P, cfg=cfg,
             loss=P, coef=P, stats=0, workspace=0, workspace_bytes=0)
    a.update(kw)
    cfgp = None if a["cfg"] is None else ctypes.byref(a["cfg"])
    return [a["T"], a["logp"], a["lp_old"], a["lp_roll"], a["lp_ref"], a["adv"], a["off"], a["S"],
            a["mask"], cfgp, a["loss"], a["coef"], a["stats"], a["workspace"],
            a["workspace_bytes"], None]


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(cfg=None), dict(kl=4), dict(kl=-1), dict(aggregation=3), dict(ratio=3),
    dict(kl=3, lp_ref=0), dict(kl=1, lp_ref=P, beta=-0.1), dict(kl=1, lp_ref=P, beta=float("inf")),
    dict(T=0), dict(S=5), dict(logp=0), dict(coef=0),
    dict(workspace=1 << 24, workspace_bytes=8),
])
def test_tis_loss_fwd_ex_rejects(kw):
    lib = dart.load_library()
    assert lib.dart_tis_loss_fwd_ex(*_loss_ex_args(lib, **kw)) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("inv_temp,flags", [(0.0, 0), (-1.0, 0), (float("inf"), 0),
                                            (float("nan"), 0), (1.0, 2), (1.0, 0x80000000)])
def test_ex_temperature_and_flags_rejected(inv_temp, flags):
    lib = dart.load_library()
    assert lib.dart_tok_stats_ex(P, 1, 4, 8, 8, P, inv_temp if flags == 0 else 0.0, P, P, P,
                                 None) == dart.DART_ERR_INVALID_ARG
    assert lib.dart_tis_grad_ex(P, 1, 4, 8, 8, P, P, P, P, inv_temp, flags, 1 << 20, 8,
                                None) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [dict(reward=0), dict(traj=0), dict(grp=0), dict(off=0), dict(adv=0),
                                dict(n_traj=0), dict(G=0), dict(G=5), dict(S=0), dict(S=11)])
def test_grpo_advantage_rejects(kw):
    lib = dart.load_library()
    a = dict(reward=P, n_traj=4, traj=P, grp=P, G=2, off=P, S=8, T=10, adv=P)
    a.update(kw)
    assert lib.dart_grpo_advantage(a["reward"], a["n_traj"], a["traj"], a["grp"], a["G"], a["off"],
                                   a["S"], a["T"], a["adv"], None, None, None) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [dict(grp=0), dict(G=0), dict(G=9), dict(rho=1.5), dict(S=0),
                                dict(entropy=0), dict(mask=0)])
def test_step_select_groups_rejects(kw):
    lib = dart.load_library()
    a = dict(entropy=P, T=10, off=P, S=8, grp=P, G=2, rho=0.5, sh=P, mask=P)
    a.update(kw)
    assert lib.dart_step_select_groups(a["entropy"], a["T"], a["off"], a["S"], a["grp"], a["G"],
                                       a["rho"], a["sh"], a["mask"], None, None) == dart.DART_ERR_INVALID_ARG


def _lm_args(**kw):
    a = dict(hidden=1 << 20, T=4, d=16, ld_h=16, weight=1 << 21, V=300, ld_w=16, target=P,
             logp=P, H=P, lse=P, workspace=1 << 22, ws_bytes=1 << 20)
    a.update(kw)
    return list(a.values()) + [None]


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(hidden=0), dict(weight=0), dict(target=0), dict(logp=0), dict(H=0), dict(lse=0),
    dict(workspace=0), dict(T=0), dict(V=0), dict(d=4, ld_h=4, ld_w=4), dict(d=12, ld_h=16, ld_w=16),
    dict(ld_h=12), dict(ld_w=20), dict(ld_h=8), dict(hidden=(1 << 20) + 8),
    dict(weight=(1 << 21) + 2), dict(workspace=(1 << 22) + 4), dict(ws_bytes=4 * 2 * 16 + 15),
])
def test_lmhead_stats_rejects(kw):
    lib = dart.load_library()
    assert lib.dart_lmhead_tok_stats(*_lm_args(**kw)) == dart.DART_ERR_INVALID_ARG
    a = _lm_args(**kw)
    assert lib.dart_lmhead_tok_stats_ex(*a[:8], 1.0, *a[8:]) == dart.DART_ERR_INVALID_ARG


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("inv_temp", [0.0, -1.0, float("inf"), float("nan"), -0.0])
def test_lmhead_inverse_temperature_rejects(inv_temp):
    """An inverse temperature that is not finite and positive, with every other
    argument valid, is INVALID_ARG for the statistics and the backward."""
    lib = dart.load_library()
    a = _lm_args()
    assert lib.dart_lmhead_tok_stats_ex(*a[:8], inv_temp, *a[8:]) == dart.DART_ERR_INVALID_ARG
    assert (lib.dart_lmhead_backward_ex(*_lm_bwd_ex_args(inv_temp=inv_temp))
            == dart.DART_ERR_INVALID_ARG)
    g = _lm_grad_args()
    assert lib.dart_lmhead_dlogits_ex(*g[:11], inv_temp, *g[11:]) == dart.DART_ERR_INVALID_ARG


def test_lmhead_workspace_bytes():
    """One 16-byte partial triple per row and 256-column slice, plus the
    target logit per row."""
    f = dart.load_library().dart_lmhead_stats_workspace_bytes
    assert f(0, 10) == 0 and f(10, 0) == 0 and f(1 << 31, 5) == 0
    assert f(4, 300) == 4 * 2 * 16 + 16
    assert f(4096, 152064) == 4096 * 594 * 16 + 4096 * 4


def _lm_grad_args(**kw):
    a = dict(hidden=1 << 20, T=4, d=16, ld_h=16, weight=1 << 21, V=300, ld_w=16, target=P,
             lse=P, logp=P, coef=P, out=1 << 23, ld_out=304)
    a.update(kw)
    return list(a.values()) + [None]


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(hidden=0), dict(weight=0), dict(target=0), dict(lse=0), dict(logp=0), dict(coef=0),
    dict(out=0), dict(T=0), dict(V=0), dict(d=12, ld_h=16, ld_w=16), dict(ld_w=12),
    dict(ld_out=296), dict(ld_out=302), dict(out=(1 << 23) + 8), dict(hidden=(1 << 20) + 2),
])
def test_lmhead_dlogits_rejects(kw):
    lib = dart.load_library()
    assert lib.dart_lmhead_dlogits(*_lm_grad_args(**kw)) == dart.DART_ERR_INVALID_ARG
    g = _lm_grad_args(**kw)
    assert lib.dart_lmhead_dlogits_ex(*g[:11], 1.0, *g[11:]) == dart.DART_ERR_INVALID_ARG


def _lm_bwd_args(**kw):
    a = dict(hidden=1 << 20, T=4, d=16, ld_h=16, weight=1 << 21, V=300, ld_w=16, target=P,
             lse=P, logp=P, coef=P, dh=1 << 23, ld_dh=16, dw=1 << 24, ld_dw=16, chunk=2,
             workspace=1 << 22, ws_bytes=2 * 304 * 2)
    a.update(kw)
    return list(a.values()) + [None]


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(hidden=0), dict(weight=0), dict(target=0), dict(lse=0), dict(logp=0), dict(coef=0),
    dict(dh=0), dict(dw=0), dict(workspace=0), dict(T=0), dict(V=0), dict(d=4, ld_h=4, ld_w=4),
    dict(ld_dh=15), dict(ld_dw=8), dict(chunk=0), dict(ws_bytes=2 * 304 * 2 - 1),
    dict(chunk=9, ws_bytes=4 * 304 * 2 - 2), dict(workspace=(1 << 22) + 8),
])
def test_lmhead_backward_rejects(kw):
    lib = dart.load_library()
    assert lib.dart_lmhead_backward(*_lm_bwd_args(**kw)) == dart.DART_ERR_INVALID_ARG


def test_lmhead_backward_workspace_bytes():
    """One bfloat16 dlogits chunk with rows padded to a multiple of 8 columns."""
    f = dart.load_library().dart_lmhead_backward_workspace_bytes
    assert f(0, 10) == 0 and f(10, 0) == 0 and f(1 << 31, 5) == 0
    assert f(2, 300) == 2 * 304 * 2 and f(3, 8) == 3 * 8 * 2
    assert f(1024, 152064) == 1024 * 152064 * 2


@pytest.mark.skipif("_gpu_visible()")
def test_lmhead_leading_dimension_limit():
    """Leading dimensions beyond 2^22 elements do not fit the tile's 32-bit
    row offsets: UNSUPPORTED before anything is launched."""
    lib = dart.load_library()
    big = (1 << 22) + 8
    assert lib.dart_lmhead_tok_stats(*_lm_args(ld_h=big)) == dart.DART_ERR_UNSUPPORTED
    assert lib.dart_lmhead_tok_stats(*_lm_args(ld_w=big)) == dart.DART_ERR_UNSUPPORTED
    assert lib.dart_lmhead_dlogits(*_lm_grad_args(ld_w=big)) == dart.DART_ERR_UNSUPPORTED


def _lm_bwd_ex_args(flags=0, chunk_cols=300, inv_temp=1.0, **kw):
    a = _lm_bwd_args(**kw)[:-1]
    return a[:11] + [inv_temp] + a[11:16] + [chunk_cols, flags] + a[16:] + [None]


@pytest.mark.skipif("_gpu_visible()")
@pytest.mark.parametrize("kw", [
    dict(hidden=0), dict(weight=0), dict(target=0), dict(lse=0), dict(logp=0), dict(coef=0),
    dict(dh=0), dict(dw=0), dict(workspace=0), dict(T=0), dict(V=0), dict(d=4, ld_h=4, ld_w=4),
    dict(ld_dh=15), dict(ld_dw=8), dict(chunk=0), dict(ws_bytes=2 * 304 * 2 - 1),
    dict(workspace=(1 << 22) + 8), dict(flags=2), dict(flags=8), dict(flags=1 << 31),
    dict(chunk_cols=0), dict(flags=1, ws_bytes="one short"), dict(flags=1, ws_bytes=2 * 304 * 2),
    dict(flags=4, chunk_cols=100, ws_bytes="one short"),
])
def test_lmhead_backward_ex_rejects(kw):
    """Bad arguments, unknown flags and a workspace too small for the row
    compaction are INVALID_ARG before anything is enqueued."""
    lib = dart.load_library()
    if kw.get("ws_bytes") == "one short":
        kw["ws_bytes"] = dart.dart_lmhead_backward_ex_workspace_bytes(
            4, 16, 300, 2, kw.get("chunk_cols", 300), kw["flags"]) - 1
    assert lib.dart_lmhead_backward_ex(*_lm_bwd_ex_args(**kw)) == dart.DART_ERR_INVALID_ARG


def test_lmhead_backward_ex_workspace_bytes():
    """The parts of the workspace, each starting at a multiple of 256 bytes: the
    bf16 dlogits block; with bf16 gradients, an fp32 accumulator for each
    output that several blocks add to (dweight when the rows come in several
    blocks, dhidden when the vocabulary does, but not with rows skipped); with
    rows skipped, the compact hidden rows (bf16), their fp32 dhidden, five [T]
    int/float arrays and a counter. chunk_cols >= V with flags = 0 needs what
    dart_lmhead_backward needs."""
    f = dart.dart_lmhead_backward_ex_workspace_bytes
    plain = dart.dart_lmhead_backward_workspace_bytes
    up = lambda x: -(-x // 256) * 256
    c8 = lambda x: -(-x // 8) * 8
    SKIP, BF = dart.DART_LMHEAD_SKIP_ZERO_ROWS, dart.DART_LMHEAD_BF16_GRADS
    for T, d, V, cr, cc in ((4, 16, 300, 2, 300), (4, 16, 300, 9, 100), (4096, 3584, 152064, 4096, 65536),
                            (5, 8, 7, 1, 1), (300, 136, 2100, 512, 700), (300, 136, 2100, 100, 5000),
                            (152569, 3584, 152064, 15360, 17408)):
        for flags in (0, SKIP, BF, SKIP | BF):
            bf16, skip = bool(flags & BF), bool(flags & SKIP)
            R, C = min(cr, T), min(cc, V)
            parts = [R * c8(C) * 2]
            if bf16 and R < T:
                parts.append(V * d * 4)
            if bf16 and C < V and not skip:
                parts.append(T * d * 4)
            if skip:
                parts += [T * d * 2, T * d * 4] + [T * 4] * 5 + [4]
            want = sum(up(x) for x in parts[:-1]) + parts[-1]
            assert f(T, d, V, cr, cc, flags) == want, (T, d, V, cr, cc, flags)
            if flags == 0 and C == V:
                assert want == plain(R, V)
    assert f(0, 16, 300, 2, 5, 1) == 0 and f(4, 0, 300, 2, 5, 1) == 0 and f(4, 16, 0, 2, 5, 1) == 0
    assert f(4, 16, 300, 0, 5, 1) == 0 and f(4, 16, 300, 2, 0, 1) == 0
    assert f(4, 16, 300, 2, 5, 2) == 0 and f(4, 16, 300, 2, 5, 8) == 0
    assert f(1 << 31, 16, 8, 1, 1, 0) == 0


def test_lmhead_backward_plan():
    """All rows with vocabulary chunks when T << V, near-square blocks when
    T ~ V; whole 256-wide tiles within the byte budget, and the cost (summed
    outputs rewritten) no larger than that of any other such block."""
    plan = dart.lmhead_backward_plan
    assert plan(4096, 152064) == (4096, 65536)
    assert plan(500, 1000) == (500, 1000) and plan(100, 50) == (100, 50)
    for T, V in ((152569, 152064), (34585, 152064), (16384, 151936), (4096, 152064)):
        r, c = plan(T, V)
        assert (r == T or r % 256 == 0) and (c == V or c % 256 == 0)
        assert r * c * 2 <= 512 << 20
        cost = -(-T // r) * V + -(-V // c) * T
        for r2 in range(256, T + 1, 256):
            c2 = min(V, (((512 << 20) // 2) // r2) // 256 * 256)
            if c2 >= 256:
                assert cost <= -(-T // r2) * V + -(-V // c2) * T
    r, c = plan(152569, 152064)
    assert 8192 <= r <= 32768 and 8192 <= c <= 32768


def test_stream_must_be_on_the_inputs_device():
    """A torch stream of another device is refused before any call (kernels
    would run on that device against these pointers); a raw handle is taken as
    given."""
    import torch

    class FakeStream:
        def __init__(self, device, handle):
            self.device, self.cuda_stream = torch.device(device), handle

    assert dart._stream_handle(FakeStream("cuda:0", 1234), torch.device("cuda:0")) == 1234
    with pytest.raises(ValueError):
        dart._stream_handle(FakeStream("cuda:1", 1234), torch.device("cuda:0"))
    assert dart._stream_handle(5678, torch.device("cuda:0")) == 5678


@pytest.mark.skipif("_gpu_visible()")
def test_launch_limits_are_unsupported():
    """Sizes whose launch would exceed 2^32 - 1 work-items are UNSUPPORTED,
    decided on the host before anything is touched (fake pointers here)."""
    lib = dart.load_library()
    U = dart.DART_ERR_UNSUPPORTED
    big = (1 << 31) - 1
    # step selection: one wave per step, 1024-thread workgroups
    assert lib.dart_step_select(P, big, P, 67108864, ctypes.c_double(0.5), P, P, P, None) == U
    # per-group selection: one 1024-thread workgroup per group
    assert lib.dart_step_select_groups(P, big, P, 1 << 23, P, 4194304, ctypes.c_double(0.5), P, P,
                                       P, None) == U
    # GRPO advantage: one 256-thread workgroup per group
    assert lib.dart_grpo_advantage(P, 1 << 25, P, P, 16777216, P, 1 << 25, big, P, P, P, None) == U
    # LM head: 8,388,608 tiles of 256 x 256
    assert lib.dart_lmhead_tok_stats(P, big, 8, 8, P, 8, 8, P, P, P, P, P, (1 << 64) - 1,
                                     None) == U


def test_autograd_lmhead_plan():
    """The LM-head autograd backward: the default plan with bf16 gradients, or
    the caller's block and flags with bf16 gradients added; a block needs both
    sizes."""
    from paper_2509_23866_amd.autograd import lmhead_grad_plan

    bf = dart.DART_LMHEAD_BF16_GRADS
    assert lmhead_grad_plan(4096, 152064) == (4096, 65536, bf)
    assert lmhead_grad_plan(300, 5000, 256, 1000, dart.DART_LMHEAD_SKIP_ZERO_ROWS) == \
        (256, 1000, bf | dart.DART_LMHEAD_SKIP_ZERO_ROWS)
    assert lmhead_grad_plan(300, 5000, 256, 1000) == (256, 1000, bf)
    with pytest.raises(ValueError):
        lmhead_grad_plan(300, 5000, 256, None)


def test_hip_builds_disable_packed_fp32():
    """Every HIP compile of the package and of the generator's device twin
    targets gfx950 with the packed-FP32 VALU forms disabled (the kernels are
    plain scalar fp32 code)."""
    from paper_2509_23866_amd import _build
    import synth.native as sn

    want = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    for flags in (_build.HIPCC_FLAGS, sn.HIP_FLAGS):
        flags = list(flags)
        assert "--offload-arch=gfx950" in flags
        assert any(flags[i:i + 4] == want for i in range(len(flags) - 3)), flags
