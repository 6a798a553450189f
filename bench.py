#!/usr/bin/env python3
"""Benchmark of the DART policy-update hot path on one MI355X (gfx950).

One step = one pass of the whole path over one step group held in HBM:
dart_tok_stats -> dart_select_tis_loss_fwd (step means, selection, coefficients
and loss; one launch up to 4096 tokens) -> dart_tis_grad, on one stream. The K timed steps run back to back; per-kernel durations come from
a second pass of K steps with HIP events around each kernel. The default workload is the 7B-VLM vocabulary group: T = 4096
action tokens in 64 steps, V = 152064, bf16 logits, separate gradient buffer.

Prints one JSON line. `value` is logit elements per second (T*V per step
time); `hbm_frac_step` counts 2 reads + 1 write of the T x V logits per step
against 8 TB/s; `roofline` covers the dominant kernel (the gradient pass, one
read + one write of T x V), timed with HIP events on its own stream;
`cpu_baseline` times the float64 oracle on the host cores.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "logit elements/s for fused entropy+TIS loss fwd+bwd; % of HBM peak"
HBM_PEAK_GBS = 8000.0
DOMINANT = "tis_grad_kernel"


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # a cold GPU runs its first ~25 steps up to 15% slower while its clocks
    # ramp (per-step HIP events at vlm7b: 0.67 ms, then ~0.61, then ~0.585);
    # 30 untimed steps (~20 ms) reach the steady state a training run sees
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="vlm7b",
                    choices=["tiny", "vlm7b", "microbatch", "longhorizon", "edge"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="0 = the CPU share of one GPU (16 cores) or the process's affinity if smaller")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the separately reported variants and the copy ceiling "
                         "(profiling runs of the headline step)")
    ap.add_argument("--headline-only", action="store_true",
                    help="measure only --workload, not the other workloads first "
                         "(profiling runs of the headline step)")
    ap.add_argument("--skip-rows-step", action="store_true",
                    help="the step's gradient pass skips reading rows with a zero coefficient "
                         "(profiling runs of the read-skipping gradient; not the headline)")
    ap.add_argument("--no-lmhead", action="store_true",
                    help="leave the fused LM-head variant out")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the timed steps, run one plain device copy of this many MiB "
                         "(torch copy kernel) so that hardware counters can be scaled by it")
    return ap.parse_args()


def kernel_source_hash():
    src = os.path.join(ROOT, "paper_2509_23866_amd", "csrc", "dart.hip")
    with open(src, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


CPU_SAMPLE_MAX_ROWS = 8192
# host cores one GPU's share of the machine provides: the oracle baseline runs
# that many OpenMP threads (fewer if the process's affinity is smaller)
CPU_SHARE = 16


def _steps_prefix(wl, max_rows):
    """The workload cut to its first whole steps holding at most max_rows
    tokens (at least one step): the same rows, targets and per-token inputs."""
    import dataclasses

    import numpy as np

    off = np.asarray(wl.off, dtype=np.int64)
    n = max(1, int(np.searchsorted(off, max_rows, side="right")) - 1)
    Ts = int(off[n])
    cut = {k: getattr(wl, k)[:Ts] for k in ("kind", "src_row", "spike_col", "spike_val", "target",
                                            "adv", "old_offset", "roll_offset")}
    if wl.ref_offset is not None:
        cut["ref_offset"] = wl.ref_offset[:Ts]
    return dataclasses.replace(wl, T=Ts, off=wl.off[:n + 1].copy(), **cut), n


def cpu_baseline(wl, threads, min_seconds=1.5, max_passes=20):
    """The float64 oracle, as it stands: token stats, step entropy, selection,
    loss and the gradient (rows streamed in chunks, gradient rows discarded),
    over the whole workload when it has at most CPU_SAMPLE_MAX_ROWS tokens, else
    over its first whole steps within that many tokens (their own selection).
    Passes repeat until min_seconds have passed; the rate is that of the median
    pass. Input generation and the old-policy log-probs (an untimed oracle pass)
    are outside the timed region."""
    import numpy as np

    import oracle
    import synth
    import synth.native as sn

    sub, nsteps = (wl, wl.S) if wl.T <= CPU_SAMPLE_MAX_ROWS else _steps_prefix(
        wl, CPU_SAMPLE_MAX_ROWS)
    z = sn.logits_rows_host(sub, np.arange(sub.T), nthreads=threads)
    logp0, _, _ = oracle.token_stats(z, sub.target, nthreads=threads)
    lp_old, lp_roll = synth.perturbed_logprobs(sub, logp0)
    f = lambda x: float(np.float32(x))  # noqa: E731

    def one_pass():
        t0 = time.perf_counter()
        logp, H, lse = oracle.token_stats(z, sub.target, nthreads=threads)
        _, Hs32 = oracle.step_entropy(H, sub.off)
        mask, _ = oracle.step_mask(Hs32, sub.rho)
        res = oracle.tis_loss(logp, lp_old, lp_roll, sub.adv, sub.off, mask, f(sub.eps_low),
                              f(sub.eps_high), f(sub.C))
        chunk = 256
        for r0 in range(0, sub.T, chunk):
            r1 = min(sub.T, r0 + chunk)
            oracle.dlogits(z[r0:r1], sub.target[r0:r1], lse[r0:r1], logp[r0:r1],
                           res["g"][r0:r1], nthreads=threads)
        return time.perf_counter() - t0

    times = []
    while len(times) < max_passes and (not times or sum(times) < min_seconds):
        times.append(one_pass())
    dt = float(np.median(times))
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")),
                         None)
    except OSError:
        pass
    what = (f"whole workload ({sub.T} rows x {sub.V})" if sub is wl else
            f"first {nsteps} of {wl.S} steps ({sub.T} of {wl.T} rows x {sub.V})")
    return {"value": sub.T * sub.V / dt, "unit": "logit elements/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 3), "passes": len(times),
            "cpu_seconds": round(sum(times) * threads, 1), "cpu_model": model,
            "sample": f"{what}, float64 C oracle, OpenMP over rows; median of {len(times)} passes"}


def graph_variant(step, stream, dev, n, warm=30):
    """The same step captured once into a HIP graph and replayed n times back to
    back (one pair of events around the replays): the launch gaps a trainer
    that replays a captured step would see. Never the headline."""
    import torch

    side = torch.cuda.Stream(device=dev)
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        step(s=side)
    torch.cuda.synchronize(dev)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        step(s=side)
    torch.cuda.synchronize(dev)
    for _ in range(max(1, warm)):  # untimed replays: the same warm-up as the eager step
        g.replay()
    torch.cuda.synchronize(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(n):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize(dev)
    return {"ms_per_step": e0.elapsed_time(e1) / n, "replays": n}


def lmhead_variant(wl, dev, stream, target, coef, n):
    """The LM head fused in (never the headline): statistics and gradients of
    the logits h W^T formed on the matrix cores, at this workload's T and V and
    the 7B VLM's hidden size, with the headline step's own loss coefficients;
    beside it the library GEMM that materialises the same logits. Above 16384
    tokens the calls that need a whole [T, V] buffer (dlogits written whole,
    the one-block backward, the library GEMM) are left out and every backward
    runs in blocks within 512 MiB. Per-launch HIP events on the bench stream;
    medians of n launches after one warm-up."""
    import numpy as np
    import torch

    import paper_2509_23866_amd as dart
    import synth
    import synth.native as sn
    from synth.gen import STREAM_HIDDEN, STREAM_WEIGHT

    prob = synth.lmhead_problem(wl.name)
    T, V, d = wl.T, wl.V, prob.d
    whole = T <= 16384
    bf = torch.bfloat16
    h = torch.empty((T, d), dtype=bf, device=dev)
    w = torch.empty((V, d), dtype=bf, device=dev)
    sn.fill_gaussian_device(h, wl.seed, STREAM_HIDDEN, prob.sigma_h)
    sn.fill_gaussian_device(w, wl.seed, STREAM_WEIGHT, prob.sigma_w)
    logp, ent, lse = (torch.empty(T, dtype=torch.float32, device=dev) for _ in range(3))
    ws = torch.empty(dart.dart_lmhead_stats_workspace_bytes(T, V), dtype=torch.uint8, device=dev)
    dh = torch.empty((T, d), dtype=torch.float32, device=dev)
    dw = torch.empty((V, d), dtype=torch.float32, device=dev)

    def timed(f):
        f()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n)]
        for a, b in ev:
            a.record(stream)
            f()
            b.record(stream)
        torch.cuda.synchronize(dev)
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    flop = 2.0 * T * V * d
    peak = 2500.0  # dense bf16 MFMA, TFLOP/s

    def tf(ms, k=1):
        return k * flop / (ms * 1e-3) / 1e12

    stats_ms = timed(lambda: dart.dart_lmhead_tok_stats(h, w, target, logp, ent, lse, workspace=ws,
                                                        stream=stream))
    del ws
    out = {"shape": {"T": T, "d": d, "V": V}, "flop_per_gemm": flop, "peak_TFLOPs": peak,
           "stats_kernels_ms": stats_ms, "stats_TFLOPs": tf(stats_ms),
           "stats_mfma_frac": tf(stats_ms) / peak,
           "logits_bytes_not_materialised": T * V * 2}
    if whole:
        zbuf = torch.empty((T, V), dtype=bf, device=dev)
        wsb = torch.empty(dart.dart_lmhead_backward_workspace_bytes(T, V), dtype=torch.uint8,
                          device=dev)
        dl_ms = timed(lambda: dart.dart_lmhead_dlogits(h, w, target, lse, logp, coef,
                                                       dlogits=zbuf, stream=stream))
        bwd_ms = timed(lambda: dart.dart_lmhead_backward(h, w, target, lse, logp, coef,
                                                         chunk_rows=T, dhidden=dh, dweight=dw,
                                                         workspace=wsb, stream=stream))
        del wsb
        out.update({"dlogits_ms": dl_ms, "dlogits_TFLOPs": tf(dl_ms),
                    "dlogits_mfma_frac": tf(dl_ms) / peak, "backward_ms": bwd_ms,
                    "backward_chunk_rows": T, "backward_TFLOPs": tf(bwd_ms, 3)})

    kept = int(torch.count_nonzero(coef).item())

    def blocked(rows, cols, flags):
        gdt = torch.bfloat16 if flags & dart.DART_LMHEAD_BF16_GRADS else torch.float32
        dhx = torch.empty((T, d), dtype=gdt, device=dev)
        dwx = torch.empty((V, d), dtype=gdt, device=dev)
        wsx = torch.empty(dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, flags),
                          dtype=torch.uint8, device=dev)
        ms = timed(lambda: dart.dart_lmhead_backward_ex(h, w, target, lse, logp, coef,
                                                        chunk_rows=rows, chunk_cols=cols,
                                                        flags=flags, dhidden=dhx, dweight=dwx,
                                                        workspace=wsx, stream=stream))
        # three GEMM-equivalents over the rows the call forms
        formed = kept / T if flags & dart.DART_LMHEAD_SKIP_ZERO_ROWS else 1.0
        return {"chunk_rows": min(rows, T), "chunk_cols": min(cols, V), "flags": flags,
                "workspace_bytes": wsx.numel(), "ms": ms, "TFLOPs": tf(ms, 3) * formed}

    skip = dart.DART_LMHEAD_SKIP_ZERO_ROWS
    pr, pc = dart.lmhead_backward_plan(T, V)
    sr, sc = (T, V) if whole else (pr, pc)
    out["backward_skip_zero_rows"] = blocked(sr, sc, skip)
    out["rows_with_gradient"] = kept
    # memory-bounded blockings within 512 MiB of dlogits: the plan, with fp32
    # and with bf16 gradients, and whole vocabulary rows in row chunks
    rows_only = max(256, ((512 << 20) // (2 * ((V + 7) // 8 * 8))) // 256 * 256)
    out["backward_chunked"] = {
        "plan_fp32": blocked(pr, pc, 0),
        "plan_bf16": blocked(pr, pc, dart.DART_LMHEAD_BF16_GRADS),
        "rows_only_fp32": blocked(rows_only, V, 0),
    }
    if whole:
        gemm_ms = timed(lambda: torch.matmul(h, w.t(), out=zbuf))
        tstats_ms = timed(lambda: dart.dart_tok_stats(zbuf, target, logp, ent, lse,
                                                      stream=stream))
        out.update({"library_gemm_logits_ms": gemm_ms, "library_gemm_TFLOPs": tf(gemm_ms),
                    "unfused_stats_ms": gemm_ms + tstats_ms})
        out["training_step"] = training_steps(wl, dev, stream, h, w, target, zbuf, timed)
    return out


def _median_ms(fn, stream, dev, n):
    """Median over n calls of fn(), each between its own pair of HIP events on
    the stream, after one untimed call."""
    import numpy as np
    import torch

    fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize(dev)
    return float(np.median([a.elapsed_time(b) for a, b in ev]))


def objective_variant(wl, dev, stream, logits, target, off, adv, lp_old, lp_roll, dlogits,
                      default_step, n):
    """The objective's variants on the same two passes (never the headline):
    one whole step with inverse temperature 1.25 in both passes, the KL term
    (k3 estimator, beta = 0.1) against the workload's reference log-probs,
    step-mean aggregation and step-level (geometric-mean) ratios, beside the
    default step; medians of n steps."""
    import torch

    import paper_2509_23866_amd as dart

    T, V, S = wl.T, wl.V, wl.S
    f = lambda k: torch.empty(k, dtype=torch.float32, device=dev)  # noqa: E731
    logp, ent, lse, coef, sh, st = f(T), f(T), f(T), f(T), f(S), f(6)
    mask = torch.empty(S, dtype=torch.uint8, device=dev)
    nk = torch.empty(1, dtype=torch.int32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    ws = torch.empty(dart.dart_tis_loss_workspace_bytes(T), dtype=torch.uint8, device=dev)
    inv_temp = 1.25
    dart.dart_tok_stats(logits, target, logp, ent, lse, stream=stream, inv_temp=inv_temp)
    torch.cuda.synchronize(dev)
    lp_ref = (logp.double() + torch.from_numpy(wl.ref_offset).to(dev)).float()

    def step():
        dart.dart_tok_stats(logits, target, logp, ent, lse, stream=stream, inv_temp=inv_temp)
        dart.dart_step_select(ent, off, wl.rho, sh, mask, nk, stream=stream)
        dart.dart_tis_loss_fwd_ex(logp, lp_old, lp_roll, adv, off, mask, wl.eps_low, wl.eps_high,
                                  wl.C, logp_ref=lp_ref, kl="k3", beta=0.1,
                                  aggregation="step_mean", ratio="step_geomean", loss=loss,
                                  tok_coef=coef, stats=st, stream=stream, workspace=ws)
        dart.dart_tis_grad(logits, target, logp, lse, coef, dlogits, stream=stream,
                           inv_temp=inv_temp)

    # the two steps alternate, so that both see the same clocks
    import numpy as np

    step()
    default_step()
    pairs = []
    for _ in range(n):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(stream)
        step()
        ev[1].record(stream)
        default_step()
        ev[2].record(stream)
        pairs.append(ev)
    torch.cuda.synchronize(dev)
    ms = float(np.median([e[0].elapsed_time(e[1]) for e in pairs]))
    base = float(np.median([e[1].elapsed_time(e[2]) for e in pairs]))
    return {"inv_temp": inv_temp, "kl": "k3", "beta": 0.1, "aggregation": "step_mean",
            "ratio": "step_geomean", "ms_per_step": ms, "default_ms_per_step": base,
            "logit_elements_per_s": T * V / (ms * 1e-3)}


def groups_variant(wl, dev, stream, ent, off, n):
    """The steps on either side of the path (never the headline): the
    step-wise GRPO advantage and the per-group selection, with the workload's
    steps cut into trajectories of at most 30 steps and task groups of 8
    trajectories (the paper's episode cap and rollouts per task) and a seeded
    0/1 reward per trajectory; medians of n calls, beside the one-group
    selection of the headline step."""
    import numpy as np
    import torch

    import paper_2509_23866_amd as dart

    S, T = wl.S, wl.T
    traj = np.r_[np.arange(0, S, 30), S].astype(np.int32)
    n_traj = traj.size - 1
    groups = np.r_[np.arange(0, n_traj, 8), n_traj].astype(np.int32)
    G = groups.size - 1
    reward = np.random.default_rng(wl.seed).integers(0, 2, n_traj).astype(np.float32)
    dv = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    reward_d, traj_d, groups_d, gsteps_d = dv(reward), dv(traj), dv(groups), dv(traj[groups])
    adv = torch.empty(T, dtype=torch.float32, device=dev)
    gm, gs = (torch.empty(G, dtype=torch.float32, device=dev) for _ in range(2))
    sh = torch.empty(S, dtype=torch.float32, device=dev)
    mask = torch.empty(S, dtype=torch.uint8, device=dev)
    nk = torch.empty(G, dtype=torch.int32, device=dev)
    nk1 = torch.empty(1, dtype=torch.int32, device=dev)
    grpo_ms = _median_ms(lambda: dart.dart_grpo_advantage(reward_d, traj_d, groups_d, off, T=T,
                                                          adv=adv, group_mean=gm, group_std=gs,
                                                          stream=stream), stream, dev, n)
    sel_ms = _median_ms(lambda: dart.dart_step_select_groups(ent, off, gsteps_d, wl.rho, sh, mask,
                                                             nk, stream=stream), stream, dev, n)
    one_ms = _median_ms(lambda: dart.dart_step_select(ent, off, wl.rho, sh, mask, nk1,
                                                      stream=stream), stream, dev, n)
    return {"trajectories": n_traj, "groups": G, "grpo_advantage_us": grpo_ms * 1e3,
            "step_select_groups_us": sel_ms * 1e3, "step_select_one_group_us": one_ms * 1e3}


def training_steps(wl, dev, stream, h, w, target, zbuf, timed):
    """One whole LM-head training step with bf16 gradients, two ways: fused
    (statistics, selection, loss and the blocked backward in its 512 MiB plan;
    the logits are formed twice and never stored), also with the rows whose
    coefficient is zero skipped in the backward, and through the library (the
    logits and the dlogits materialised in bf16: GEMM, statistics, selection,
    loss, gradient pass, two GEMMs), with the workload's steps, advantages and
    old-policy log-probs."""
    import torch

    import paper_2509_23866_amd as dart

    T, V, d = h.shape[0], w.shape[0], h.shape[1]
    dv = lambda a: torch.from_numpy(a).to(dev)  # noqa: E731
    off, adv = dv(wl.off.astype("int32")), dv(wl.adv)
    f = lambda n: torch.empty(n, dtype=torch.float32, device=dev)  # noqa: E731
    logp, ent, lse, coef, sh, st = f(T), f(T), f(T), f(T), f(wl.S), f(4)
    mask = torch.empty(wl.S, dtype=torch.uint8, device=dev)
    nk = torch.empty(1, dtype=torch.int32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    dart.dart_lmhead_tok_stats(h, w, target, logp, ent, lse, stream=stream)
    torch.cuda.synchronize(dev)
    lp_old = (logp.double() + dv(wl.old_offset)).float()
    lp_roll = (lp_old.double() + dv(wl.roll_offset)).float()
    lws = torch.empty(dart.dart_tis_loss_workspace_bytes(T), dtype=torch.uint8, device=dev)
    sws = torch.empty(dart.dart_lmhead_stats_workspace_bytes(T, V), dtype=torch.uint8, device=dev)
    rows, cols = dart.lmhead_backward_plan(T, V)
    bf = dart.DART_LMHEAD_BF16_GRADS
    bws = torch.empty(dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, bf),
                      dtype=torch.uint8, device=dev)
    dh = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((V, d), dtype=torch.bfloat16, device=dev)
    dzbuf = torch.empty_like(zbuf)

    def loss_part():
        dart.dart_select_tis_loss_fwd(ent, logp, lp_old, lp_roll, adv, off, wl.rho, wl.eps_low,
                                      wl.eps_high, wl.C, sh, mask, nk, loss, coef, st,
                                      workspace=lws, stream=stream)

    skip = bf | dart.DART_LMHEAD_SKIP_ZERO_ROWS
    kws = torch.empty(dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, skip),
                      dtype=torch.uint8, device=dev)

    def fused(flags=bf, ws=bws):
        dart.dart_lmhead_tok_stats(h, w, target, logp, ent, lse, workspace=sws, stream=stream)
        loss_part()
        dart.dart_lmhead_backward_ex(h, w, target, lse, logp, coef, chunk_rows=rows,
                                     chunk_cols=cols, flags=flags, dhidden=dh, dweight=dw,
                                     workspace=ws, stream=stream)

    def library():
        with torch.cuda.stream(stream):
            torch.matmul(h, w.t(), out=zbuf)
            dart.dart_tok_stats(zbuf, target, logp, ent, lse, stream=stream)
            loss_part()
            dart.dart_tis_grad(zbuf, target, logp, lse, coef, dzbuf, stream=stream)
            torch.matmul(dzbuf, w, out=dh)
            torch.matmul(dzbuf.t(), h, out=dw)

    fused_ms, library_ms = timed(fused), timed(library)
    skip_ms = timed(lambda: fused(skip, kws))
    return {"fused_ms": fused_ms, "fused_workspace_bytes": sws.numel() + bws.numel(),
            "fused_skip_zero_rows_ms": skip_ms,
            "fused_skip_zero_rows_workspace_bytes": sws.numel() + kws.numel(),
            "library_ms": library_ms, "library_logits_bytes": 2 * zbuf.numel() * 2,
            "block": [rows, cols]}


# the other workloads, measured before the headline; edge last, whose kernels
# have the headline's row lengths (~1% faster headline than with the in-place
# long-horizon group last, alternating A/B on MI355X)
SWEEP_ORDER = ("tiny", "longhorizon", "microbatch", "edge")


def measured_profile(kernel, workload, variant=""):
    """The committed PMC record of a kernel at a workload (``variant``: e.g.
    "skip" for the read-skipping gradient), if it was taken on the current
    kernel source (else None)."""
    name = f"{kernel}_{workload}{'_' + variant if variant else ''}_traffic.json"
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return rec


def measure_workload(wl, args, dev, headline):
    """One workload: inputs generated in HBM, W untimed steps, K timed steps
    back to back, K more steps with events around each kernel, the
    read-skipping gradient and the statistics pass alone, and a plain
    elementwise copy of the same bytes. With ``headline`` also the variants
    that are reported only for the headline workload. Returns a dict of
    results; every buffer is freed on return."""
    import numpy as np
    import torch

    import paper_2509_23866_amd as dart
    import synth.native as sn

    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    esize = 4 if wl.dtype == "f32" else 2
    T, V, S = wl.T, wl.V, wl.S

    # ---- inputs resident in HBM (untimed set-up)
    logits = torch.empty((T, V), dtype=tdt, device=dev)
    sn.fill_logits_device(sn.DeviceRecipe(wl), logits)
    pristine = logits.clone() if wl.inplace else None
    target = torch.from_numpy(wl.target).to(dev)
    adv = torch.from_numpy(wl.adv).to(dev)
    off = torch.from_numpy(wl.off).to(dev)
    logp, ent, lse = dart.dart_tok_stats(logits, target)
    # old/rollout log-probs: the workload's perturbation of the current policy's
    # log-prob of each target (the same pass a trainer runs for pi_old)
    base = logp.double()
    lp_old = (base + torch.from_numpy(wl.old_offset).to(dev)).float()
    lp_roll = (lp_old.double() + torch.from_numpy(wl.roll_offset).to(dev)).float()
    step_H = torch.empty(S, dtype=torch.float32, device=dev)
    mask = torch.empty(S, dtype=torch.uint8, device=dev)
    n_kept = torch.empty(1, dtype=torch.int32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    coef = torch.empty(T, dtype=torch.float32, device=dev)
    stats = torch.empty(4, dtype=torch.float32, device=dev)
    workspace = torch.empty(dart.dart_tis_loss_workspace_bytes(T), dtype=torch.uint8, device=dev)
    dlogits = logits if wl.inplace else torch.empty((T, V), dtype=tdt, device=dev)
    eps_low, eps_high, C = float(np.float32(wl.eps_low)), float(np.float32(wl.eps_high)), float(np.float32(wl.C))
    stream = torch.cuda.current_stream(dev)

    def step(ev=None, s=stream):
        if ev:
            ev[0].record(s)
        dart.dart_tok_stats(logits, target, logp, ent, lse, stream=s)
        if ev:
            ev[1].record(s)
        dart.dart_select_tis_loss_fwd(ent, logp, lp_old, lp_roll, adv, off, wl.rho, eps_low,
                                      eps_high, C, step_H, mask, n_kept, loss, coef, stats,
                                      stream=s, workspace=workspace)
        if ev:
            ev[2].record(s)
        dart.dart_tis_grad(logits, target, logp, lse, coef, dlogits, stream=s,
                           skip_zero_rows=args.skip_rows_step)
        if ev:
            ev[3].record(s)

    if headline and args.calib_copy_mib:
        # a plain elementwise kernel that reads and writes exactly this many
        # bytes (a same-dtype copy_ would go to the DMA engine, not a kernel)
        n = args.calib_copy_mib * (1 << 20) // 2
        src = torch.ones(n, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize(dev)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize(dev)
        del src, dst

    for _ in range(args.warmup):
        if pristine is not None:
            logits.copy_(pristine)
        step()
    torch.cuda.synchronize(dev)

    # ---- timed region: K steps back to back on one stream, nothing recorded
    # between their kernels. An in-place workload restores its logits before
    # each step, outside a per-step event pair; otherwise one pair of events
    # brackets the K steps (the longer of it and the wall clock counts).
    ev_new = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    torch.cuda.synchronize(dev)
    if pristine is None:
        e0, e1 = ev_new(), ev_new()
        t0 = time.perf_counter()
        e0.record(stream)
        for i in range(args.steps):
            step()
        e1.record(stream)
        t_enq = time.perf_counter() - t0
        torch.cuda.synchronize(dev)
        wall = time.perf_counter() - t0
        ev_ms = e0.elapsed_time(e1)
        ms_per_step = max(ev_ms, wall * 1e3) / args.steps
        timing = {"events_ms_per_step": ev_ms / args.steps, "wall_ms_per_step": wall * 1e3 / args.steps,
                  "host_enqueue_ms_per_step": t_enq * 1e3 / args.steps}
    else:
        es = [(ev_new(), ev_new()) for _ in range(args.steps)]
        for i in range(args.steps):
            logits.copy_(pristine)  # untimed: outside the step's events
            es[i][0].record(stream)
            step()
            es[i][1].record(stream)
        torch.cuda.synchronize(dev)
        ms_per_step = float(np.mean([a.elapsed_time(b) for a, b in es]))
        timing = {"events_ms_per_step": ms_per_step}

    # ---- kernel durations: K more steps with HIP events around each kernel
    # on the launch stream (the events add idle gaps between kernels, which is
    # why the timed region above has none)
    evs = [[ev_new() for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        if pristine is not None:
            logits.copy_(pristine)
        step(evs[i])
    torch.cuda.synchronize(dev)

    # separately reported variants (never the headline value): the gradient
    # pass with zero-coefficient rows written without reading them, and the
    # statistics pass alone (the forward-only recompute of pi_old's log-probs)
    variants = {}
    if not args.no_variants:
        zero_rows = float((coef == 0).float().mean().item())
        skip_out = torch.empty_like(logits) if wl.inplace else dlogits
        ev_v = [[ev_new() for _ in range(2)] for _ in range(args.steps)]
        for i in range(args.steps):
            ev_v[i][0].record(stream)
            dart.dart_tis_grad(pristine if wl.inplace else logits, target, logp, lse, coef,
                               skip_out, stream=stream, skip_zero_rows=True)
            ev_v[i][1].record(stream)
        torch.cuda.synchronize(dev)
        del skip_out
        skip_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev_v]))
        model_bytes = (2.0 - zero_rows) * T * V * esize
        rec = measured_profile(DOMINANT, wl.name, "skip")
        meas = rec.get("hbm_bytes_per_launch") if rec else None
        variants["grad_skip_zero_rows"] = {
            "zero_row_fraction": zero_rows, "grad_ms": skip_ms,
            "model_bytes_per_launch": model_bytes,
            "hbm_bytes_per_launch_measured": meas,
            "measured_over_model": (meas / model_bytes) if meas else None,
            "achieved_GBps": (meas if meas else model_bytes) / (skip_ms * 1e-3) / 1e9,
            "bytes_source": (f"rocprofv3 --pmc FETCH_SIZE, WRITE_SIZE: {rec['summary']}" if rec
                             else "model (2 - f) T V b; no counter record on this source")}
        ev_s = [[ev_new() for _ in range(2)] for _ in range(args.steps)]
        for i in range(args.steps):
            ev_s[i][0].record(stream)
            dart.dart_tok_stats(pristine if wl.inplace else logits, target, logp, ent, lse,
                                stream=stream)
            ev_s[i][1].record(stream)
        torch.cuda.synchronize(dev)
        stats_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev_s]))
        variants["stats_only"] = {"ms": stats_ms, "logit_elements_per_s": T * V / (stats_ms * 1e-3),
                                  "achieved_GBps": T * V * esize / (stats_ms * 1e-3) / 1e9}

    if headline and not wl.inplace and not args.no_variants:
        variants["hip_graph"] = graph_variant(step, stream, dev, args.steps, args.warmup)
        variants["objective_variants"] = objective_variant(
            wl, dev, stream, logits, target, off, adv, lp_old, lp_roll, dlogits, step,
            min(args.steps, 20))
    if headline and not args.no_variants:
        variants["groups"] = groups_variant(wl, dev, stream, ent, off, min(args.steps, 20))
    if headline and not args.no_variants and not args.no_lmhead:
        variants["lmhead_fused"] = lmhead_variant(wl, dev, stream, target, coef,
                                                  min(args.steps, 10))

    # empirical ceiling beside the 8 TB/s peak: a plain torch elementwise kernel
    # reading and writing the same T x V bytes as the gradient pass
    copy_ceiling = None
    if not args.no_variants:
        src_c = pristine if wl.inplace else logits
        copy_ev = [(ev_new(), ev_new()) for _ in range(min(args.steps, 10))]
        torch.mul(src_c, 1.0, out=dlogits)  # first launch loads the kernel's code
        for a, b in copy_ev:
            a.record(stream)
            torch.mul(src_c, 1.0, out=dlogits)
            b.record(stream)
        torch.cuda.synchronize(dev)
        copy_ms = float(np.median([a.elapsed_time(b) for a, b in copy_ev]))
        copy_gbs = 2 * T * V * esize / (copy_ms * 1e-3) / 1e9
        copy_ceiling = {"kernel": "torch elementwise multiply by 1 (T x V read + write)",
                        "ms": copy_ms, "GBps": copy_gbs, "frac": copy_gbs / HBM_PEAK_GBS}

    k1_ms = [e[0].elapsed_time(e[1]) for e in evs]
    mid_ms = [e[1].elapsed_time(e[2]) for e in evs]
    grad_ms = [e[2].elapsed_time(e[3]) for e in evs]
    elems = T * V
    grad_bytes = 2 * elems * esize
    achieved = grad_bytes / (float(np.mean(grad_ms)) * 1e-3) / 1e9
    rec = measured_profile(DOMINANT, wl.name)
    zero_frac = float((coef == 0).float().mean().item())
    out = {
        "wl": wl, "T": T, "V": V, "S": S, "dtype": wl.dtype, "in_place": wl.inplace,
        "logits_bytes": elems * esize, "ms_per_step": ms_per_step,
        "zero_row_fraction": zero_frac,
        "value": elems / (ms_per_step * 1e-3),
        "hbm_frac_step": (3 * elems * esize / (ms_per_step * 1e-3) / 1e9) / HBM_PEAK_GBS,
        "kernel_ms": {"tok_stats_kernel": float(np.mean(k1_ms)),
                      "tis_grad_kernel": float(np.mean(grad_ms)),
                      "step_select+tis_loss_fwd": float(np.mean(mid_ms))},
        "tok_stats_GBps": elems * esize / (float(np.mean(k1_ms)) * 1e-3) / 1e9,
        "roofline": {"kernel": DOMINANT, "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": rec.get("hbm_bytes_per_launch") if rec else None,
                     "algorithmic_bytes_per_launch": grad_bytes},
        "variants": variants, "copy_ceiling": copy_ceiling, "timing": timing,
    }
    del logits, pristine, dlogits
    torch.cuda.synchronize(dev)
    torch.cuda.empty_cache()
    return out


def workload_summary(r, cpu):
    """The per-workload record of the JSON line's ``workloads`` object."""
    v = r["variants"]
    return {
        "T": r["T"], "V": r["V"], "S": r["S"], "dtype": r["dtype"], "in_place": r["in_place"],
        "ms_per_step": r["ms_per_step"], "logit_elements_per_s": r["value"],
        "hbm_frac_step": r["hbm_frac_step"], "kernel_ms": r["kernel_ms"],
        "tis_grad_GBps": r["roofline"]["achieved"], "tis_grad_frac": r["roofline"]["frac"],
        "tis_grad_traffic": r["roofline"]["traffic"], "tok_stats_GBps": r["tok_stats_GBps"],
        "grad_skip_zero_rows": v.get("grad_skip_zero_rows"),
        "stats_only_GBps": (v.get("stats_only") or {}).get("achieved_GBps"),
        "copy_ceiling_GBps": (r["copy_ceiling"] or {}).get("GBps"),
        "timing": r["timing"], "cpu_baseline": cpu,
    }


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path; "
              "run with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    affinity = len(os.sched_getaffinity(0))
    threads = args.cpu_threads or min(CPU_SHARE, affinity)

    # every other workload first (in the same process; each one's buffers are
    # freed before the next), then the headline workload; the oracle baselines
    # run on the host after all of them, so that the GPU work follows the
    # sweep without the host-only pauses in between (~1.5-2 s each, during
    # which the GPU's clocks fall, and 5 warm-up steps do not bring them back)
    sweep = {}
    if not args.headline_only:
        for name in SWEEP_ORDER:
            if name == args.workload:
                continue
            wl = synth.make_workload(name)
            print(f"[bench] workload {name}: T={wl.T} V={wl.V}", file=sys.stderr, flush=True)
            sweep[name] = (wl, measure_workload(wl, args, dev, headline=False))

    wl = synth.make_workload(args.workload)
    print(f"[bench] headline {wl.name}: T={wl.T} V={wl.V}", file=sys.stderr, flush=True)
    r = measure_workload(wl, args, dev, headline=True)
    sweep_lines = {}
    for name, (swl, sr) in sweep.items():
        scpu = None if args.no_cpu_baseline else cpu_baseline(swl, threads)
        sweep_lines[name] = workload_summary(sr, scpu)
    cpu = None if args.no_cpu_baseline else cpu_baseline(wl, threads)
    if cpu is not None:
        cpu["affinity_cores"] = affinity
    workloads = {**sweep_lines, wl.name: workload_summary(r, cpu)}
    workloads = {k: workloads[k] for k in ("tiny", "vlm7b", "microbatch", "longhorizon", "edge")
                 if k in workloads}

    line = {
        "metric": METRIC,
        "value": r["value"],
        "unit": "logit elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded counter-based generator; shapes of the workload description)",
        "config": {"workload": f"{wl.name}: {wl.description}", "T": wl.T, "V": wl.V, "S": wl.S,
                   "rho": wl.rho, "eps_low": wl.eps_low, "eps_high": wl.eps_high, "C": wl.C,
                   "in_place": wl.inplace, "logits_bytes": r["logits_bytes"],
                   "grad_skip_zero_rows_step": bool(args.skip_rows_step)},
        "hbm_frac_step": r["hbm_frac_step"],
        "zero_row_fraction": r["zero_row_fraction"],
        "kernel_ms": r["kernel_ms"],
        "roofline": r["roofline"],
        "variants": r["variants"],
        "copy_ceiling": r["copy_ceiling"],
        "timing": r["timing"],
        "workloads": workloads,
        "workloads_order": ([k for k in SWEEP_ORDER if k in sweep] + [wl.name]),
    }
    if cpu is not None:
        line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
