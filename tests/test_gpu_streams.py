"""The header's claim that concurrent calls on different streams are safe:
two step groups run the whole path interleaved on two streams (default
priority), and each gives bit-identical results to its own run alone."""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _problem(seed, T, V, S):
    import torch

    rng = np.random.default_rng(seed)
    c = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    logits = torch.from_numpy(rng.normal(0, 3, (T, V)).astype(np.float32)).cuda().to(torch.bfloat16)
    target = c(rng.integers(0, V, T).astype(np.int32))
    off = c(np.r_[0, np.sort(rng.choice(np.arange(1, T), S - 1, replace=False)), T].astype(np.int32))
    base = rng.normal(-3, 1, T).astype(np.float32)
    lp_old = c(base)
    lp_roll = c(base + rng.normal(0, 0.1, T).astype(np.float32))
    adv = c(rng.normal(0, 1, T).astype(np.float32))
    return logits, target, lp_old, lp_roll, adv, off


def _run(p, stream):
    import paper_2509_23866_amd as dart

    out = dart.policy_update(*p, 0.8, 0.2, 0.28, 2.0, stream=stream)
    return [out[k] for k in ("logp", "entropy", "lse", "step_mask", "loss", "tok_coef", "dlogits")]


def test_two_streams_interleaved():
    import torch

    pa = _problem(1, 5000, 8192, 40)   # many-workgroup loss
    pb = _problem(2, 3000, 20001, 25)  # one-workgroup loss, ragged rows
    ra = [x.clone() for x in _run(pa, None)]
    rb = [x.clone() for x in _run(pb, None)]
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(3):
        with torch.cuda.stream(sa):
            oa = _run(pa, sa)
        with torch.cuda.stream(sb):
            ob = _run(pb, sb)
        outs.append((oa, ob))
    torch.cuda.synchronize()
    for oa, ob in outs:
        for x, y in zip(oa, ra):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
        for x, y in zip(ob, rb):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


def _lm_problem(seed, T, d, V):
    import torch

    rng = np.random.default_rng(seed)
    c = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    h = c(rng.normal(0, 1, (T, d)).astype(np.float32)).to(torch.bfloat16)
    w = c(rng.normal(0, 3.0 / np.sqrt(d), (V, d)).astype(np.float32)).to(torch.bfloat16)
    y = c(rng.integers(0, V, T).astype(np.int32))
    coef = c(np.where(rng.random(T) < 0.2, 0.0, rng.uniform(-1e-2, 1e-2, T)).astype(np.float32))
    return h, w, y, coef


def _lm_run(p, stream, rows, cols, flags):
    import paper_2509_23866_amd as dart

    h, w, y, coef = p
    logp, ent, lse = dart.dart_lmhead_tok_stats(h, w, y, stream=stream)
    dh, dw = dart.dart_lmhead_backward_ex(h, w, y, lse, logp, coef, chunk_rows=rows,
                                          chunk_cols=cols, flags=flags, stream=stream)
    return [logp, ent, lse, dh, dw]


def test_lmhead_two_streams_interleaved():
    """The LM-head statistics and blocked backward (its GEMMs included) of two
    problems interleaved on two streams, each bit-identical to its own run
    alone: the library keeps no state between calls, so nothing is shared. One
    problem has few rows against a long vocabulary (a small GEMM output over a
    long sum)."""
    import torch

    pa = _lm_problem(3, 64, 256, 20000)
    pb = _lm_problem(4, 300, 512, 16384)
    ka = dict(rows=64, cols=4096, flags=0)
    kb = dict(rows=128, cols=5000, flags=4)  # bf16 gradients, fp32 accumulators in the workspace
    ra = [x.clone() for x in _lm_run(pa, None, **ka)]
    rb = [x.clone() for x in _lm_run(pb, None, **kb)]
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(3):
        with torch.cuda.stream(sa):
            oa = _lm_run(pa, sa, **ka)
        with torch.cuda.stream(sb):
            ob = _lm_run(pb, sb, **kb)
        outs.append((oa, ob))
    torch.cuda.synchronize()
    for oa, ob in outs:
        for x, y in zip(oa, ra):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
        for x, y in zip(ob, rb):
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
