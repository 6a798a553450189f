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
