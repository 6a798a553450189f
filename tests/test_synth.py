"""The seeded input generator: its three twins agree and the workloads have
the shapes and structure their descriptions state."""

import numpy as np
import pytest
import torch

import synth
import synth.native as sn
from synth import gen


def test_normal_table_properties():
    q = synth.normal_table()
    assert q.shape == (65536,)
    assert np.all(np.diff(q) > 0)
    assert np.allclose(q, -q[::-1], atol=1e-12)
    assert abs(q[0] + 4.3249) < 1e-4 and abs(q[-1] - 4.3249) < 1e-4
    assert abs(q.mean()) < 1e-12 and abs(q.std() - 1.0) < 2e-3


def test_splitmix64_known_values():
    """SplitMix64 with state 0: the first outputs of the reference sequence
    (state advanced by the golden gamma before mixing)."""
    h = gen._splitmix64(np.array([0], dtype=np.uint64))
    assert int(h[0]) == 0xE220A8397B1DCDAF


def test_uniform_strictly_inside():
    u = synth.draw_uniform(5, 3, np.arange(100000), 0)
    assert u.min() > 0 and u.max() < 1
    assert abs(u.mean() - 0.5) < 0.01


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.normal(0, 3, 100000) * rng.choice([1e-30, 1, 1e20], 100000)).astype(np.float32)
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_host_twin_matches_numpy(name):
    wl = synth.make_workload(name)
    rows = np.unique(np.r_[0, 1, wl.T - 1, np.linspace(0, wl.T - 1, 7).astype(np.int64)])
    a = synth.logits_rows_numpy(wl, rows)
    b = sn.logits_rows_host(wl, rows)
    assert a.dtype == b.dtype and np.array_equal(a, b)


def test_workload_shapes():
    w = synth.make_workload("tiny")
    assert (w.T, w.V, w.S, w.dtype) == (512, 4096, 16, "f32")
    assert np.all(np.diff(w.off) == 32) and (w.rho, w.eps_low, w.C) == (0.5, 0.2, 2.0)
    w = synth.make_workload("vlm7b")
    lens = np.diff(w.off)
    assert (w.T, w.V, w.S) == (4096, 152064, 64) and lens.min() >= 16 and lens.max() <= 128
    w = synth.make_workload("microbatch")
    lens = np.diff(w.off)
    assert w.S == 240 and lens.min() >= 32 and lens.max() <= 256 and 30000 < w.T < 40000
    adv_per_step = w.adv[w.off[:-1]]
    assert np.all(adv_per_step.reshape(8, 30) == adv_per_step.reshape(8, 30)[:, :1])
    w = synth.make_workload("longhorizon")
    lens = np.diff(w.off)
    assert w.S == 1600 and lens.min() >= 32 and lens.max() <= 160 and w.inplace
    assert (w.rho, w.eps_low, w.eps_high, w.C) == (0.5, 0.28, 0.28, 5.0)
    w = synth.make_workload("edge")
    assert (w.T, w.V, w.S, w.rho) == (16384, 151936, 256, 0.25)


def test_edge_structure():
    w = synth.make_workload("edge")
    kinds = np.bincount(w.kind, minlength=3)
    assert kinds.tolist() == [5632, 5376, 5376]
    # copy blocks: 4 steps of identical rows
    copy_rows = np.flatnonzero(w.src_row != np.arange(w.T))
    assert copy_rows.size > 0
    t = int(copy_rows[5])
    a = synth.logits_rows_numpy(w, [t, int(w.src_row[t])])
    assert np.array_equal(a[0], a[1]) and w.target[t] == w.target[w.src_row[t]]
    flat = int(np.flatnonzero(w.kind == gen.KIND_FLAT)[3])
    assert np.all(synth.logits_rows_numpy(w, [flat]) == 0)
    hot = int(np.flatnonzero(w.kind == gen.KIND_ONEHOT)[3])
    row = synth.bf16_bits_to_f32(synth.logits_rows_numpy(w, [hot])[0])
    assert np.count_nonzero(row) == 1 and row[w.spike_col[hot]] == 30.0
    hot_rows = w.kind == gen.KIND_ONEHOT
    frac_on_target = np.mean(w.spike_col[hot_rows] == w.target[hot_rows])
    assert 0.4 < frac_on_target < 0.6
    # ratio and rollout offsets span the stated ranges
    r = np.exp(-w.old_offset)
    assert r.min() > 0.5 and r.max() < 1.5 and r.min() < 0.52 and r.max() > 1.48
    d = -w.roll_offset
    assert d.min() > -3 and d.max() < 3 and np.mean(d >= np.log(2.0)) > 0.3


def test_perturbation_model_std():
    w = synth.make_workload("vlm7b")
    assert abs(w.old_offset.std() - 0.05) < 0.005 and abs(w.roll_offset.std() - 0.1) < 0.01
    lp_old, lp_roll = synth.perturbed_logprobs(w, np.full(w.T, -3.0))
    assert lp_old.dtype == np.float32 and lp_roll.dtype == np.float32
    assert np.allclose(lp_old, -3.0 + w.old_offset, atol=1e-6)


def test_gaussian_matrix_twins():
    """The LM-head inputs: numpy definition and the C twin agree bit for bit;
    rows generated from an offset equal the same rows of the whole matrix."""
    import synth.native as sn

    a = synth.gaussian_bits(7, synth.gen.STREAM_WEIGHT, 53, 40, 0.3)
    assert np.array_equal(a, sn.gaussian_bits_host(7, synth.gen.STREAM_WEIGHT, 53, 40, 0.3))
    assert np.array_equal(a[17:20], synth.gaussian_bits(7, synth.gen.STREAM_WEIGHT, 3, 40, 0.3, row0=17))
    vals = synth.bf16_bits_to_f32(synth.gaussian_bits(1, synth.gen.STREAM_HIDDEN, 200, 256, 1.0))
    assert abs(vals.std() - 1.0) < 0.02 and abs(vals.mean()) < 0.02
