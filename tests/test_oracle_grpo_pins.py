"""Pins of the step-wise GRPO advantage (Sec. 3.3) and of the per-group step
selection (Sec. 4.3 applied to each task's step group)."""

import math

import numpy as np
import pytest

import oracle


def _layout(traj_steps, group_trajs, step_len=1):
    """CSR offsets: steps per trajectory, trajectories per group, tokens per step."""
    traj_off = np.r_[0, np.cumsum(traj_steps)].astype(np.int32)
    grp_off = np.r_[0, np.cumsum(group_trajs)].astype(np.int32)
    S = int(traj_off[-1])
    lens = np.full(S, step_len) if np.isscalar(step_len) else np.asarray(step_len)
    off = np.r_[0, np.cumsum(lens)].astype(np.int32)
    return traj_off, grp_off, off


def test_two_equal_trajectories_give_plus_minus_one():
    traj_off, grp_off, off = _layout([3, 3], [2])
    adv, mean, std = oracle.grpo_advantage([1.0, 0.0], traj_off, grp_off, off)
    assert np.allclose(adv, [1, 1, 1, -1, -1, -1], atol=1e-15)
    assert mean[0] == 0.5 and std[0] == 0.5


def test_steps_weight_the_group_statistics():
    """Each step is one element of D: a 3-step success and a 1-step failure
    give Rbar = 3/4, sigma = sqrt(3/16), A = +1/sqrt(3) and -sqrt(3)."""
    traj_off, grp_off, off = _layout([3, 1], [2], step_len=[2, 1, 4, 5])
    adv, mean, std = oracle.grpo_advantage([1.0, 0.0], traj_off, grp_off, off)
    assert abs(mean[0] - 0.75) < 1e-15 and abs(std[0] - math.sqrt(3) / 4) < 1e-15
    assert np.allclose(adv[:7], 1 / math.sqrt(3), rtol=1e-14)
    assert np.allclose(adv[7:], -math.sqrt(3), rtol=1e-14)


@pytest.mark.parametrize("seed", range(4))
def test_zero_mean_unit_variance_over_steps_and_affine_invariance(seed):
    """Over the steps of each group the advantages have mean 0 and population
    variance 1, and they do not change under R -> a R + b (a > 0)."""
    rng = np.random.default_rng(seed)
    groups = rng.integers(2, 9, 3)
    traj_steps = rng.integers(1, 30, int(groups.sum()))
    lens = rng.integers(1, 6, int(traj_steps.sum()))
    traj_off, grp_off, off = _layout(traj_steps, groups, step_len=lens)
    R = rng.random(int(groups.sum())).astype(np.float32)
    adv, _, _ = oracle.grpo_advantage(R, traj_off, grp_off, off)
    step_adv = adv[off[:-1]]
    for g in range(len(groups)):
        a, b = traj_off[grp_off[g]], traj_off[grp_off[g + 1]]
        assert abs(step_adv[a:b].mean()) < 1e-12
        assert abs((step_adv[a:b] ** 2).mean() - 1) < 1e-12
    adv2, _, _ = oracle.grpo_advantage((R * np.float32(4) + np.float32(-2)).astype(np.float32),
                                       traj_off, grp_off, off)
    assert np.allclose(adv, adv2, atol=1e-6)  # float32 rewards: 4R - 2 rounds


def test_constant_rewards_give_zero_advantage():
    traj_off, grp_off, off = _layout([2, 5, 1], [3])
    adv, mean, std = oracle.grpo_advantage([0.7, 0.7, 0.7], traj_off, grp_off, off)
    assert np.all(adv == 0.0) and std[0] == 0.0


def test_groups_are_independent():
    traj_off, grp_off, off = _layout([2, 2, 1, 3], [2, 2])
    a, _, _ = oracle.grpo_advantage([1, 0, 0.25, 0.75], traj_off, grp_off, off)
    t1, g1, o1 = _layout([1, 3], [2])
    b, _, _ = oracle.grpo_advantage([0.25, 0.75], t1, g1, o1)
    assert np.allclose(a[4:], b, atol=1e-15)


def test_step_mask_groups_is_per_group_top_k():
    """Each group keeps ceil(rho S_g) of its own steps, by its own ranking."""
    Hs = np.array([5, 1, 3, 2, 9, 9, 0.5, 4, 4, 4], np.float32)
    gso = np.array([0, 4, 7, 10], np.int32)
    mask, ks = oracle.step_mask_groups(Hs, gso, 0.5)
    assert ks.tolist() == [2, 2, 2]
    assert mask.tolist() == [1, 0, 1, 0, 1, 1, 0, 1, 1, 0]
