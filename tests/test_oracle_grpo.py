"""Pins for the oracle's GRPO group statistics and advantages, Eq. 1 (CPU only).

Checked against torch's mean/std (float64, unbiased and not), the closed form
for binary rewards (k successes out of K: A = +-sqrt((1-p)/p) or
-sqrt(p/(1-p)) with the population std), hand-worked two-sample groups,
and invariants: advantages sum to zero, have unit RMS (ddof 0) or sum of
squares K - 1 (ddof 1) when eps_std = 0, are unchanged by a shift or a
positive scaling of the rewards, flip sign with them, and are zero for a
group of equal rewards.
"""
import numpy as np
import pytest
import torch

from oracle import advantage, advantage_f32, group_stats


def _rewards(R=50, K=8, seed=0):
    return np.random.default_rng(seed).standard_normal((R, K)) * 3.0 + 1.0


@pytest.mark.parametrize("ddof", [0, 1])
def test_stats_match_torch(ddof):
    r = _rewards()
    mu, sd = group_stats(r, ddof=ddof)
    t = torch.from_numpy(r)
    np.testing.assert_allclose(mu, t.mean(dim=1).numpy(), rtol=1e-14)
    np.testing.assert_allclose(sd, t.std(dim=1, correction=ddof).numpy(), rtol=1e-13)
    ref = (t - t.mean(dim=1, keepdim=True)) / (t.std(dim=1, correction=ddof, keepdim=True) + 1e-6)
    np.testing.assert_allclose(advantage(r, ddof=ddof), ref.numpy(), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("k,K", [(1, 8), (3, 8), (7, 8), (2, 4), (5, 16)])
def test_binary_rewards_closed_form(k, K):
    r = np.zeros((1, K))
    r[0, :k] = 1.0
    p = k / K
    a = advantage(r, eps_std=0.0, ddof=0)[0]
    np.testing.assert_allclose(a[:k], np.sqrt((1 - p) / p), rtol=1e-14)
    np.testing.assert_allclose(a[k:], -np.sqrt(p / (1 - p)), rtol=1e-14)


def test_two_sample_group_by_hand():
    r = np.array([[0.0, 1.0]])
    np.testing.assert_allclose(advantage(r, eps_std=0.0, ddof=0)[0], [-1.0, 1.0], rtol=1e-15)
    np.testing.assert_allclose(advantage(r, eps_std=0.0, ddof=1)[0], [-np.sqrt(0.5), np.sqrt(0.5)], rtol=1e-15)
    np.testing.assert_allclose(advantage(r, eps_std=0.5, ddof=0)[0], [-0.5, 0.5], rtol=1e-15)


@pytest.mark.parametrize("ddof", [0, 1])
def test_invariants(ddof):
    r = _rewards(seed=2)
    a = advantage(r, eps_std=0.0, ddof=ddof)
    np.testing.assert_allclose(a.sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose((a * a).sum(axis=1), 8 - ddof, rtol=1e-12)
    np.testing.assert_allclose(advantage(r + 123.0, eps_std=0.0, ddof=ddof), a, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(advantage(r * 7.5, eps_std=0.0, ddof=ddof), a, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(advantage(-r, eps_std=0.0, ddof=ddof), -a, rtol=1e-14, atol=1e-15)


def test_equal_rewards_and_single_sample_groups_give_zero():
    assert np.all(advantage(np.full((3, 8), 0.7)) == 0.0)
    assert np.all(advantage(np.array([[5.0], [-2.0]]), ddof=1) == 0.0)
    assert np.all(advantage(np.array([[5.0], [-2.0]]), ddof=0) == 0.0)


def test_f32_outputs_are_the_rounded_f64_values():
    r = _rewards(seed=3).astype(np.float32)
    a32, mu32, sd32 = advantage_f32(r)
    assert a32.dtype == np.float32
    assert np.array_equal(a32, advantage(r).astype(np.float32))
    mu, sd = group_stats(r)
    assert np.array_equal(mu32, mu.astype(np.float32)) and np.array_equal(sd32, sd.astype(np.float32))
