"""GRPO group statistics and advantages (Eq. 1), written out in float64.

For a group of K rewards r_1..r_K (one prompt's K sampled responses),
mu = (sum r_i) / K, sigma = sqrt(sum (r_i - mu)^2 / (K - ddof)) and
A_i = (r_i - mu) / (sigma + eps_std). The paper calls sigma the standard
deviation of the K rewards and eps_std a small stabiliser without fixing
either; the readings taken: ddof = 1 (the unbiased estimate, the default of
common GRPO implementations) with ddof = 0 available, eps_std = 1e-6, and
sigma = 0 for a one-sample group under ddof = 1. Results are returned in
float64; ``advantage_f32`` rounds them to float32 (nearest even).
"""
import numpy as np

EPS_STD = 1e-6


def group_stats(rewards, *, ddof=1):
    """mean, std per group of a [R][K] reward array (float64)."""
    r = np.asarray(rewards, dtype=np.float64)
    K = r.shape[-1]
    mu = r.sum(axis=-1) / K
    dev = r - mu[..., None]
    den = K - ddof
    var = (dev * dev).sum(axis=-1) / den if den > 0 else np.zeros_like(mu)
    return mu, np.sqrt(var)


def advantage(rewards, *, eps_std=EPS_STD, ddof=1):
    r = np.asarray(rewards, dtype=np.float64)
    mu, sd = group_stats(r, ddof=ddof)
    return (r - mu[..., None]) / (sd[..., None] + eps_std)


def advantage_f32(rewards, *, eps_std=EPS_STD, ddof=1):
    mu, sd = group_stats(rewards, ddof=ddof)
    return (advantage(rewards, eps_std=eps_std, ddof=ddof).astype(np.float32), mu.astype(np.float32),
            sd.astype(np.float32))
