"""Seeded raw attention projections for the pre-attention side of a decode step.

For ``S`` sequences this draws the new token's q, k and v projections before
normalisation (bf16 bit patterns as uint16: q ``[S][Hq][d]``, k and v
``[S][Hkv][d]``) and the learned per-channel norm weights of q and k (bf16
``[d]``, shared by every head of the layer).

Projections are ``N(0, 1)`` times a per-(head, channel) magnitude drawn once
from a log-normal (sigma 0.5), so a few channels dominate as in trained
projection outputs; the norm weights are ``exp(0.3 N(0, 1))``. Draw order from
``default_rng(seed)``: q magnitudes, k magnitudes, v magnitudes, q, k, v, q
weights, k weights. Nothing here normalises or rotates.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .gen import _to_bf16_bits


@dataclass
class QkPrepInputs:
    q_in: np.ndarray      # [S][Hq][d] uint16
    k_in: np.ndarray      # [S][Hkv][d] uint16
    v_in: np.ndarray      # [S][Hkv][d] uint16
    q_norm_w: np.ndarray  # [d] uint16
    k_norm_w: np.ndarray  # [d] uint16


def make_qkprep_inputs(*, num_seqs: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                       seed: int, scale: float = 1.0) -> QkPrepInputs:
    rng = np.random.default_rng(seed)
    S, d = num_seqs, head_dim
    mags = [rng.lognormal(0.0, 0.5, size=(h, d)).astype(np.float32) * np.float32(scale)
            for h in (num_q_heads, num_kv_heads, num_kv_heads)]
    raw = [rng.standard_normal((S, h, d), dtype=np.float32) * m[None]
           for h, m in zip((num_q_heads, num_kv_heads, num_kv_heads), mags)]
    wq = np.exp(0.3 * rng.standard_normal(d)).astype(np.float32)
    wk = np.exp(0.3 * rng.standard_normal(d)).astype(np.float32)
    return QkPrepInputs(q_in=_to_bf16_bits(raw[0]), k_in=_to_bf16_bits(raw[1]), v_in=_to_bf16_bits(raw[2]),
                        q_norm_w=_to_bf16_bits(wq), k_norm_w=_to_bf16_bits(wk))
