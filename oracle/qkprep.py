"""Pre-attention side of one decode step of a Qwen3-style attention layer, from the definitions.

The paper's policy is Qwen3-1.7B (Section 5.1); its attention layer normalises
every query and key head with an RMS norm before the rotary position embedding
and only then appends k and v to the cache. The paper gives none of the
constants; the readings taken are those of the public model: RMS epsilon
1e-6, rotary base 1,000,000, rotation of element pairs (i, i + d/2).

For sequence ``s`` in group ``g`` the new token's position is
``prefix_lens[g] + resp_lens[s]`` (the tokens already in its cache). For one
head vector ``x`` of length ``d`` with learned weights ``w``:

    rms_norm(x) = x / sqrt(mean(x^2) + eps) * w
    rope(y, pos)[i]       = y[i] cos(a_i) - y[i + d/2] sin(a_i)
    rope(y, pos)[i + d/2] = y[i + d/2] cos(a_i) + y[i] sin(a_i),   a_i = pos * base^(-2i/d)

for i < d/2, all in float64; q and k outputs are rounded to bf16 (nearest,
ties to even). v is appended unchanged.
"""
import numpy as np

from .append import kv_append
from .formats import bf16_to_f64, f64_to_bf16_bits

RMS_EPS = 1e-6
ROPE_BASE = 1_000_000.0


def rms_norm(x, w, eps=RMS_EPS):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(w, dtype=np.float64)


def rope(y, pos, base=ROPE_BASE):
    """Rotate the pairs (i, i + d/2) of y [..., d] by pos * base^(-2i/d); pos broadcasts over y[..., 0]."""
    y = np.asarray(y, dtype=np.float64)
    d = y.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    c, s = np.cos(ang), np.sin(ang)
    y1, y2 = y[..., :half], y[..., half:]
    return np.concatenate([y1 * c - y2 * s, y2 * c + y1 * s], axis=-1)


def decode_positions(seq_to_group, prefix_lens, resp_lens):
    return np.asarray(prefix_lens, dtype=np.int64)[np.asarray(seq_to_group)] + np.asarray(resp_lens, dtype=np.int64)


def qk_prep(*, q_in, k_in, q_norm_w, k_norm_w, positions, eps=RMS_EPS, base=ROPE_BASE):
    """bf16 bits of the normalised and rotated q [S][Hq][d] and k [S][Hkv][d], and their fp64 values."""
    pos = np.asarray(positions, dtype=np.float64)[:, None]          # one position per sequence, all heads
    q = rope(rms_norm(bf16_to_f64(q_in), bf16_to_f64(q_norm_w), eps), pos, base)
    k = rope(rms_norm(bf16_to_f64(k_in), bf16_to_f64(k_norm_w), eps), pos, base)
    return f64_to_bf16_bits(q), f64_to_bf16_bits(k), q, k


def decode_step_prep(*, q_in, k_in, v_in, q_norm_w, k_norm_w, k_pages, v_pages, k_scale, v_scale, kv_dtype,
                     page_size, seq_to_group, prefix_lens, resp_lens, resp_block_table, eps=RMS_EPS,
                     base=ROPE_BASE):
    """q bits, k bits, and the pool after appending (k, v) at slot resp_lens[s] of every sequence."""
    pos = decode_positions(seq_to_group, prefix_lens, resp_lens)
    q_bits, k_bits, _, _ = qk_prep(q_in=q_in, k_in=k_in, q_norm_w=q_norm_w, k_norm_w=k_norm_w, positions=pos,
                                   eps=eps, base=base)
    pool = kv_append(k_pages=k_pages, v_pages=v_pages, k_scale=k_scale, v_scale=v_scale, kv_dtype=kv_dtype,
                     page_size=page_size, resp_lens=resp_lens, resp_block_table=resp_block_table,
                     k_new=k_bits, v_new=np.asarray(v_in))
    return q_bits, k_bits, pool
