"""Shared-prefix prefill, straight from the definitions: each GRPO group's prompt
is attended once and its K/V pages are written once.

Every response of a GRPO group is sampled from the same prompt (paper,
Section 2.1; the rollout engine serves the K responses of a prompt, Section 4),
so the prompt is processed once per group rather than once per response; its
K/V go into the group's prefix pages, which every response then reads while
decoding.

Tokens of all groups are packed: group ``g`` owns rows
``prefix_offs[g] .. prefix_offs[g+1]-1`` of ``q [T][Hq][d]`` and of
``k, v [T][Hkv][d]`` (bf16 bit patterns as uint16).

Causal attention, token ``t`` of group ``g`` and query head ``j`` (kv-head
``h = j // (Hq / Hkv)``), with ``sigma`` the caller's fp32 scale widened:

    s_u = sigma * <q_t[j], k_u[h]>            for tokens u <= t of the same group
    lse = ln sum_u exp(s_u),  out = sum_u exp(s_u - lse) v_u[h]

KV write: token ``t`` of group ``g`` goes to page ``prefix_block_table[g][t // ps]``,
row ``t % ps``. bf16 pools copy the bit patterns. fp8 (OCP e4m3fn) pools give each
(page, kv-head) of the prompt, in fp32, ``scale = amax / 448`` over the page's
written rows (1.0 when ``amax == 0``), and store ``encode(x / scale)`` (round to
nearest even, saturate at 448) in those rows. Rows past the prompt are untouched.
"""
import numpy as np

from .formats import bf16_to_f32, bf16_to_f64, e4m3_encode

_F448 = np.float32(448.0)


def prefill_attention(q, k, v, prefix_offs, softmax_scale):
    """fp64 ``(out [T][Hq][d], lse [T][Hq])`` of causal attention within each group."""
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    n_rep = Hq // Hkv
    sigma = np.float64(np.float32(softmax_scale))
    offs = np.asarray(prefix_offs, dtype=np.int64)
    out = np.zeros((T, Hq, d), dtype=np.float64)
    lse = np.full((T, Hq), -np.inf, dtype=np.float64)
    for g in range(len(offs) - 1):
        a, b = int(offs[g]), int(offs[g + 1])
        n = b - a
        if n <= 0:
            continue
        future = np.triu(np.ones((n, n), dtype=bool), k=1)      # key u > query t
        for j in range(Hq):
            h = j // n_rep
            Q = bf16_to_f64(q[a:b, j, :])
            K = bf16_to_f64(k[a:b, h, :])
            V = bf16_to_f64(v[a:b, h, :])
            s = sigma * (Q @ K.T)
            s[future] = -np.inf
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            z = e.sum(axis=1, keepdims=True)
            lse[a:b, j] = (m + np.log(z))[:, 0]
            out[a:b, j, :] = (e / z) @ V
    return out, lse


def prefill_kv_write(*, k_pages, v_pages, k_scale, v_scale, kv_dtype, page_size,
                     prefix_block_table, prefix_offs, k, v):
    """Copies of the pools (and fp8 scales) with every group's prompt K/V written."""
    kp, vp = np.array(k_pages, copy=True), np.array(v_pages, copy=True)
    ks = None if k_scale is None else np.array(k_scale, dtype=np.float32, copy=True)
    vs = None if v_scale is None else np.array(v_scale, dtype=np.float32, copy=True)
    offs = np.asarray(prefix_offs, dtype=np.int64)
    k, v = np.asarray(k), np.asarray(v)
    Hkv = kp.shape[1]
    for g in range(len(offs) - 1):
        a, b = int(offs[g]), int(offs[g + 1])
        for p0 in range(0, b - a, page_size):
            rows = min(page_size, b - a - p0)
            page = int(prefix_block_table[g][p0 // page_size])
            for pool, scales, src in ((kp, ks, k), (vp, vs, v)):
                for h in range(Hkv):
                    x = src[a + p0:a + p0 + rows, h, :]
                    if kv_dtype == "fp8":
                        xf = bf16_to_f32(x)
                        amax = np.float32(np.abs(xf).max())
                        scale = np.float32(amax / _F448) if amax > 0 else np.float32(1.0)
                        pool[page, h, :rows, :] = e4m3_encode(xf / scale)
                        scales[page, h] = scale
                    else:
                        pool[page, h, :rows, :] = x
    return kp, vp, ks, vs
