"""Decode attention over a paged, group-shared KV cache, straight from the definition.

For sequence ``s`` in group ``g = seq_to_group[s]`` the keys are the group's
prompt-prefix tokens ``t < prefix_lens[g]`` (page ``prefix_block_table[g][t // ps]``,
row ``t % ps``) followed by the sequence's own response tokens ``t < resp_lens[s]``
(page ``resp_block_table[s][t // ps]``, row ``t % ps``). Every response of a GRPO
group is sampled from the same prompt (paper, Section 2.1), which is why the
prefix is stored once per group.

Query head ``j`` reads kv-head ``j // (Hq / Hkv)`` (consecutive query heads share
a kv-head). With ``sigma`` the caller's fp32 scale widened to fp64:

    s_t = sigma * sum_i q_i k_{t,i}
    lse = log(sum_t exp(s_t))            (natural log; computed as m + log sum exp(s_t - m))
    out = sum_t exp(s_t - lse) v_t

An empty key set gives ``out = 0`` and ``lse = -inf``.
"""
import numpy as np

from .formats import bf16_to_f64, e4m3_to_f64


def key_slots(seq_to_group, prefix_lens, prefix_block_table, resp_lens, resp_block_table,
              s, page_size):
    """(physical page, row) of every key of sequence ``s``: prefix first, then response."""
    g = int(seq_to_group[s])
    P = int(prefix_lens[g])
    L = int(resp_lens[s])
    tp = np.arange(P)
    tr = np.arange(L)
    pages = np.concatenate([np.asarray(prefix_block_table[g])[tp // page_size],
                            np.asarray(resp_block_table[s])[tr // page_size]]).astype(np.int64)
    rows = np.concatenate([tp % page_size, tr % page_size]).astype(np.int64)
    return pages, rows


def _gather(pages_arr, scales, kv_dtype, pages, rows, h):
    """Decoded fp64 [N][d] rows of kv-head ``h`` at the given (page, row) slots."""
    raw = pages_arr[pages, h, rows, :]
    if kv_dtype == "fp8":
        return e4m3_to_f64(raw) * scales[pages, h].astype(np.float64)[:, None]
    return bf16_to_f64(raw)


def decode_attention(*, k_pages, v_pages, k_scale, v_scale, kv_dtype, page_size,
                     seq_to_group, prefix_lens, prefix_block_table, resp_lens,
                     resp_block_table, q, softmax_scale, seqs=None):
    """fp64 ``(out [n][Hq][d], lse [n][Hq])`` for the sequences in ``seqs`` (default: all)."""
    q = np.asarray(q)
    S, Hq, d = q.shape
    Hkv = k_pages.shape[1]
    n_rep = Hq // Hkv
    sigma = np.float64(np.float32(softmax_scale))
    seqs = range(S) if seqs is None else seqs
    seqs = list(seqs)
    out = np.zeros((len(seqs), Hq, d), dtype=np.float64)
    lse = np.full((len(seqs), Hq), -np.inf, dtype=np.float64)
    for i, s in enumerate(seqs):
        pages, rows = key_slots(seq_to_group, prefix_lens, prefix_block_table,
                                resp_lens, resp_block_table, s, page_size)
        if pages.size == 0:
            continue
        qs = bf16_to_f64(q[s])                                   # [Hq][d]
        for h in range(Hkv):
            K = _gather(k_pages, k_scale, kv_dtype, pages, rows, h)   # [N][d]
            V = _gather(v_pages, v_scale, kv_dtype, pages, rows, h)
            for j in range(h * n_rep, (h + 1) * n_rep):
                sc = sigma * (K @ qs[j])                         # [N]
                m = sc.max()
                lse_j = m + np.log(np.exp(sc - m).sum())
                out[i, j] = np.exp(sc - lse_j) @ V
                lse[i, j] = lse_j
    return out, lse


def attention_for_workload(wl, seqs=None, pool=None):
    """Oracle result for a generated workload.

    When the workload includes an append, ``pool`` must be the post-append pool
    ``(k_pages, v_pages, k_scale, v_scale)`` from ``oracle.kv_append``; attention
    then reads ``resp_lens + 1`` response keys.
    """
    if pool is None:
        if wl.append:
            raise ValueError("workload appends a token: pass the post-append pool")
        pool = (wl.k_pages, wl.v_pages, wl.k_scale, wl.v_scale)
    kp, vp, ks, vs = pool
    return decode_attention(k_pages=kp, v_pages=vp, k_scale=ks, v_scale=vs,
                            kv_dtype=wl.kv_dtype, page_size=wl.page_size,
                            seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                            prefix_block_table=wl.prefix_block_table,
                            resp_lens=wl.attn_resp_lens, resp_block_table=wl.resp_block_table,
                            q=wl.q, softmax_scale=wl.softmax_scale, seqs=seqs)
