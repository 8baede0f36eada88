"""Pins for the oracle's shared-prefix prefill (CPU only).

Causal attention is checked against torch's scaled_dot_product_attention with
is_causal (float64, CPU), against the independently pinned decode oracle (the
last prompt token attends exactly the prefix that decoding later reads),
closed forms (token 0, q = 0) and invariants (causality, group independence).
The page write is checked bytewise (bf16), against the append oracle's
first-row rule (fp8, one-row prompts), and against the quantisation bounds.
"""
import numpy as np
import pytest
import torch

from oracle import decode_attention, e4m3_to_f64, kv_append, prefill_attention, prefill_kv_write
from oracle.formats import bf16_to_f64
from workloads import make_prefill_workload


def _wl(P=(5, 17, 0, 33), Hq=4, Hkv=2, d=64, seed=3, kv_dtype="bf16"):
    return make_prefill_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, prefix_lens=list(P),
                                 seed=seed, kv_dtype=kv_dtype)


def _attn(w, q=None, k=None, v=None):
    return prefill_attention(w.q if q is None else q, w.k if k is None else k, w.v if v is None else v,
                             w.prefix_offs, w.softmax_scale)


CASES = [((5, 17, 0, 33), 4, 2, 64), ((40,), 8, 2, 64), ((16, 1, 31), 16, 8, 128), ((9, 12), 4, 4, 32),
         ((20,), 8, 1, 64)]


@pytest.mark.parametrize("P,Hq,Hkv,d", CASES)
def test_matches_torch_causal_sdpa_fp64(P, Hq, Hkv, d):
    w = _wl(P, Hq, Hkv, d, seed=sum(P) + d)
    out, lse = _attn(w)
    n_rep = Hq // Hkv
    sigma = float(np.float32(w.softmax_scale))
    for g in range(len(P)):
        a, b = w.prefix_offs[g], w.prefix_offs[g + 1]
        if b == a:
            continue
        q = torch.from_numpy(bf16_to_f64(w.q[a:b])).permute(1, 0, 2)                   # [Hq][n][d]
        k = torch.from_numpy(bf16_to_f64(w.k[a:b])).permute(1, 0, 2).repeat_interleave(n_rep, 0)
        v = torch.from_numpy(bf16_to_f64(w.v[a:b])).permute(1, 0, 2).repeat_interleave(n_rep, 0)
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True, scale=sigma)
        s = (q @ k.transpose(1, 2)) * sigma
        s = s.masked_fill(torch.triu(torch.ones(b - a, b - a, dtype=torch.bool), 1), float("-inf"))
        np.testing.assert_allclose(out[a:b], o.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[a:b], torch.logsumexp(s, -1).permute(1, 0).numpy(), rtol=0, atol=1e-12)


def test_last_prompt_token_equals_decode_over_the_written_prefix():
    # Decoding the last prompt token over the written prefix pages, with no
    # response, is the prefill's last row: ties the two oracles together.
    w = _wl((5, 17, 33), Hq=8, Hkv=2, d=64, seed=11)
    out, lse = _attn(w)
    kp, vp, _, _ = prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=None, v_scale=None,
                                    kv_dtype="bf16", page_size=16, prefix_block_table=w.prefix_block_table,
                                    prefix_offs=w.prefix_offs, k=w.k, v=w.v)
    G = w.num_groups
    last = w.prefix_offs[1:] - 1
    o2, l2 = decode_attention(k_pages=kp, v_pages=vp, k_scale=None, v_scale=None, kv_dtype="bf16", page_size=16,
                              seq_to_group=np.arange(G), prefix_lens=w.prefix_lens,
                              prefix_block_table=w.prefix_block_table, resp_lens=np.zeros(G, np.int32),
                              resp_block_table=np.zeros((G, 1), np.int32), q=w.q[last],
                              softmax_scale=w.softmax_scale)
    np.testing.assert_allclose(out[last], o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse[last], l2, rtol=0, atol=1e-12)


def test_first_token_returns_its_own_value_and_score():
    w = _wl()
    out, lse = _attn(w)
    n_rep = w.num_q_heads // w.num_kv_heads
    sigma = np.float64(np.float32(w.softmax_scale))
    for g in range(w.num_groups):
        a, b = w.prefix_offs[g], w.prefix_offs[g + 1]
        if b == a:
            continue
        for j in range(w.num_q_heads):
            h = j // n_rep
            np.testing.assert_array_equal(out[a, j], bf16_to_f64(w.v[a, h]))
            s = sigma * float(bf16_to_f64(w.q[a, j]) @ bf16_to_f64(w.k[a, h]))
            assert abs(lse[a, j] - s) < 1e-12


def test_zero_query_gives_log_count_and_running_mean():
    w = _wl()
    out, lse = _attn(w, q=np.zeros_like(w.q))
    n_rep = w.num_q_heads // w.num_kv_heads
    for g in range(w.num_groups):
        a, b = w.prefix_offs[g], w.prefix_offs[g + 1]
        for t in range(b - a):
            np.testing.assert_allclose(lse[a + t], np.log(t + 1), rtol=0, atol=1e-13)
            for j in range(w.num_q_heads):
                mean = bf16_to_f64(w.v[a:a + t + 1, j // n_rep]).mean(axis=0)
                np.testing.assert_allclose(out[a + t, j], mean, rtol=0, atol=1e-13)


def test_future_tokens_do_not_change_earlier_outputs():
    w = _wl((33,), seed=5)
    out, lse = _attn(w)
    k2, v2 = w.k.copy(), w.v.copy()
    rng = np.random.default_rng(0)
    k2[20:] = rng.integers(0, 0x3F00, size=k2[20:].shape, dtype=np.uint16)
    v2[20:] = rng.integers(0, 0x3F00, size=v2[20:].shape, dtype=np.uint16)
    o2, l2 = _attn(w, k=k2, v=v2)
    np.testing.assert_array_equal(out[:20], o2[:20])
    np.testing.assert_array_equal(lse[:20], l2[:20])
    assert not np.allclose(out[20:], o2[20:])


def test_groups_are_independent():
    w = _wl((12, 19), seed=9)
    out, _ = _attn(w)
    k2 = w.k.copy()
    k2[12:] ^= np.uint16(0x0100)          # perturb only group 1
    o2, _ = _attn(w, k=k2)
    np.testing.assert_array_equal(out[:12], o2[:12])
    assert not np.allclose(out[12:], o2[12:])


def test_bf16_write_copies_rows_and_leaves_the_rest():
    w = _wl((5, 17, 0, 33))
    kp, vp, _, _ = prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=None, v_scale=None,
                                    kv_dtype="bf16", page_size=16, prefix_block_table=w.prefix_block_table,
                                    prefix_offs=w.prefix_offs, k=w.k, v=w.v)
    written = np.zeros(kp.shape[:1] + kp.shape[2:3], dtype=bool)   # [page][row]
    for g in range(w.num_groups):
        a = w.prefix_offs[g]
        for t in range(w.prefix_lens[g]):
            page, row = w.prefix_block_table[g][t // 16], t % 16
            np.testing.assert_array_equal(kp[page, :, row], w.k[a + t])
            np.testing.assert_array_equal(vp[page, :, row], w.v[a + t])
            written[page, row] = True
    assert np.all(kp[~written[:, None, :].repeat(kp.shape[1], 1)] == w.k_pages[0, 0, 0, 0])


def test_fp8_one_row_prompt_matches_the_append_rule_for_a_first_row():
    # A one-token prompt writes row 0 of a fresh page: the append oracle's rule
    # for a first row (scale = amax / 448) must give the same bytes.
    w = _wl((1, 1, 1), Hq=4, Hkv=2, d=64, seed=21, kv_dtype="fp8")
    kp, vp, ks, vs = prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale, v_scale=w.v_scale,
                                      kv_dtype="fp8", page_size=16, prefix_block_table=w.prefix_block_table,
                                      prefix_offs=w.prefix_offs, k=w.k, v=w.v)
    G = w.num_groups
    ka, va, ksa, vsa = kv_append(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale, v_scale=w.v_scale,
                                 kv_dtype="fp8", page_size=16, resp_lens=np.zeros(G, np.int32),
                                 resp_block_table=w.prefix_block_table[:, :1], k_new=w.k, v_new=w.v)
    np.testing.assert_array_equal(kp, ka)
    np.testing.assert_array_equal(vp, va)
    np.testing.assert_array_equal(ks, ksa)
    np.testing.assert_array_equal(vs, vsa)


def test_fp8_write_scale_and_rounding_bounds():
    w = _wl((40, 16, 3), Hq=4, Hkv=2, d=64, seed=8, kv_dtype="fp8")
    kp, vp, ks, vs = prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale, v_scale=w.v_scale,
                                      kv_dtype="fp8", page_size=16, prefix_block_table=w.prefix_block_table,
                                      prefix_offs=w.prefix_offs, k=w.k, v=w.v)
    for g in range(w.num_groups):
        a, P = w.prefix_offs[g], w.prefix_lens[g]
        for p0 in range(0, P, 16):
            page, rows = w.prefix_block_table[g][p0 // 16], min(16, P - p0)
            for pool, sc, src in ((kp, ks, w.k), (vp, vs, w.v)):
                for h in range(2):
                    x = bf16_to_f64(src[a + p0:a + p0 + rows, h])
                    amax = np.abs(x).max()
                    assert sc[page, h] == np.float32(np.float32(amax) / np.float32(448.0))
                    dec = e4m3_to_f64(pool[page, h, :rows]) * np.float64(sc[page, h])
                    # e4m3 has 3 mantissa bits: half an ulp is 2^-4 relative (normal range).
                    err = np.abs(dec - x)
                    assert np.all(err <= np.maximum(np.abs(x) * 2.0 ** -4, 2.0 ** -10 * sc[page, h]) + 1e-12)
                    assert np.abs(dec).max() == pytest.approx(amax, rel=2.0 ** -4)


def test_fp8_all_zero_page_gets_scale_one():
    w = _wl((16,), Hq=2, Hkv=1, d=32, seed=2, kv_dtype="fp8")
    zk = np.zeros_like(w.k)
    kp, _, ks, _ = prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale, v_scale=w.v_scale,
                                    kv_dtype="fp8", page_size=16, prefix_block_table=w.prefix_block_table,
                                    prefix_offs=w.prefix_offs, k=zk, v=w.v)
    page = w.prefix_block_table[0][0]
    assert ks[page, 0] == np.float32(1.0)
    assert np.all(kp[page, 0] == 0)
