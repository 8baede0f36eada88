"""Pins for the oracle's paged decode attention (CPU only).

The oracle is checked against torch's scaled_dot_product_attention (float64,
CPU) on dense copies of the keys, against closed forms (constant V, one key,
q = 0, one dominant key at every slot) and against invariants (page
permutations, shared vs duplicated prefix, GQA head mapping).
"""
import numpy as np
import pytest
import torch

from oracle import decode_attention
from tests.paged import (bf16_bits, bf16_value, dense_keys, oracle_on, paged_from_dense,
                         random_dense)


def sdpa_ref(q_bits, K, V, scale, n_rep):
    """torch SDPA over dense fp64 K, V [N][Hkv][d] for one sequence's q [Hq][d]."""
    q = torch.from_numpy(bf16_value(q_bits))[:, None, :]             # [Hq][1][d]
    k = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(n_rep, 0)   # [Hq][N][d]
    v = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(n_rep, 0)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=float(scale))
    s = (q @ k.transpose(1, 2))[:, 0, :] * float(scale)
    return o[:, 0, :].numpy(), torch.logsumexp(s, dim=-1).numpy()


CASES = [
    # S, G, Hq, Hkv, d, prefix_lens, resp_lens
    (4, 1, 4, 2, 64, [128], [61, 52, 59, 32]),
    (6, 2, 8, 2, 64, [17, 33], [0, 1, 15, 16, 17, 40]),
    (5, 3, 16, 8, 128, [64, 0, 5], [3, 100, 0, 31, 48]),
    (3, 3, 4, 4, 32, [1, 2, 3], [0, 0, 7]),        # MHA (n_rep = 1)
    (4, 2, 8, 1, 64, [20, 20], [9, 0, 33, 2]),      # n_rep = 8
]


@pytest.mark.parametrize("case", CASES)
def test_matches_torch_sdpa_fp64(case):
    S, G, Hq, Hkv, d, P, L = case
    rng = np.random.default_rng(sum(P) + sum(L) + d)
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=Hq, Hkv=Hkv, d=d,
                                          prefix_lens=P, resp_lens=L)
    wl = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=Hkv, seed=1, softmax_scale=0.1)
    out, lse = oracle_on(wl)
    for s in range(S):
        K, V = dense_keys(pk, pv, rk, rv, s2g, s)
        o_ref, l_ref = sdpa_ref(q[s], K, V, np.float64(np.float32(0.1)), Hq // Hkv)
        np.testing.assert_allclose(out[s], o_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[s], l_ref, rtol=0, atol=1e-12)


def _wl(seed=0, S=4, G=2, Hq=4, Hkv=2, d=64, P=(20, 37), L=(0, 5, 16, 33)):
    rng = np.random.default_rng(seed)
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=Hq, Hkv=Hkv, d=d,
                                          prefix_lens=list(P), resp_lens=list(L))
    return pk, pv, rk, rv, s2g, q


def test_constant_v_returns_constant():
    pk, pv, rk, rv, s2g, q = _wl(1)
    c = bf16_bits(np.full(1, 0.8125))[0]
    pv = [np.full_like(x, c) for x in pv]
    rv = [np.full_like(x, c) for x in rv]
    out, _ = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2))
    np.testing.assert_allclose(out, 0.8125, rtol=0, atol=1e-14)


@pytest.mark.parametrize("where", ["prefix", "response"])
def test_single_key_returns_its_value_and_score(where):
    rng = np.random.default_rng(2)
    P, L = (1, 0) if where == "prefix" else (0, 1)
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=1, G=1, Hq=4, Hkv=2, d=64, prefix_lens=[P],
                                          resp_lens=[L])
    wl = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2)
    out, lse = oracle_on(wl)
    K, V = dense_keys(pk, pv, rk, rv, s2g, 0)
    sigma = np.float64(np.float32(wl.softmax_scale))
    for j in range(4):
        h = j // 2
        assert np.array_equal(out[0, j], V[0, h])
        assert lse[0, j] == pytest.approx(sigma * float(bf16_value(q[0, j]) @ K[0, h]), abs=1e-13)


def test_zero_query_gives_log_count_and_mean():
    pk, pv, rk, rv, s2g, q = _wl(3, P=(20, 37), L=(0, 5, 16, 333))
    q = np.zeros_like(q)
    wl = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2)
    out, lse = oracle_on(wl)
    for s in range(4):
        K, V = dense_keys(pk, pv, rk, rv, s2g, s)
        N = K.shape[0]
        np.testing.assert_allclose(lse[s], np.log(N), rtol=0, atol=1e-12)
        np.testing.assert_allclose(out[s], np.repeat(V.mean(0), 2, axis=0), rtol=0, atol=1e-12)


def test_empty_key_set():
    pk, pv, rk, rv, s2g, q = _wl(4, S=2, G=2, P=(0, 3), L=(0, 0))
    out, lse = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2))
    assert np.all(out[0] == 0) and np.all(lse[0] == -np.inf)
    assert np.all(np.isfinite(lse[1]))


def test_dominant_key_at_every_slot_is_selected():
    """q parallel to one key with a huge score picks exactly that key's V, at every slot."""
    d, P, L = 64, 37, 21
    rng = np.random.default_rng(5)
    base = random_dense(rng, S=1, G=1, Hq=2, Hkv=1, d=d, prefix_lens=[P], resp_lens=[L])
    pk, pv, rk, rv, s2g, _ = base
    for t in range(P + L):
        kk = [x.copy() for x in pk], [x.copy() for x in rk]
        Kd = kk[0][0] if t < P else kk[1][0]
        row = t if t < P else t - P
        Kd[:] = bf16_bits(np.zeros((Kd.shape[0], 1, d)))
        Kd[row, 0, :] = bf16_bits(np.full((d,), 1.0))
        q = bf16_bits(np.full((1, 2, d), 4.0))                  # score 4*64/8 = 32 vs 0
        wl = paged_from_dense(kk[0], pv, kk[1], rv, s2g, q, num_kv_heads=1, seed=t)
        out, _ = oracle_on(wl)
        V = dense_keys(pk, pv, rk, rv, s2g, 0)[1]
        np.testing.assert_allclose(out[0, 0], V[t, 0], rtol=0, atol=1e-9 * (P + L) * 10)


def test_physical_page_permutation_is_bitwise_invariant():
    pk, pv, rk, rv, s2g, q = _wl(6, P=(40, 70), L=(3, 50, 0, 99))
    o1, l1 = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2, seed=11))
    o2, l2 = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2, seed=12,
                                        pad_pages=5))
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_logical_page_order_permutation_within_tolerance():
    pk, pv, rk, rv, s2g, q = _wl(7, S=2, G=1, P=(64,), L=(96, 48))
    wl = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2)
    o1, l1 = oracle_on(wl)
    # Reverse the (full) page order of every sequence's response and of the prefix.
    wl.resp_block_table[0, :6] = wl.resp_block_table[0, :6][::-1].copy()
    wl.resp_block_table[1, :3] = wl.resp_block_table[1, :3][::-1].copy()
    wl.prefix_block_table[0, :4] = wl.prefix_block_table[0, :4][::-1].copy()
    o2, l2 = oracle_on(wl)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def test_shared_prefix_equals_duplicated_prefix():
    pk, pv, rk, rv, s2g, q = _wl(8, S=4, G=2, P=(45, 16), L=(7, 0, 33, 16))
    shared = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2))
    # Each sequence gets a private copy: prefix length 0, response = prefix ++ response.
    S = 4
    empty = [pk[0][:0]] * S
    drk = [np.concatenate([pk[s2g[s]], rk[s]]) for s in range(S)]
    drv = [np.concatenate([pv[s2g[s]], rv[s]]) for s in range(S)]
    dup = oracle_on(paged_from_dense(empty, empty, drk, drv, np.arange(S), q, num_kv_heads=2))
    np.testing.assert_allclose(shared[0], dup[0], rtol=0, atol=1e-13)
    np.testing.assert_allclose(shared[1], dup[1], rtol=0, atol=1e-13)


def test_gqa_mapping_nonzero_v_in_one_kv_head():
    pk, pv, rk, rv, s2g, q = _wl(9, S=2, G=1, Hq=8, Hkv=4, P=(20,), L=(5, 9))
    zero = bf16_bits(np.zeros(1))[0]
    for arrs in (pv, rv):
        for x in arrs:
            x[:, [0, 1, 3], :] = zero                            # only kv-head 2 nonzero
    out, _ = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=4))
    nz = np.abs(out).sum(axis=2) > 0                            # [S][Hq]
    assert np.array_equal(nz, np.tile([False, False, False, False, True, True, False, False], (2, 1)))


def test_padding_rows_are_never_read():
    """Pools are poisoned with NaN beyond each page's valid rows; results stay finite."""
    pk, pv, rk, rv, s2g, q = _wl(10, P=(19, 33), L=(1, 15, 17, 31))
    out, lse = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=2))
    assert np.isfinite(out).all() and np.isfinite(lse).all()


def test_fp8_pool_matches_sdpa_on_dequantised_values():
    """e4m3 codes times the per-(page, head) scale, checked with torch's own fp8 decode."""
    from workloads import make_workload
    wl = make_workload(num_q_heads=4, num_kv_heads=2, head_dim=64, seq_to_group=[0, 0, 1],
                       prefix_lens=[20, 40], resp_lens=[3, 30, 17], seed=4, kv_dtype="fp8")
    out, lse = oracle_on(wl)
    def deq(codes, scales, pages, rows, h):
        c = torch.from_numpy(codes[pages, h, rows, :]).view(torch.float8_e4m3fn).double().numpy()
        return c * scales[pages, h][:, None].astype(np.float64)
    ps = wl.page_size
    for s in range(3):
        g = wl.seq_to_group[s]
        P, L = wl.prefix_lens[g], wl.resp_lens[s]
        pages = np.concatenate([wl.prefix_block_table[g][np.arange(P) // ps],
                                wl.resp_block_table[s][np.arange(L) // ps]])
        rows = np.concatenate([np.arange(P) % ps, np.arange(L) % ps])
        K = np.stack([deq(wl.k_pages, wl.k_scale, pages, rows, h) for h in range(2)], 1)
        V = np.stack([deq(wl.v_pages, wl.v_scale, pages, rows, h) for h in range(2)], 1)
        o_ref, l_ref = sdpa_ref(wl.q[s], K, V, np.float64(wl.softmax_scale), 2)
        np.testing.assert_allclose(out[s], o_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[s], l_ref, rtol=0, atol=1e-12)


def test_scale_is_the_callers_fp32_value_widened():
    """A float64 scale argument is first rounded to fp32 (what a C caller passes)."""
    rng = np.random.default_rng(31)
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=2, G=1, Hq=2, Hkv=1, d=64, prefix_lens=[40],
                                          resp_lens=[10, 70])
    wl = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=1)
    out, lse = decode_attention(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=None, v_scale=None,
                                kv_dtype="bf16", page_size=16, seq_to_group=wl.seq_to_group,
                                prefix_lens=wl.prefix_lens, prefix_block_table=wl.prefix_block_table,
                                resp_lens=wl.resp_lens, resp_block_table=wl.resp_block_table,
                                q=wl.q, softmax_scale=0.1)
    for s in range(2):
        K, V = dense_keys(pk, pv, rk, rv, s2g, s)
        o_ref, l_ref = sdpa_ref(q[s], K, V, np.float64(np.float32(0.1)), 2)
        np.testing.assert_allclose(lse[s], l_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(out[s], o_ref, rtol=0, atol=1e-12)
