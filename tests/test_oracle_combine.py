"""Pins for the oracle's log-sum-exp merge (CPU only)."""
import numpy as np

from oracle import lse_combine
from tests.paged import oracle_on, paged_from_dense, random_dense


def test_split_prefix_and_response_then_combine_equals_unsplit():
    rng = np.random.default_rng(21)
    S, G, Hq, Hkv, d = 5, 2, 8, 4, 64
    P, L = [30, 77], [0, 12, 16, 50, 129]
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=Hq, Hkv=Hkv, d=d,
                                          prefix_lens=P, resp_lens=L, seq_to_group=[0, 1, 1, 0, 1])
    full = oracle_on(paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=Hkv))
    empty_p = [x[:0] for x in pk]
    empty_r = [x[:0] for x in rk]
    # Three disjoint key subsets: the prefix, the first half of the response, the rest.
    half = [len(x) // 2 for x in rk]
    parts = [oracle_on(paged_from_dense(pk, pv, empty_r, empty_r, s2g, q, num_kv_heads=Hkv)),
             oracle_on(paged_from_dense(empty_p, empty_p, [x[:h] for x, h in zip(rk, half)],
                                        [x[:h] for x, h in zip(rv, half)], s2g, q, num_kv_heads=Hkv)),
             oracle_on(paged_from_dense(empty_p, empty_p, [x[h:] for x, h in zip(rk, half)],
                                        [x[h:] for x, h in zip(rv, half)], s2g, q, num_kv_heads=Hkv))]
    R = S * Hq
    o_parts = np.stack([p[0].reshape(R, d) for p in parts], axis=1).reshape(3 * R, d)
    l_parts = np.stack([p[1].reshape(R) for p in parts], axis=1).reshape(3 * R)
    out, lse = lse_combine(o_parts, l_parts, np.arange(R + 1) * 3)
    np.testing.assert_allclose(out, full[0].reshape(R, d), rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, full[1].reshape(R), rtol=0, atol=1e-13)


def test_equal_lse_parts_average_and_add_log2():
    o = np.array([[1.0, 2.0], [3.0, -2.0]])
    out, lse = lse_combine(o, np.array([0.7, 0.7]), [0, 2])
    np.testing.assert_allclose(out[0], [2.0, 0.0], atol=1e-15)
    np.testing.assert_allclose(lse[0], 0.7 + np.log(2.0), atol=1e-15)


def test_weights_follow_exp_lse():
    o = np.array([[1.0], [0.0]])
    out, lse = lse_combine(o, np.array([np.log(3.0), 0.0]), [0, 2])   # weights 3 : 1
    np.testing.assert_allclose(out[0, 0], 0.75, atol=1e-15)
    np.testing.assert_allclose(lse[0], np.log(4.0), atol=1e-15)


def test_empty_part_is_a_no_op_even_with_garbage_output():
    o = np.array([[0.25, -1.0], [np.nan, np.inf]])
    out, lse = lse_combine(o, np.array([1.5, -np.inf]), [0, 2])
    np.testing.assert_array_equal(out[0], [0.25, -1.0])
    assert lse[0] == 1.5


def test_rows_without_parts_or_with_only_empty_parts():
    o = np.array([[5.0, 5.0]])
    out, lse = lse_combine(o, np.array([-np.inf]), [0, 0, 1])
    assert np.all(out == 0) and np.all(lse == -np.inf)
