"""Pins for the oracle's pre-attention decode step (CPU only).

The fp64 -> bf16 rounding is checked against torch's float32 -> bfloat16 cast
(where the input is a float32 value), against hand-worked ties, and at values
that a detour through float32 would round differently. The RMS norm is
checked against torch's rms_norm (float64) and its invariants. The rotary
embedding is checked against complex multiplication, closed-form angles that
pin its frequency exponent and its pairing, and the invariants that make it a
relative position code (norm-preserving, composes additively, dot products
depend only on the position difference). The step as a whole is checked for
positions, per-head independence, and the pool rows it writes.
"""
import numpy as np
import pytest
import torch

from oracle import decode_positions, decode_step_prep, kv_append, qk_prep, rms_norm, rope
from oracle.formats import bf16_to_f64, f64_to_bf16_bits
from workloads import make_qkprep_inputs, make_workload


# ---------------------------------------------------------------- bf16 rounding

def test_bf16_round_matches_torch_on_float32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1e-40, -3e-39, 3.3e38, -3.3e38], dtype=np.float32)]).astype(np.float32)
    ours = f64_to_bf16_bits(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_round_ties_to_even_by_hand():
    one = 0x3F80
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: even mantissa (1.0) wins.
    assert f64_to_bf16_bits(1.0 + 2.0 ** -8) == one
    # 1 + 3 * 2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: the even one is 1 + 2^-6.
    assert f64_to_bf16_bits(1.0 + 3 * 2.0 ** -8) == one + 2
    assert f64_to_bf16_bits(-(1.0 + 3 * 2.0 ** -8)) == 0x8000 | (one + 2)
    # The smallest subnormal 2^-133, and half of it (a tie to zero).
    assert f64_to_bf16_bits(2.0 ** -133) == 1
    assert f64_to_bf16_bits(2.0 ** -134) == 0
    assert f64_to_bf16_bits(1.5 * 2.0 ** -133) == 2


def test_bf16_round_is_single_rounding_from_float64():
    # Just above a bf16 tie by less than a float32 ulp: float32 would land on
    # the tie and round to even (down); a single rounding goes up.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert np.float32(x) == np.float32(1.0 + 2.0 ** -8)
    assert f64_to_bf16_bits(x) == 0x3F81
    # Every bf16 value round-trips exactly.
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = bf16_to_f64(bits)
    ok = np.isfinite(vals) & ~((bits == 0x8000))
    assert np.array_equal(f64_to_bf16_bits(vals[ok]), bits[ok])


def test_bf16_round_rejects_non_finite():
    with pytest.raises(ValueError):
        f64_to_bf16_bits(np.array([1.0, np.inf]))


# ---------------------------------------------------------------- RMS norm

def test_rms_norm_matches_torch_fp64():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 7, 128)) * 3.0
    w = rng.standard_normal(128)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (128,), torch.from_numpy(w), eps=1e-6).numpy()
    np.testing.assert_allclose(rms_norm(x, w, 1e-6), ref, rtol=1e-13, atol=1e-15)


def test_rms_norm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((9, 64))
    y = rms_norm(x, np.ones(64), eps=0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-14)
    np.testing.assert_allclose(rms_norm(37.5 * x, np.ones(64), eps=0.0), y, rtol=1e-13)
    # A negative scale flips the sign only.
    np.testing.assert_allclose(rms_norm(-2.0 * x, np.ones(64), eps=0.0), -y, rtol=1e-13)


def test_rms_norm_constant_vector_closed_form():
    w = np.linspace(0.5, 2.0, 32)
    for c, eps in ((3.0, 0.0), (-0.25, 0.0), (1e-3, 1e-6), (0.0, 1e-6)):
        got = rms_norm(np.full(32, c), w, eps)
        np.testing.assert_allclose(got, w * c / np.sqrt(c * c + eps), rtol=1e-14, atol=0)


# ---------------------------------------------------------------- rotary embedding

def test_rope_is_complex_rotation_of_half_pairs():
    rng = np.random.default_rng(3)
    d, base = 128, 1e6
    y = rng.standard_normal((4, d))
    pos = np.array([0.0, 1.0, 1234.0, 40000.0])
    z = y[:, : d // 2] + 1j * y[:, d // 2:]
    freq = np.exp(-np.log(base) * np.arange(0, d, 2) / d)
    r = z * np.exp(1j * pos[:, None] * freq)
    got = rope(y, pos, base)
    # The two forms compute the angle pos * freq with different roundings: at
    # pos 4e4 that is a few 1e-12 apart.
    np.testing.assert_allclose(got[:, : d // 2], r.real, rtol=0, atol=1e-10)
    np.testing.assert_allclose(got[:, d // 2:], r.imag, rtol=0, atol=1e-10)


def test_rope_angles_closed_form():
    # d = 128, base 1e6: pair 0 turns by pos, pair 32 by pos * 1e-3 (exponent
    # 2 * 32 / 128 = 1/2), pair 48 by pos * 10^-4.5; pair i mixes only
    # elements i and i + 64.
    d = 128
    for i, rate in ((0, 1.0), (32, 1e-3), (48, 10 ** -4.5), (63, 1e6 ** (-126 / 128))):
        e = np.zeros(d)
        e[i] = 1.0
        pos = 1000.0
        out = rope(e, pos, 1e6)
        mask = np.ones(d, dtype=bool)
        mask[[i, i + 64]] = False
        assert np.all(out[mask] == 0.0)
        np.testing.assert_allclose(np.arctan2(out[i + 64], out[i]), np.angle(np.exp(1j * pos * rate)), atol=1e-12)


def test_rope_position_zero_is_identity_and_preserves_pair_norms():
    rng = np.random.default_rng(4)
    y = rng.standard_normal((3, 64))
    np.testing.assert_array_equal(rope(y, np.zeros(3)), y)
    out = rope(y, np.array([7.0, 999.0, 123456.0]))
    np.testing.assert_allclose(out[:, :32] ** 2 + out[:, 32:] ** 2, y[:, :32] ** 2 + y[:, 32:] ** 2, rtol=1e-12)


def test_rope_composes_and_encodes_relative_position():
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    np.testing.assert_allclose(rope(rope(q, 300.0), 1700.0), rope(q, 2000.0), rtol=1e-9, atol=1e-12)
    dots = [rope(q, m) @ rope(k, m - 250.0) for m in (250.0, 1000.0, 5000.0, 33333.0)]
    np.testing.assert_allclose(dots, dots[0], rtol=1e-9)


# ---------------------------------------------------------------- the decode-side step

def test_decode_positions_by_hand():
    got = decode_positions([1, 0, 1, 2], [10, 20, 0], [0, 5, 7, 3])
    assert got.tolist() == [20, 15, 27, 3]


def test_qk_prep_heads_are_independent_and_use_their_sequence_position():
    x = make_qkprep_inputs(num_seqs=3, num_q_heads=8, num_kv_heads=2, head_dim=64, seed=6)
    pos = np.array([0, 17, 4099])
    qb, kb, q, k = qk_prep(q_in=x.q_in, k_in=x.k_in, q_norm_w=x.q_norm_w, k_norm_w=x.k_norm_w, positions=pos)
    wq, wk = bf16_to_f64(x.q_norm_w), bf16_to_f64(x.k_norm_w)
    for s in range(3):
        for h in range(8):
            one = rope(rms_norm(bf16_to_f64(x.q_in[s, h]), wq), float(pos[s]))
            np.testing.assert_allclose(q[s, h], one, rtol=1e-14, atol=1e-15)
        for h in range(2):
            one = rope(rms_norm(bf16_to_f64(x.k_in[s, h]), wk), float(pos[s]))
            np.testing.assert_allclose(k[s, h], one, rtol=1e-14, atol=1e-15)
    # Position 0: the output is just the normalised input.
    np.testing.assert_allclose(q[0], rms_norm(bf16_to_f64(x.q_in[0]), wq), rtol=1e-14)
    # Rounded outputs are within half a bf16 ulp of the exact values.
    for b, e in ((qb, q), (kb, k)):
        err = np.abs(bf16_to_f64(b) - e)
        assert np.all(err <= np.ldexp(1.0, np.frexp(np.abs(e))[1] - 9) + 1e-300)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_decode_step_prep_writes_rotated_k_and_raw_v(kv_dtype):
    S, Hq, Hkv, d = 6, 8, 2, 64
    wl = make_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, seq_to_group=[0, 0, 0, 1, 1, 1],
                       prefix_lens=[40, 3], resp_lens=[0, 15, 16, 31, 1, 50], seed=7, append=True,
                       kv_dtype=kv_dtype)
    x = make_qkprep_inputs(num_seqs=S, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, seed=8)
    qb, kb, pool = decode_step_prep(q_in=x.q_in, k_in=x.k_in, v_in=x.v_in, q_norm_w=x.q_norm_w,
                                    k_norm_w=x.k_norm_w, k_pages=wl.k_pages, v_pages=wl.v_pages,
                                    k_scale=wl.k_scale, v_scale=wl.v_scale, kv_dtype=kv_dtype, page_size=16,
                                    seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                                    resp_lens=wl.resp_lens, resp_block_table=wl.resp_block_table)
    pos = wl.prefix_lens[wl.seq_to_group] + wl.resp_lens
    assert pos.tolist() == [40, 55, 56, 34, 4, 53]
    qb2, kb2, _, _ = qk_prep(q_in=x.q_in, k_in=x.k_in, q_norm_w=x.q_norm_w, k_norm_w=x.k_norm_w, positions=pos)
    assert np.array_equal(qb, qb2) and np.array_equal(kb, kb2)
    kp, vp, ks, vs = pool
    for s in range(S):
        t = int(wl.resp_lens[s])
        page, r = int(wl.resp_block_table[s][t // 16]), t % 16
        if kv_dtype == "bf16":
            assert np.array_equal(kp[page, :, r], kb[s]) and np.array_equal(vp[page, :, r], x.v_in[s])
        else:
            # Dequantised rows within the e4m3 half-ulp bound (3 mantissa bits) of their sources.
            for pages, sc, src in ((kp, ks, kb[s]), (vp, vs, x.v_in[s])):
                from oracle import e4m3_to_f64
                deq = e4m3_to_f64(pages[page, :, r]) * sc[page][:, None]
                ref = bf16_to_f64(src)
                assert np.all(np.abs(deq - ref) <= np.abs(ref) / 16 + sc[page][:, None] * 2.0 ** -9 + 1e-30)
    # Every other row of the pool is untouched.
    ref_pool = kv_append(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale, v_scale=wl.v_scale,
                         kv_dtype=kv_dtype, page_size=16, resp_lens=wl.resp_lens,
                         resp_block_table=wl.resp_block_table, k_new=kb, v_new=x.v_in)
    for a, b in zip(pool, ref_pool):
        if a is not None:
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
