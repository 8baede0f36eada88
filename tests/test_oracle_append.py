"""Pins for the oracle's KV append (CPU only)."""
import numpy as np
import pytest

from oracle import append_for_workload, attention_for_workload, bf16_to_f32, e4m3_to_f64
from tests.paged import bf16_bits
from workloads import make_workload


def _wl(kv_dtype, resp_lens, seed=0, **kw):
    S = len(resp_lens)
    return make_workload(num_q_heads=4, num_kv_heads=2, head_dim=64, seq_to_group=np.arange(S) % 2,
                         prefix_lens=[20, 33], resp_lens=resp_lens, seed=seed, append=True,
                         kv_dtype=kv_dtype, **kw)


def test_bf16_append_writes_exactly_the_new_slots():
    wl = _wl("bf16", [0, 15, 16, 31, 40])
    kp, vp, _, _ = append_for_workload(wl)
    changed = set()
    for pool, new, old in ((kp, wl.k_new, wl.k_pages), (vp, wl.v_new, wl.v_pages)):
        diff = np.argwhere(pool != old)
        changed |= {(int(p), int(h), int(r)) for p, h, r, _ in diff}
        for s, L in enumerate(wl.resp_lens):     # brute force: look the slot up by hand
            page = wl.resp_block_table[s][L // 16]
            for h in range(2):
                assert np.array_equal(pool[page, h, L % 16], new[s, h])
    want = {(int(wl.resp_block_table[s][L // 16]), h, int(L % 16))
            for s, L in enumerate(wl.resp_lens) for h in range(2)}
    assert changed == want


def test_appended_token_is_the_last_key_attention_reads():
    wl = _wl("bf16", [0, 7, 16, 33])
    d = 64
    wl.k_new[:] = bf16_bits(np.full((4, 2, d), 3.0))
    wl.q[:] = bf16_bits(np.full((4, 4, d), 3.0))   # new key's score 72 dominates N(0,1) keys
    out, _ = attention_for_workload(wl, pool=append_for_workload(wl))
    vn = bf16_to_f32(wl.v_new).astype(np.float64)
    np.testing.assert_allclose(out, np.repeat(vn, 2, axis=1), rtol=0, atol=1e-6)


def _fp8_slot(wl, pool, s):
    kp, vp, ks, vs = pool
    L = int(wl.resp_lens[s])
    page = int(wl.resp_block_table[s][L // 16])
    return page, L % 16


@pytest.mark.parametrize("which", ["k", "v"])
def test_fp8_first_row_sets_scale_from_amax(which):
    wl = _wl("fp8", [0, 16, 32, 48])
    pool = append_for_workload(wl)
    codes, scales = (pool[0], pool[2]) if which == "k" else (pool[1], pool[3])
    new = wl.k_new if which == "k" else wl.v_new
    for s in range(4):
        page, r = _fp8_slot(wl, pool, s)
        assert r == 0
        for h in range(2):
            x = bf16_to_f32(new[s, h])
            amax = np.abs(x).max()
            assert scales[page, h] == np.float32(amax / np.float32(448))
            row = e4m3_to_f64(codes[page, h, 0])
            assert np.abs(row).max() == 448.0           # the max-abs element maps to +-448
            err = np.abs(row * scales[page, h] - x)
            ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(x) / scales[page, h], 2.0 ** -6))) - 3)
            assert np.all(err <= ulp / 2 * scales[page, h] * (1 + 1e-6))


def test_fp8_keep_scale_when_new_row_fits_and_leave_old_rows():
    wl = _wl("fp8", [5, 9])
    # Shrink the new token so it fits the existing scale.
    wl.k_new[:] = bf16_bits(bf16_to_f32(wl.k_new) * np.float32(1e-3))
    pool = append_for_workload(wl)
    for s in range(2):
        page, r = _fp8_slot(wl, pool, s)
        for h in range(2):
            assert pool[2][page, h] == wl.k_scale[page, h]
            assert np.array_equal(pool[0][page, h, :r], wl.k_pages[page, h, :r])
            y = bf16_to_f32(wl.k_new[s, h]).astype(np.float64) / wl.k_scale[page, h]
            got = e4m3_to_f64(pool[0][page, h, r])
            ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(y), 2.0 ** -6))) - 3)
            assert np.all(np.abs(got - y) <= ulp / 2 * (1 + 1e-6))


def test_fp8_growing_amax_rescales_and_requantises_previous_rows():
    wl = _wl("fp8", [5, 9])
    wl.v_new[:] = bf16_bits(bf16_to_f32(wl.v_new) * np.float32(50.0))
    pool = append_for_workload(wl)
    for s in range(2):
        page, r = _fp8_slot(wl, pool, s)
        for h in range(2):
            old_s, new_s = wl.v_scale[page, h], pool[3][page, h]
            x = bf16_to_f32(wl.v_new[s, h])
            assert new_s == np.float32(np.abs(x).max() / np.float32(448)) and new_s > old_s
            before = e4m3_to_f64(wl.v_pages[page, h, :r]) * old_s
            after = e4m3_to_f64(pool[1][page, h, :r]) * new_s
            # Requantising at a coarser scale moves each value by at most half a new ulp.
            ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(before) / new_s, 2.0 ** -6))) - 3) * new_s
            assert np.all(np.abs(after - before) <= ulp / 2 * (1 + 1e-6) + 1e-30)


def test_fp8_append_is_idempotent():
    wl = _wl("fp8", [0, 5, 16, 21], seed=3)
    wl.k_new[:] = bf16_bits(bf16_to_f32(wl.k_new) * np.float32(20.0))
    once = append_for_workload(wl)
    wl2 = _wl("fp8", [0, 5, 16, 21], seed=3)
    wl2.k_new[:] = wl.k_new
    wl2.k_pages, wl2.v_pages, wl2.k_scale, wl2.v_scale = once
    twice = append_for_workload(wl2)
    for a, b in zip(once, twice):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("growth,rescaled", [(1.02, True), (1.0, False)])
def test_fp8_rescale_threshold_is_448_times_old_scale(growth, rescaled):
    """amax_new just above 448 * scale_old rescales; exactly at it keeps the scale."""
    wl = _wl("fp8", [5, 9], seed=5)
    for s in range(2):
        L = int(wl.resp_lens[s])
        page = int(wl.resp_block_table[s][L // 16])
        for h in range(2):
            x = bf16_to_f32(wl.k_new[s, h]).copy()
            target = np.float32(448) * wl.k_scale[page, h] * np.float32(growth)
            x = x / np.abs(x).max() * target
            x[np.argmax(np.abs(x))] = target          # the max element sits exactly on the target
            bits = bf16_bits(x)
            if growth == 1.0:      # bf16 rounding moved the max: put the old scale exactly on it
                wl.k_scale[page, h] = np.float32(np.abs(bf16_to_f32(bits)).max()) / np.float32(448)
            wl.k_new[s, h] = bits
    pool = append_for_workload(wl)
    for s in range(2):
        L = int(wl.resp_lens[s])
        page = int(wl.resp_block_table[s][L // 16])
        for h in range(2):
            amax = np.abs(bf16_to_f32(wl.k_new[s, h])).max()
            fits = amax <= np.float32(448) * wl.k_scale[page, h]
            assert fits != rescaled
            assert (pool[2][page, h] != wl.k_scale[page, h]) == rescaled
