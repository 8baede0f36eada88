"""Pins for the oracle's bf16 / e4m3fn codecs (CPU only)."""
import os

import numpy as np
import pytest
import torch

from oracle import bf16_to_f64, e4m3_encode, e4m3_to_f64

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3fn_spec_values.txt")


def test_bf16_decode_matches_torch_all_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_e4m3_decode_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ours = e4m3_to_f64(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    nan = np.isnan(ref)
    assert nan.sum() == 2 and nan[0x7F] and nan[0xFF]
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def test_e4m3_decode_matches_spec_table():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    assert len(rows) >= 10
    for code, val in rows:
        got = e4m3_to_f64(np.uint8(int(code, 16)))
        want = float(val)
        if np.isnan(want):
            assert np.isnan(got), code
        else:
            assert got == want and np.signbit(got) == np.signbit(want), (code, got, want)


def _torch_encode(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_e4m3_encode_matches_torch_on_grid_midpoints_and_random():
    pos = e4m3_to_f64(np.arange(127, dtype=np.uint8))
    mids = (pos[1:] + pos[:-1]) / 2                       # exact ties (representable in fp32)
    near = np.concatenate([np.nextafter(mids.astype(np.float32), np.float32(np.inf)),
                           np.nextafter(mids.astype(np.float32), np.float32(0))])
    rnd = np.random.default_rng(7).standard_normal(200_000).astype(np.float32) * 30
    x = np.concatenate([pos, mids, near, rnd, [0.0, 447.9, 448.0, 463.9]]).astype(np.float32)
    x = x[np.abs(x) < 464]                                # torch overflows to NaN from 464 on
    x = np.concatenate([x, -x])
    assert np.array_equal(e4m3_encode(x), _torch_encode(x))


def test_e4m3_encode_saturates_and_keeps_sign():
    x = np.array([448.0, 464.0, 1e6, -1e6, -0.0, 0.0, 2.0 ** -11], dtype=np.float32)
    assert list(e4m3_encode(x)) == [0x7E, 0x7E, 0x7E, 0xFE, 0x80, 0x00, 0x00]
    with pytest.raises(ValueError):
        e4m3_encode(np.array([np.nan], dtype=np.float32))


def test_e4m3_roundtrip_error_within_half_ulp():
    x = np.random.default_rng(3).uniform(-448, 448, 100_000).astype(np.float32)
    y = e4m3_to_f64(e4m3_encode(x))
    a = np.abs(x.astype(np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -6)))
    ulp = 2.0 ** (e - 3)
    assert np.all(np.abs(y - x) <= ulp / 2)


def test_e4m3_lookup_equals_the_bit_field_definition_on_pool_shapes():
    """The decode table is the bit-field definition evaluated per code: same values on any array."""
    from oracle.formats import _e4m3_decode_definition
    codes = np.random.default_rng(5).integers(0, 256, (3, 2, 16, 8)).astype(np.uint8)
    a, b = e4m3_to_f64(codes), _e4m3_decode_definition(codes)
    assert a.shape == codes.shape and a.dtype == np.float64
    nan = np.isnan(b)
    assert np.array_equal(np.isnan(a), nan) and np.array_equal(a[~nan], b[~nan])
    assert np.array_equal(np.signbit(a[~nan]), np.signbit(b[~nan]))
