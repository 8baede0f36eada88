"""Bit-level decoding of bf16 and OCP FP8 e4m3fn, and round-to-nearest-even encoding.

bf16 is the upper half of an IEEE-754 binary32, so decoding is a 16-bit left
shift. OCP e4m3fn (OCP 8-bit Floating Point Specification v1.0): 1 sign bit,
4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 encodes
subnormals m * 2^-9; there are no infinities and only S.1111.111 is NaN, so the
largest finite magnitude is 1.75 * 2^8 = 448.
"""
import numpy as np

E4M3_MAX = 448.0


def bf16_to_f32(bits) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(bits) -> np.ndarray:
    with np.errstate(invalid="ignore"):       # signalling-NaN patterns widen to quiet NaN
        return bf16_to_f32(bits).astype(np.float64)


def _e4m3_decode_definition(codes) -> np.ndarray:
    """e4m3fn code -> value, straight from the bit fields (sign, exponent, mantissa)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = (c >> 7) & 1
    e = (c >> 3) & 0xF
    m = c & 0x7
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(sign == 1, -mag, mag)


# The definition evaluated once for each of the 256 codes; decoding a pool is
# then a lookup (the same values, without the per-element field arithmetic).
_E4M3_VALUES = _e4m3_decode_definition(np.arange(256, dtype=np.uint8))


def e4m3_to_f64(codes) -> np.ndarray:
    return _E4M3_VALUES[np.asarray(codes, dtype=np.uint8)]


# Magnitudes of the 127 non-negative finite codes 0x00..0x7E, increasing with the code.
_POS_VALUES = e4m3_to_f64(np.arange(127, dtype=np.uint8))


def e4m3_encode(x) -> np.ndarray:
    """Encode float32 values to e4m3fn codes, rounding to nearest, ties to even.

    Magnitudes at or above 448 saturate to 448 (code 0x7E); NaN is never
    produced. The sign bit is copied from the input, so -0.0 encodes as 0x80.
    On the code grid of non-negative values, "even" is a code with a clear
    least significant (mantissa) bit.
    """
    x = np.asarray(x, dtype=np.float32)
    if np.isnan(x).any():
        raise ValueError("e4m3_encode: NaN input")
    sign = (x.view(np.uint32) >> np.uint32(31)).astype(np.uint8)
    a = np.abs(x).astype(np.float64)
    hi = np.searchsorted(_POS_VALUES, a, side="left")       # first value >= a
    hi = np.minimum(hi, 126)
    lo = np.maximum(hi - 1, 0)
    d_hi = _POS_VALUES[hi] - a
    d_lo = a - _POS_VALUES[lo]
    exact = d_hi == 0
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(exact, hi, np.where(pick_hi, hi, lo))
    code = np.where(a >= E4M3_MAX, 126, code)
    return (code.astype(np.uint8) | (sign << np.uint8(7))).astype(np.uint8)


def f64_to_bf16_bits(x) -> np.ndarray:
    """Round float64 values to bf16 (nearest, ties to even) in one step; bit patterns as uint16.

    A bf16 value is a multiple of ulp = 2^(e - 7) where 2^e <= |x| < 2^(e+1)
    (e clamped at -126 below, the subnormal range); |x| / ulp < 2^8, so the
    rounding of that quotient in float64 is exact. Finite inputs only.
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.isfinite(x).all():
        raise ValueError("f64_to_bf16_bits: non-finite input")
    a = np.abs(x)
    _, e = np.frexp(a)                     # a = f * 2^e with 0.5 <= f < 1, so 2^(e-1) <= a
    e = np.maximum(e - 1, -126)
    ulp = np.ldexp(1.0, e - 7)
    r = np.rint(a / ulp) * ulp             # np.rint rounds half to even
    v = np.where(np.signbit(x), -r, r).astype(np.float32)   # exact: r is a bf16 value
    return (v.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
