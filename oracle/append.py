"""Append one new token's K and V per sequence into its response pages.

The new token of sequence ``s`` goes to response slot ``t = resp_lens[s]`` (the
pre-append length): page ``resp_block_table[s][t // ps]``, row ``t % ps``, for
every kv-head. The lengths themselves are not changed; the caller advances them.

bf16 pools: the bf16 bit patterns are copied.

fp8 (OCP e4m3fn) pools keep one fp32 scale per (page, kv-head), separately for K
and for V. With ``x`` the new token's row for that head (bf16 widened to fp32),
``amax = max |x|`` and ``r = t % ps``, all in fp32 arithmetic:

* ``r == 0`` (first row of the page): ``scale = amax / 448``, or 1.0 when ``amax == 0``;
* ``r > 0`` and ``amax <= 448 * scale_old``: the scale is kept;
* ``r > 0`` otherwise: ``scale = amax / 448`` and rows ``0..r-1`` are requantised
  from their dequantised values ``decode(code) * scale_old``;
* the new row is stored as ``encode(x / scale)`` (round to nearest even, saturate
  at 448).
"""
import numpy as np

from .formats import bf16_to_f32, e4m3_encode, e4m3_to_f64

_F448 = np.float32(448.0)


def _append_fp8_row(codes, scales, page, h, r, x):
    amax = np.float32(np.abs(x).max())
    old = np.float32(scales[page, h])
    if r == 0:
        scale = amax / _F448 if amax > 0 else np.float32(1.0)
    elif amax <= _F448 * old:
        scale = old
    else:
        scale = amax / _F448
        prev = e4m3_to_f64(codes[page, h, :r, :]).astype(np.float32) * old
        codes[page, h, :r, :] = e4m3_encode(prev / scale)
    scale = np.float32(scale)
    codes[page, h, r, :] = e4m3_encode(x / scale)
    scales[page, h] = scale


def kv_append(*, k_pages, v_pages, k_scale, v_scale, kv_dtype, page_size,
              resp_lens, resp_block_table, k_new, v_new):
    """Return the post-append pool ``(k_pages, v_pages, k_scale, v_scale)`` as new arrays."""
    kp, vp = k_pages.copy(), v_pages.copy()
    ks = None if k_scale is None else k_scale.copy()
    vs = None if v_scale is None else v_scale.copy()
    S, Hkv, _ = k_new.shape
    for s in range(S):
        t = int(resp_lens[s])
        page = int(resp_block_table[s][t // page_size])
        r = t % page_size
        for h in range(Hkv):
            if kv_dtype == "fp8":
                _append_fp8_row(kp, ks, page, h, r, bf16_to_f32(k_new[s, h]))
                _append_fp8_row(vp, vs, page, h, r, bf16_to_f32(v_new[s, h]))
            else:
                kp[page, h, r, :] = k_new[s, h]
                vp[page, h, r, :] = v_new[s, h]
    return kp, vp, ks, vs


def append_for_workload(wl):
    """Post-append pool of a generated workload (which must carry ``k_new``/``v_new``)."""
    return kv_append(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale,
                     v_scale=wl.v_scale, kv_dtype=wl.kv_dtype, page_size=wl.page_size,
                     resp_lens=wl.resp_lens, resp_block_table=wl.resp_block_table,
                     k_new=wl.k_new, v_new=wl.v_new)
