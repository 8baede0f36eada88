"""Log-sum-exp merge of attention partials over disjoint key subsets.

If part ``i`` of a row is attention over key subset ``T_i`` with
``lse_i = log sum_{t in T_i} exp(s_t)`` and ``o_i = sum_{t in T_i} exp(s_t - lse_i) v_t``,
then over the union ``lse = log sum_i exp(lse_i)`` and
``out = sum_i exp(lse_i - lse) o_i``. A part with ``lse_i = -inf`` (no keys) adds
nothing; a row with no parts, or only empty ones, gives ``out = 0``, ``lse = -inf``.
"""
import numpy as np


def lse_combine(o_parts, lse_parts, row_part_offsets):
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    offs = np.asarray(row_part_offsets, dtype=np.int64)
    R = offs.shape[0] - 1
    d = o_parts.shape[1] if o_parts.ndim == 2 else 0
    out = np.zeros((R, d), dtype=np.float64)
    lse = np.full(R, -np.inf, dtype=np.float64)
    for r in range(R):
        a, b = int(offs[r]), int(offs[r + 1])
        if b <= a:
            continue
        l = lse_parts[a:b]
        keep = l > -np.inf              # an empty part contributes nothing, whatever its o
        if not keep.any():
            continue
        l, o = l[keep], o_parts[a:b][keep]
        m = l.max()
        total = m + np.log(np.exp(l - m).sum())
        out[r] = np.exp(l - total) @ o
        lse[r] = total
    return out, lse
