"""Seeded inputs for the shared-prefix prefill (one prompt per GRPO group).

Layout produced (the one the library consumes):

* packed prompt tokens: group ``g`` owns rows ``prefix_offs[g] .. prefix_offs[g+1]-1``
  of ``q [T][Hq][d]`` and ``k, v [T][Hkv][d]`` (bf16 bit patterns as uint16),
  ``prefix_offs[g+1] - prefix_offs[g] = prefix_lens[g]``;
* ``prefix_block_table [G][max_prefix_pages]`` (int32), each group's pages drawn
  from a random permutation of the pool, unused entries 0;
* empty pools ``[num_pages][Hkv][ps][d]`` filled with the NaN poison (bf16
  0x7FC0, fp8 0x7F) so rows that are never written stay recognisable, and for
  fp8 the scales filled with -1.

Draw order from ``default_rng(seed)``: prompt lengths (given or drawn), the
physical-page permutation, q, k, v (fp32 N(0, 1), K times ``k_mult``, rounded to
nearest-even bf16). Nothing here computes attention.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from .gen import BF16_POISON, FP8_POISON, _to_bf16_bits


@dataclass
class PrefillWorkload:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    kv_dtype: str
    prefix_lens: np.ndarray        # [G] int32
    prefix_offs: np.ndarray        # [G+1] int32
    prefix_block_table: np.ndarray  # [G][max_prefix_pages] int32
    q: np.ndarray                  # [T][Hq][d] uint16
    k: np.ndarray                  # [T][Hkv][d] uint16
    v: np.ndarray
    k_pages: np.ndarray            # [num_pages][Hkv][ps][d] uint16 or uint8 (poison)
    v_pages: np.ndarray
    k_scale: Optional[np.ndarray]  # [num_pages][Hkv] float32 (fp8 only)
    v_scale: Optional[np.ndarray]
    softmax_scale: float

    @property
    def num_groups(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.prefix_offs[-1])

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])


def make_prefill_workload(*, num_q_heads: int, num_kv_heads: int, head_dim: int,
                          prefix_lens: Sequence[int], seed: int, kv_dtype: str = "bf16",
                          page_size: int = 16, k_mult: float = 1.0, spare_pages: int = 3) -> PrefillWorkload:
    rng = np.random.default_rng(seed)
    P = np.asarray(prefix_lens, dtype=np.int32)
    G = int(P.shape[0])
    offs = np.zeros(G + 1, dtype=np.int32)
    offs[1:] = np.cumsum(P)
    T = int(offs[-1])
    pages_per = (P.astype(np.int64) + page_size - 1) // page_size
    mpp = max(1, int(pages_per.max(initial=0)))
    num_pages = int(pages_per.sum()) + spare_pages
    perm = rng.permutation(num_pages).astype(np.int32)
    pbt = np.zeros((G, mpp), dtype=np.int32)
    o = 0
    for g in range(G):
        n = int(pages_per[g])
        pbt[g, :n] = perm[o:o + n]
        o += n
    q = _to_bf16_bits(rng.standard_normal((T, num_q_heads, head_dim), dtype=np.float32))
    k = _to_bf16_bits(rng.standard_normal((T, num_kv_heads, head_dim), dtype=np.float32) * np.float32(k_mult))
    v = _to_bf16_bits(rng.standard_normal((T, num_kv_heads, head_dim), dtype=np.float32))
    shape = (num_pages, num_kv_heads, page_size, head_dim)
    if kv_dtype == "fp8":
        kp = np.full(shape, FP8_POISON, dtype=np.uint8)
        vp = np.full(shape, FP8_POISON, dtype=np.uint8)
        ks = np.full((num_pages, num_kv_heads), -1.0, dtype=np.float32)
        vs = np.full((num_pages, num_kv_heads), -1.0, dtype=np.float32)
    else:
        kp = np.full(shape, BF16_POISON, dtype=np.uint16)
        vp = np.full(shape, BF16_POISON, dtype=np.uint16)
        ks = vs = None
    return PrefillWorkload(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim=head_dim,
                           page_size=page_size, kv_dtype=kv_dtype, prefix_lens=P, prefix_offs=offs,
                           prefix_block_table=pbt, q=q, k=k, v=v, k_pages=kp, v_pages=vp,
                           k_scale=ks, v_scale=vs, softmax_scale=float(1.0 / np.sqrt(head_dim)))
