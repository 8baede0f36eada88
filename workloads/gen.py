"""Seeded generation of paged-KV decode-attention inputs.

Layout produced (the same one the library consumes):

* ``k_pages`` / ``v_pages``: ``[num_pages][Hkv][page_size][head_dim]``; bf16 bit
  patterns as ``uint16`` or OCP e4m3fn codes as ``uint8``.
* ``k_scale`` / ``v_scale``: fp32 ``[num_pages][Hkv]`` (fp8 only).
* Group layout: ``seq_to_group[S]``, ``prefix_lens[G]``,
  ``prefix_block_table[G][max_prefix_pages]``, ``resp_lens[S]``,
  ``resp_block_table[S][max_resp_pages]`` (int32). Unused table entries hold 0.
* ``q``: bf16 ``[S][Hq][head_dim]``; ``k_new`` / ``v_new``: bf16 ``[S][Hkv][head_dim]``.

``resp_lens`` counts the response tokens already cached. When ``append`` is set
the slot ``resp_lens[s]`` is still empty (it receives ``k_new``/``v_new``) and
attention afterwards spans ``resp_lens[s] + 1`` response keys.

Rows of a page beyond its valid length are filled with NaN (bf16 0x7FC0, fp8
code 0x7F) so that any read of a padding row poisons the result.

Random draws: one main ``numpy.random.default_rng(seed)`` stream draws, in this
order, prefix lengths, response lengths, live counts, the sequence-to-group
permutation, the physical-page permutation, q, and the new k/v. K/V page
contents come from independent streams ``default_rng([seed, 1, block])`` per
block of physical pages so they can be generated in parallel threads.

For fp8 pools the per-(page, kv-head) scale is ``amax / 448`` over the valid
rows (1.0 for an empty page) and the codes are torch's float8_e4m3fn cast of
``x / scale``; this only prepares inputs and is not the append path.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .configs import DecodeConfig

BF16_POISON = np.uint16(0x7FC0)
FP8_POISON = np.uint8(0x7F)
FP8_MAX = np.float32(448.0)
PAGE_BLOCK = 64  # physical pages per K/V generation stream


@dataclass
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    kv_dtype: str
    seq_to_group: np.ndarray
    prefix_lens: np.ndarray
    prefix_block_table: np.ndarray
    resp_lens: np.ndarray
    resp_block_table: np.ndarray
    k_pages: np.ndarray
    v_pages: np.ndarray
    k_scale: Optional[np.ndarray]
    v_scale: Optional[np.ndarray]
    q: np.ndarray
    k_new: Optional[np.ndarray]
    v_new: Optional[np.ndarray]
    softmax_scale: np.float32
    append: bool

    @property
    def num_seqs(self) -> int:
        return int(self.seq_to_group.shape[0])

    @property
    def num_groups(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])

    @property
    def attn_resp_lens(self) -> np.ndarray:
        """Response tokens that attention reads (after the append, if any)."""
        return self.resp_lens + (1 if self.append else 0)

    @property
    def kv_elem_bytes(self) -> int:
        return 1 if self.kv_dtype == "fp8" else 2


# The casts run on the generator's worker threads. Casting through torch in
# large pieces would start an OpenMP thread team per worker thread, and a
# process holding such teams cannot safely fork afterwards (the oracle's CPU
# baseline forks its workers from the process that generated the workload:
# the forked workers were seen to block forever in the unwinder's lock). So
# bf16 rounding is done in numpy, and the fp8 cast goes through torch in
# pieces below ATen's parallel grain (32768 elements), which run on the
# calling thread alone.
_CAST_PIECE = 16384


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, rounded to nearest even (NaN -> a quiet NaN of the same sign)."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    r = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x0040)).astype(np.uint16)
    return r


def _to_e4m3_codes(x: np.ndarray) -> np.ndarray:
    import torch
    f = np.ascontiguousarray(x, dtype=np.float32)
    flat = f.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint8)
    for i in range(0, flat.size, _CAST_PIECE):
        t = torch.from_numpy(flat[i:i + _CAST_PIECE]).to(torch.float8_e4m3fn)
        out[i:i + _CAST_PIECE] = t.view(torch.uint8).numpy()
    return out.reshape(f.shape)


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def make_workload(*, num_q_heads: int, num_kv_heads: int, head_dim: int,
                  seq_to_group, prefix_lens, resp_lens, seed: int,
                  append: bool = False, kv_dtype: str = "bf16", k_mult: float = 1.0,
                  page_size: int = 16, max_prefix_pages: Optional[int] = None,
                  max_resp_pages: Optional[int] = None, name: str = "custom",
                  rng: Optional[np.random.Generator] = None) -> Workload:
    """Lay out and fill a paged KV pool for the given group structure.

    ``rng`` continues an existing main stream (used by the config recipes);
    otherwise ``default_rng(seed)`` is started here.
    """
    assert kv_dtype in ("bf16", "fp8")
    assert num_q_heads % num_kv_heads == 0
    seq_to_group = np.ascontiguousarray(seq_to_group, dtype=np.int32)
    prefix_lens = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    resp_lens = np.ascontiguousarray(resp_lens, dtype=np.int32)
    S, G = seq_to_group.shape[0], prefix_lens.shape[0]
    ps = page_size
    rng = np.random.default_rng(seed) if rng is None else rng
    attn_resp = resp_lens + (1 if append else 0)

    n_pre = (prefix_lens + ps - 1) // ps
    n_rsp = (attn_resp + ps - 1) // ps
    mpp = int(max_prefix_pages if max_prefix_pages is not None else max(1, int(n_pre.max(initial=0))))
    mrp = int(max_resp_pages if max_resp_pages is not None else max(1, int(n_rsp.max(initial=0))))
    assert int(n_pre.max(initial=0)) <= mpp and int(n_rsp.max(initial=0)) <= mrp
    num_pages = int(n_pre.sum() + n_rsp.sum())
    perm = rng.permutation(max(num_pages, 1)).astype(np.int32)

    # Logical pages in order: group prefixes, then sequence responses.
    pbt = np.zeros((G, mpp), dtype=np.int32)
    rbt = np.zeros((S, mrp), dtype=np.int32)
    valid_rows = np.zeros(max(num_pages, 1), dtype=np.int32)  # indexed by physical page
    nxt = 0
    for g in range(G):
        for p in range(int(n_pre[g])):
            phys = perm[nxt]; nxt += 1
            pbt[g, p] = phys
            valid_rows[phys] = min(ps, int(prefix_lens[g]) - p * ps)
    for s in range(S):
        for p in range(int(n_rsp[s])):
            phys = perm[nxt]; nxt += 1
            rbt[s, p] = phys
            # Only already-cached rows are valid; the append slot stays poisoned.
            valid_rows[phys] = max(0, min(ps, int(resp_lens[s]) - p * ps))

    q = _to_bf16_bits(rng.standard_normal((S, num_q_heads, head_dim), dtype=np.float32))

    Hkv, d = num_kv_heads, head_dim
    is_fp8 = kv_dtype == "fp8"
    store = np.uint8 if is_fp8 else np.uint16
    k_pages = np.empty((max(num_pages, 1), Hkv, ps, d), dtype=store)
    v_pages = np.empty_like(k_pages)
    k_scale = np.ones((max(num_pages, 1), Hkv), dtype=np.float32) if is_fp8 else None
    v_scale = np.ones_like(k_scale) if is_fp8 else None
    row_idx = np.arange(ps, dtype=np.int32)

    def fill(block: int) -> None:
        lo = block * PAGE_BLOCK
        hi = min(lo + PAGE_BLOCK, k_pages.shape[0])
        brng = np.random.default_rng([seed, 1, block])
        shape = (hi - lo, Hkv, ps, d)
        kx = brng.standard_normal(shape, dtype=np.float32)
        if k_mult != 1.0:
            kx *= np.float32(k_mult)
        vx = brng.standard_normal(shape, dtype=np.float32)
        pad = row_idx[None, :] >= valid_rows[lo:hi, None]          # [n, ps]
        pad4 = np.broadcast_to(pad[:, None, :, None], shape)
        if not is_fp8:
            kb, vb = _to_bf16_bits(kx), _to_bf16_bits(vx)
            kb[pad4] = BF16_POISON
            vb[pad4] = BF16_POISON
            k_pages[lo:hi], v_pages[lo:hi] = kb, vb
            return
        for x, pages, scales in ((kx, k_pages, k_scale), (vx, v_pages, v_scale)):
            amax = np.where(pad4, np.float32(0), np.abs(x)).max(axis=(2, 3))  # [n, Hkv]
            sc = np.where(amax > 0, amax / FP8_MAX, np.float32(1.0)).astype(np.float32)
            codes = _to_e4m3_codes(x / sc[:, :, None, None])
            codes[pad4] = FP8_POISON
            pages[lo:hi], scales[lo:hi] = codes, sc

    nblocks = (k_pages.shape[0] + PAGE_BLOCK - 1) // PAGE_BLOCK
    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(nblocks)))

    k_new = v_new = None
    if append:
        k_new = _to_bf16_bits(np.float32(k_mult) * rng.standard_normal((S, Hkv, d), dtype=np.float32))
        v_new = _to_bf16_bits(rng.standard_normal((S, Hkv, d), dtype=np.float32))

    return Workload(name=name, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                    head_dim=head_dim, page_size=ps, kv_dtype=kv_dtype,
                    seq_to_group=seq_to_group, prefix_lens=prefix_lens, prefix_block_table=pbt,
                    resp_lens=resp_lens, resp_block_table=rbt, k_pages=k_pages, v_pages=v_pages,
                    k_scale=k_scale, v_scale=v_scale, q=q, k_new=k_new, v_new=v_new,
                    softmax_scale=np.float32(1.0 / np.sqrt(head_dim)), append=append)


def _draw_lengths(rng: np.random.Generator, spec: tuple, n: int) -> np.ndarray:
    kind = spec[0]
    if kind == "fixed":
        return np.full(n, spec[1], dtype=np.int32)
    if kind == "uniform":  # inclusive integer bounds
        return rng.integers(spec[1], spec[2], size=n, endpoint=True).astype(np.int32)
    if kind == "lognormal":  # median, sigma, cap; round half to even
        median, sigma, cap = spec[1], spec[2], spec[3]
        x = np.exp(rng.normal(np.log(median), sigma, size=n))
        return np.minimum(cap, np.rint(x)).astype(np.int32)
    raise ValueError(spec)


def _draw_live(rng: np.random.Generator, spec: tuple, groups: int) -> np.ndarray:
    """Live members per group: uniform counts, then +-1 on random groups until the total fits."""
    _, lo, hi, total = spec
    live = rng.integers(lo, hi, size=groups, endpoint=True).astype(np.int64)
    while live.sum() != total:
        g = int(rng.integers(0, groups))
        if live.sum() > total and live[g] > lo:
            live[g] -= 1
        elif live.sum() < total and live[g] < hi:
            live[g] += 1
    return live.astype(np.int32)


def make_config_workload(cfg: DecodeConfig, seed: Optional[int] = None) -> Workload:
    """Build one of the numbered workloads with the draw order documented above."""
    seed = cfg.seed if seed is None else int(seed)
    rng = np.random.default_rng(seed)
    G = cfg.groups
    prefix_lens = _draw_lengths(rng, cfg.prefix, G)
    if cfg.live is not None:
        n_seq = cfg.live[3]
    else:
        n_seq = G * cfg.group_size
    resp_lens = _draw_lengths(rng, cfg.resp, n_seq)
    if cfg.live is not None:
        live = _draw_live(rng, cfg.live, G)
    else:
        live = np.full(G, cfg.group_size, dtype=np.int32)
    seq_to_group = np.repeat(np.arange(G, dtype=np.int32), live)
    if cfg.random_group_map:
        seq_to_group = seq_to_group[rng.permutation(n_seq)]
    ps = cfg.page_size
    return make_workload(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads,
                         head_dim=cfg.head_dim, seq_to_group=seq_to_group,
                         prefix_lens=prefix_lens, resp_lens=resp_lens, seed=seed,
                         append=cfg.append, kv_dtype=cfg.kv_dtype, k_mult=cfg.k_mult,
                         page_size=ps, max_prefix_pages=(cfg.max_prefix + ps - 1) // ps,
                         max_resp_pages=(cfg.max_resp + ps - 1) // ps,
                         name=f"config{cfg.cid}", rng=rng)
