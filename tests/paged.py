"""Test helpers: scatter dense per-sequence K/V into a paged pool (no attention math).

These build paged layouts from dense arrays so the oracle's gather can be checked
against library attention on the dense arrays. They are independent of both the
oracle and the HIP library.
"""
import numpy as np
import torch

from workloads.gen import Workload


def bf16_bits(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_value(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).double().numpy()


def paged_from_dense(prefix_k, prefix_v, resp_k, resp_v, seq_to_group, q_bits, *, num_kv_heads,
                     page_size=16, seed=0, softmax_scale=None, pad_pages=0, poison=0x7FC0):
    """Build a bf16 Workload whose keys are exactly the given dense tokens.

    prefix_k[g]: [P_g][Hkv][d] bf16 bits; resp_k[s]: [L_s][Hkv][d] bf16 bits.
    Physical pages are a random permutation; padding rows hold ``poison``.
    """
    rng = np.random.default_rng(seed)
    G, S = len(prefix_k), len(resp_k)
    Hkv, d = num_kv_heads, q_bits.shape[2]
    ps = page_size
    chunks = []          # (owner kind, owner idx, page idx, k rows, v rows)
    for g in range(G):
        n = (len(prefix_k[g]) + ps - 1) // ps
        for p in range(n):
            chunks.append(("p", g, p, prefix_k[g][p * ps:(p + 1) * ps], prefix_v[g][p * ps:(p + 1) * ps]))
    for s in range(S):
        n = (len(resp_k[s]) + ps - 1) // ps
        for p in range(n):
            chunks.append(("r", s, p, resp_k[s][p * ps:(p + 1) * ps], resp_v[s][p * ps:(p + 1) * ps]))
    num_pages = len(chunks) + pad_pages
    perm = rng.permutation(max(num_pages, 1))
    kp = np.full((max(num_pages, 1), Hkv, ps, d), poison, dtype=np.uint16)
    vp = np.full_like(kp, poison)
    mpp = max(1, max((len(x) + ps - 1) // ps for x in prefix_k))
    mrp = max(1, max((len(x) + ps - 1) // ps for x in resp_k))
    pbt = np.zeros((G, mpp), np.int32)
    rbt = np.zeros((S, mrp), np.int32)
    for i, (kind, owner, p, kr, vr) in enumerate(chunks):
        phys = int(perm[i])
        (pbt if kind == "p" else rbt)[owner, p] = phys
        kp[phys, :, :len(kr), :] = np.transpose(kr, (1, 0, 2))
        vp[phys, :, :len(vr), :] = np.transpose(vr, (1, 0, 2))
    Hq = q_bits.shape[1]
    scale = np.float32(1.0 / np.sqrt(d)) if softmax_scale is None else np.float32(softmax_scale)
    return Workload(name="dense", num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, page_size=ps,
                    kv_dtype="bf16", seq_to_group=np.asarray(seq_to_group, np.int32),
                    prefix_lens=np.array([len(x) for x in prefix_k], np.int32),
                    prefix_block_table=pbt,
                    resp_lens=np.array([len(x) for x in resp_k], np.int32),
                    resp_block_table=rbt, k_pages=kp, v_pages=vp, k_scale=None, v_scale=None,
                    q=q_bits, k_new=None, v_new=None, softmax_scale=scale, append=False)


def random_dense(rng, *, S, G, Hq, Hkv, d, prefix_lens, resp_lens, seq_to_group=None):
    """Random bf16 dense prefix/response K, V and q (bit patterns)."""
    if seq_to_group is None:
        seq_to_group = np.arange(S) % G
    pk = [bf16_bits(rng.standard_normal((P, Hkv, d))) for P in prefix_lens]  # noqa: E501
    pv = [bf16_bits(rng.standard_normal((P, Hkv, d))) for P in prefix_lens]
    rk = [bf16_bits(rng.standard_normal((L, Hkv, d))) for L in resp_lens]
    rv = [bf16_bits(rng.standard_normal((L, Hkv, d))) for L in resp_lens]
    q = bf16_bits(rng.standard_normal((S, Hq, d)))
    return pk, pv, rk, rv, np.asarray(seq_to_group, np.int32), q


def dense_keys(pk, pv, rk, rv, seq_to_group, s):
    """Dense fp64 K, V [N][Hkv][d] of sequence s: its group's prefix, then its response."""
    g = int(seq_to_group[s])
    K = np.concatenate([bf16_value(pk[g]), bf16_value(rk[s])], axis=0)
    V = np.concatenate([bf16_value(pv[g]), bf16_value(rv[s])], axis=0)
    return K, V


def oracle_on(wl, seqs=None, resp_lens=None):
    from oracle import decode_attention
    return decode_attention(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale,
                            v_scale=wl.v_scale, kv_dtype=wl.kv_dtype, page_size=wl.page_size,
                            seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                            prefix_block_table=wl.prefix_block_table,
                            resp_lens=wl.resp_lens if resp_lens is None else resp_lens,
                            resp_block_table=wl.resp_block_table, q=wl.q,
                            softmax_scale=wl.softmax_scale, seqs=seqs)
