"""GPU: the work plan read back and checked against its contract, exactly.

The planner's output is integer data, so every field is compared bit for bit
with what the contract in include/rp.h fixes: prefix work items, member lists,
the piece length B, every response cut into B-page pieces plus a shorter last
piece, B-page pieces first in sequence order, then last pieces by decreasing
page count, each item's slot, and the part count per query row. Layouts are synthetic (lengths drawn like the benchmark workloads,
block tables random over a small pool); the plan never reads K/V.
"""
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

PAGE, PREFIX_CHUNK = 16, 16
B_STEP, B_CHOICES, UNITS_PER_CU = 32, 4, 6
HKV = 8


SMALL_B, SMALL_CAPACITY = 16, 1 << 17


def piece_pages(pages, hkv, cus, table_width):
    """The contract's piece length: the multiple of 32 pages nearest to W / (32 * 6 * compute units),
    W = response pages x kv-heads, clamped to 32..128; 16 pages instead when W is below three quarters of
    that step and the workspace was sized for 16-page pieces (sequences x table width x kv-heads <= 2^17)."""
    W = int(pages.sum()) * hkv
    unit = B_STEP * UNITS_PER_CU * cus
    B = B_STEP * min(max((W + unit // 2) // unit, 1), B_CHOICES)
    if 4 * W < 3 * unit and len(pages) * table_width * hkv <= SMALL_CAPACITY:
        B = SMALL_B
    return B


def cdiv(a, b):
    return -(-a // b)


def make_batch(s2g, prefix_lens, resp_lens, num_groups, seed, num_pages=97, Hq=16, Hkv=8, d=128):
    import paper_2606_26997_amd as rp
    rng = np.random.default_rng(seed)
    s2g = np.asarray(s2g, np.int32)
    P = np.asarray(prefix_lens, np.int32)
    L = np.asarray(resp_lens, np.int32)
    mpp = max(1, cdiv(int(P.max(initial=0)), PAGE))
    mrp = max(1, cdiv(int(L.max(initial=0)), PAGE))
    pbt = rng.integers(0, num_pages, size=(num_groups, mpp), dtype=np.int32)
    rbt = rng.integers(0, num_pages, size=(len(s2g), mrp), dtype=np.int32)
    pool = torch.zeros((num_pages, Hkv, PAGE, d), dtype=torch.bfloat16)
    q = torch.zeros((len(s2g), Hq, d), dtype=torch.bfloat16)
    b = rp.DeviceBatch(k_pages=pool, v_pages=pool, k_scale=None, v_scale=None, seq_to_group=s2g,
                       prefix_lens=P, prefix_block_table=pbt, resp_lens=L, resp_block_table=rbt, q=q,
                       num_q_heads=Hq, softmax_scale=0.1)
    return b, rbt


def check_plan(b, s2g, P, L, rbt, G):
    s2g, P, L = np.asarray(s2g), np.asarray(P, np.int64), np.asarray(L, np.int64)
    S = len(s2g)
    b.plan()
    got = b.plan_contents()
    hdr = got["hdr"]
    pages = cdiv(L, PAGE)
    B = piece_pages(pages, HKV, torch.cuda.get_device_properties(0).multi_processor_count, rbt.shape[1])
    assert hdr[3] == B
    live = np.bincount(s2g, minlength=G)
    npc = cdiv(cdiv(P, PAGE), PREFIX_CHUNK)

    want_prefix = [(g, c) for g in range(G) if live[g] > 0 for c in range(npc[g])]
    assert hdr[0] == len(want_prefix)
    assert [tuple(x) for x in got["prefix_items"]] == want_prefix

    assert np.array_equal(got["grp_off"], np.concatenate([[0], np.cumsum(live)]))
    for g in np.flatnonzero(live):
        m = got["grp_members"][got["grp_off"][g]:got["grp_off"][g + 1]]
        assert sorted(m.tolist()) == np.flatnonzero(s2g == g).tolist(), g

    nfull = pages // B
    ragged = pages % B != 0
    assert hdr[2] == nfull.sum() and hdr[1] == nfull.sum() + ragged.sum()
    items = got["resp_items"]
    want_big = [(s, c * B, min(B * PAGE, L[s] - c * B * PAGE), npc[s2g[s]] + c)
                for s in range(S) for c in range(nfull[s])]
    assert [tuple(x) for x in items[:hdr[2]]] == want_big
    tail = items[hdr[2]:]
    want_tail = sorted((s, nfull[s] * B, L[s] - nfull[s] * B * PAGE, npc[s2g[s]] + nfull[s])
                       for s in np.flatnonzero(ragged))
    assert sorted(tuple(x) for x in tail) == want_tail
    tail_pages = cdiv(tail[:, 2].astype(np.int64), PAGE)
    assert np.all(np.diff(tail_pages) <= 0), "last pieces must come by decreasing page count"
    assert np.all(tail_pages < B)
    assert np.array_equal(got["seq_parts"], npc[s2g] + cdiv(pages, B))
    return B


def _case(name):
    rng = np.random.default_rng(sum(map(ord, name)))
    if name == "qwen-layer-uniform":        # 32 groups x 8, prefix U[64,512], resp U[0,4096]
        G, S = 32, 256
        s2g = np.repeat(np.arange(G), 8)
        P, L = rng.integers(64, 513, G), rng.integers(0, 4097, S)
    elif name == "lognormal-tail":          # 64 x 16, lognormal(1500, 0.9) capped at 8193
        G, S = 64, 1024
        s2g = np.repeat(np.arange(G), 16)
        P = np.full(G, 256)
        L = np.minimum(np.exp(rng.normal(np.log(1500), 0.9, S)).astype(np.int64), 8192) + 1
    elif name == "frontier-random-map":     # 512 live of 128 groups, resp U[0,16384]
        G, S = 128, 512
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(128, 1025, G), rng.integers(0, 16385, S)
    elif name == "long-context":            # 16 x 16, resp U[8192, 32768] + 1
        G, S = 16, 256
        s2g = np.repeat(np.arange(G), 16)
        P, L = np.full(G, 256), rng.integers(8192, 32769, S) + 1
    elif name == "many-sequences":          # several planner passes
        G, S = 4096, 9000
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(0, 300, G), rng.integers(0, 3000, S)
    elif name == "many-pieces":             # several item rounds in one pass
        G, S = 500, 4000
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(0, 100, G), rng.integers(2000, 4000, S)
    elif name == "frontier-dispatch-16":    # 2 groups x 8 live sequences (the paper's F_w = 2, K = 8)
        G, S = 2, 16
        s2g = np.repeat(np.arange(G), 8)
        P, L = rng.integers(64, 513, G), rng.integers(3000, 4001, S)
    elif name == "frontier-dispatch-64":    # 8 groups x 8 live sequences, ~190 pages each
        G, S = 8, 64
        s2g = np.repeat(np.arange(G), 8)
        P, L = rng.integers(64, 513, G), rng.integers(2500, 3501, S)
    elif name == "frontier-dispatch-64-long":  # 8 groups x 8 live sequences, ~256 pages each
        G, S = 8, 64
        s2g = np.repeat(np.arange(G), 8)
        P, L = rng.integers(64, 513, G), rng.integers(3800, 4401, S)
    elif name == "few-long-sequences":      # long responses, but only 8 of them
        G, S = 2, 8
        s2g = np.repeat(np.arange(G), 4)
        P, L = np.array([100, 300]), rng.integers(6000, 9000, S)
    elif name == "empty-and-idle-groups":   # zero lengths, groups without members
        G, S = 6, 5
        s2g = np.array([0, 0, 3, 3, 5])
        P, L = np.array([0, 17, 300, 0, 5, 16]), np.array([0, 512, 0, 513, 1])
    elif name == "small-many-groups":       # single-wave planner, groups beyond the first 64 live
        G, S = 300, 40
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(0, 700, G), rng.integers(0, 2000, S)
    elif name == "small-equal-lengths":     # 64 sequences in 64 groups, ties among the last pieces
        G, S = 64, 64
        s2g = rng.permutation(S)
        P, L = rng.integers(1, 200, G), np.full(S, 1000)
    elif name == "single-sequence":
        G, S = 1, 1
        s2g = np.zeros(1, int)
        P, L = np.array([33]), np.array([4097])
    elif name == "small-all-empty":         # no prefix, no response tokens
        G, S = 3, 10
        s2g = rng.integers(0, G, S)
        P, L = np.zeros(G, int), np.zeros(S, int)
    elif name == "mid-65":                 # just past the single-wave planner's 64 sequences
        G, S = 9, 65
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(0, 600, G), rng.integers(0, 5000, S)
    elif name == "mid-100-many-groups":    # general planner, many groups without members
        G, S = 300, 100
        s2g = rng.integers(0, G, S)
        P, L = rng.integers(0, 700, G), rng.integers(0, 3000, S)
    elif name == "mid-256-equal-lengths":  # ties among all the last pieces
        G, S = 32, 256
        s2g = rng.permutation(np.repeat(np.arange(G), 8))
        P, L = rng.integers(1, 200, G), np.full(S, 1000)
    elif name == "mid-200-all-empty":      # no prefix, no response tokens
        G, S = 7, 200
        s2g = rng.integers(0, G, S)
        P, L = np.zeros(G, int), np.zeros(S, int)
    else:
        raise KeyError(name)
    return G, s2g, P, L


CASES = ["qwen-layer-uniform", "lognormal-tail", "frontier-random-map", "long-context", "many-sequences",
         "many-pieces", "frontier-dispatch-16", "frontier-dispatch-64", "frontier-dispatch-64-long",
         "few-long-sequences", "empty-and-idle-groups", "small-many-groups", "small-equal-lengths",
         "single-sequence", "small-all-empty", "mid-65", "mid-100-many-groups", "mid-256-equal-lengths",
         "mid-200-all-empty"]


@pytest.mark.parametrize("name", CASES)
def test_plan_matches_its_contract(name):
    print(f"[case] plan {name}", flush=True)
    sys.stdout.flush()
    G, s2g, P, L = _case(name)
    b, rbt = make_batch(s2g, P, L, G, seed=len(name))
    B = check_plan(b, s2g, P, L, rbt, G)
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:   # MI355X: every candidate B occurs
        want = {"frontier-dispatch-16": 16, "few-long-sequences": 16, "empty-and-idle-groups": 16,
                "frontier-dispatch-64": 64, "frontier-dispatch-64-long": 96, "small-many-groups": 16,
                "small-equal-lengths": 16, "single-sequence": 16, "small-all-empty": 16, "mid-65": 64,
                "mid-100-many-groups": 32, "mid-256-equal-lengths": 96, "mid-200-all-empty": 16}.get(name, 128)
        assert B == want, (name, B)
    # A second plan into the same workspace gives the same B-page items.
    check_plan(b, s2g, P, L, rbt, G)
