"""GPU parity of the decode step's pre-attention side through the C ABI.

q (and the optional k copy) is compared with the fp64 oracle's correctly
rounded bf16 bits: every element within one bf16 ulp, and all but a tiny
fraction bit-identical (the kernel also computes in fp64 and rounds once).
The pool after the append is compared byte for byte (codes and scales) with
the pure oracle: the append of the oracle's own rotated k and of v. Only the
slots of a (sequence, kv-head) whose kernel k differs from the oracle's k by
its one allowed ulp are named exceptions; they are listed, and there the pool
must hold the append of the kernel's k instead. End-to-end
cases run the whole decode step (prep, then attention over the advanced
lengths) at the frontier operating point of 2 groups x 8 samples and compare
it with the oracle's attention at the usual tolerances.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import compare
from workloads import make_qkprep_inputs, make_workload

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _ulps(a, b):
    """Distance in bf16 ulps between two bit arrays (signed zeros are equal)."""
    def ordered(x):
        m = (x & 0x7FFF).astype(np.int64)
        return np.where(x & 0x8000, -m, m)
    return np.abs(ordered(a) - ordered(b))


def _check_bits(got, ref, label):
    d = _ulps(got, ref)
    exact = float((d == 0).mean()) if d.size else 1.0
    assert d.max(initial=0) <= 1, f"{label}: max ulp distance {d.max()}"
    assert exact >= 0.9999, f"{label}: only {exact:.6f} bit-identical"


def _pool_bytes(b, kv_dtype):
    view = (lambda t: _bits(t)) if kv_dtype == "bf16" else (lambda t: t.cpu().numpy())
    out = [view(b.k_pages), view(b.v_pages)]
    if kv_dtype == "fp8":
        out += [b.k_scale.cpu().numpy(), b.v_scale.cpu().numpy()]
    return out


def _setup(S_groups, prefix_lens, resp_lens, Hq, Hkv, d, kv_dtype, seed, proj_scale=1.0, k_mult=1.0):
    import paper_2606_26997_amd as rp
    wl = make_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, seq_to_group=S_groups,
                       prefix_lens=prefix_lens, resp_lens=resp_lens, seed=seed, append=True, kv_dtype=kv_dtype,
                       k_mult=k_mult)
    x = make_qkprep_inputs(num_seqs=wl.num_seqs, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, seed=seed + 1,
                           scale=proj_scale)
    b = rp.DeviceBatch.from_workload(wl)
    return wl, x, b


def _oracle_prep(wl, x, resp_lens=None):
    rl = wl.resp_lens if resp_lens is None else resp_lens
    pos = oracle.decode_positions(wl.seq_to_group, wl.prefix_lens, rl)
    qb, kb, _, _ = oracle.qk_prep(q_in=x.q_in, k_in=x.k_in, q_norm_w=x.q_norm_w, k_norm_w=x.k_norm_w, positions=pos)
    return qb, kb


def _oracle_pool(wl, x, k_bits, seqs=None):
    """Append oracle of ``k_bits`` and v (only for sequences ``seqs``, default all)."""
    idx = np.arange(wl.num_seqs) if seqs is None else np.asarray(seqs)
    return oracle.kv_append(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale, v_scale=wl.v_scale,
                            kv_dtype=wl.kv_dtype, page_size=16, resp_lens=wl.resp_lens[idx],
                            resp_block_table=wl.resp_block_table[idx], k_new=k_bits[idx], v_new=x.v_in[idx])


def _check_pool(b, wl, x, k_gpu, k_ref, label, seqs=None):
    """The pool after the kernel's append against the pure oracle (its own k). A (sequence, kv-head)
    whose kernel k is one ulp off the oracle's in some element (allowed by the k check) is a named
    exception: there the k slot (bf16: the row; fp8: the whole (page, kv-head) block and its scale,
    which that row's amax may move) must equal the append of the kernel's k."""
    dt = wl.kv_dtype
    idx = np.arange(wl.num_seqs) if seqs is None else np.asarray(seqs)
    ref = [np.array(a, copy=True) for a in _oracle_pool(wl, x, k_ref, seqs) if a is not None]
    off = np.argwhere((k_gpu[idx] != k_ref[idx]).any(axis=2))      # rows of idx, kv-head
    if off.size:
        print(f"[case] {label}: k differs by one ulp at (sequence, kv-head) {[(int(idx[i]), int(h)) for i, h in off]}",
              flush=True)
        alt = [a for a in _oracle_pool(wl, x, k_gpu, seqs) if a is not None]
        for i, h in off:
            s = int(idx[i])
            t = int(wl.resp_lens[s])
            page = int(wl.resp_block_table[s][t // 16])
            if dt == "bf16":
                ref[0][page, h, t % 16] = alt[0][page, h, t % 16]
            else:
                ref[0][page, h] = alt[0][page, h]
                ref[2][page, h] = alt[2][page, h]
    got = _pool_bytes(b, dt)
    for g, r, what in zip(got, ref, ("k pages", "v pages", "k scales", "v scales")):
        np.testing.assert_array_equal(g, r, err_msg=f"{label}: {what}")
    return got


CASES = [
    # name, seq_to_group, prefix_lens, resp_lens, Hq, Hkv, d, kv dtype, projection scale, k_mult
    ("ragged-d128", [0, 0, 1, 1, 1, 2, 2], [0, 17, 1000], [0, 15, 16, 31, 1, 47, 300], 16, 8, 128, "bf16", 1.0, 1.0),
    ("ragged-d64", [0, 1, 1, 0], [33, 2], [5, 0, 64, 9], 4, 2, 64, "bf16", 1.0, 1.0),
    ("mha-d64", [0, 0, 0], [12], [3, 16, 17], 4, 4, 64, "bf16", 1.0, 1.0),
    ("fp8-requant", [0, 0, 1, 1, 1], [20, 40], [0, 5, 15, 16, 33], 16, 8, 128, "fp8", 4.0, 0.25),
    ("fp8-keep", [0, 0, 1, 1], [20, 40], [3, 7, 9, 30], 16, 8, 128, "fp8", 0.25, 8.0),
    ("fp8-d64", [0, 1, 0, 1], [8, 100], [1, 2, 17, 63], 8, 2, 64, "fp8", 2.0, 0.5),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_qk_prep_and_append(case):
    name, s2g, P, R, Hq, Hkv, d, dt, sc, km = case
    _say(f"qk prep {name}")
    wl, x, b = _setup(s2g, P, R, Hq, Hkv, d, dt, seed=len(name) * 7, proj_scale=sc, k_mult=km)
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w, keep_k=True)
    b.qk_prep()
    torch.cuda.synchronize()
    qb, kb = _oracle_prep(wl, x)
    _check_bits(_bits(b.q), qb, f"{name} q")
    k_gpu = _bits(b.k_out)
    _check_bits(k_gpu, kb, f"{name} k")
    got = _check_pool(b, wl, x, k_gpu, kb, name)
    if dt == "fp8":
        # The case exercises the scale branch it is named for on rows r > 0.
        raised = []
        for s in range(wl.num_seqs):
            t = int(wl.resp_lens[s])
            if t % 16:
                page = int(wl.resp_block_table[s][t // 16])
                raised += list(got[2][page] > wl.k_scale[page]) + list(got[3][page] > wl.v_scale[page])
        assert raised and (any(raised) if name != "fp8-keep" else not any(raised)), name
    # Same call again: the append is idempotent and q is recomputed identically.
    q1 = _bits(b.q).copy()
    b.qk_prep()
    torch.cuda.synchronize()
    assert np.array_equal(_bits(b.q), q1)
    for g, r in zip(_pool_bytes(b, dt), got):
        assert np.array_equal(g, r), name


def test_qk_prep_in_place_and_without_k_copy():
    import paper_2606_26997_amd as rp
    _say("qk prep in place")
    wl, x, b = _setup([0, 0, 1], [64, 5], [2, 17, 33], 16, 8, 128, "bf16", seed=21)
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w, keep_k=False)
    q = b.q_in  # q_out aliases q_in
    rp.decode_qk_prep(b.kv, b.append_layout, q, b.k_in, b.v_in, b.q_norm_w, b.k_norm_w, q, None)
    torch.cuda.synchronize()
    qb, kb = _oracle_prep(wl, x)
    _check_bits(_bits(q), qb, "in-place q")
    # Without k_out the rotated k is only visible in the pool (bf16: the slot rows).
    kp = _bits(b.k_pages)
    for s in range(wl.num_seqs):
        t = int(wl.resp_lens[s])
        page = int(wl.resp_block_table[s][t // 16])
        _check_bits(kp[page, :, t % 16], kb[s], f"pool k row of sequence {s}")


def test_qk_prep_slot_outside_table_gets_q_but_no_append():
    _say("qk prep slot outside the table")
    wl, x, b = _setup([0, 0, 0], [16], [4, 20, 31], 8, 2, 64, "bf16", seed=5)
    mrp = wl.resp_block_table.shape[1]
    rl = wl.resp_lens.copy()
    rl[1] = mrp * 16                      # one past the table: no slot
    b.resp_lens.copy_(torch.from_numpy(rl))
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w, keep_k=True)
    b.qk_prep()
    torch.cuda.synchronize()
    qb, kb = _oracle_prep(wl, x, resp_lens=rl)
    _check_bits(_bits(b.q), qb, "q")
    _check_bits(_bits(b.k_out), kb, "k")
    _check_pool(b, wl, x, _bits(b.k_out), kb, "slot outside the table", seqs=[0, 2])


@pytest.mark.parametrize("S", [1100, 4096])
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_qk_prep_large_batch_one_block_per_sequence(kv_dtype, S):
    # From 1024 sequences on, one block covers all heads of a sequence; 4096
    # sequences of one response page each is the prep-only launch of the
    # frontier bench.
    _say(f"qk prep {S} sequences {kv_dtype}")
    rng = np.random.default_rng(99 + S)
    G = S // 8
    s2g = rng.integers(0, G, S)
    wl, x, b = _setup(s2g, rng.integers(0, 64, G), rng.integers(0, 16 if S == 4096 else 40, S), 16, 8, 128,
                      kv_dtype, seed=31)
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w, keep_k=True)
    b.qk_prep()
    torch.cuda.synchronize()
    qb, kb = _oracle_prep(wl, x)
    _check_bits(_bits(b.q), qb, "q")
    k_gpu = _bits(b.k_out)
    _check_bits(k_gpu, kb, "k")
    _check_pool(b, wl, x, k_gpu, kb, f"{S} sequences {kv_dtype}")


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_decode_step_at_frontier_operating_point(kv_dtype):
    # Two groups of eight live samples (the frontier batch of 16 sequences):
    # 1k-token prompts, ragged responses up to ~3.5k tokens.
    _say(f"decode step 2x8 {kv_dtype}")
    rng = np.random.default_rng(7)
    s2g = np.repeat([0, 1], 8)
    R = rng.integers(1, 3500, 16)
    wl, x, b = _setup(s2g, [1024, 977], R, 16, 8, 128, kv_dtype, seed=41)
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w)
    b.decode_step()
    torch.cuda.synchronize()
    qb, kb, pool = oracle.decode_step_prep(q_in=x.q_in, k_in=x.k_in, v_in=x.v_in, q_norm_w=x.q_norm_w,
                                           k_norm_w=x.k_norm_w, k_pages=wl.k_pages, v_pages=wl.v_pages,
                                           k_scale=wl.k_scale, v_scale=wl.v_scale, kv_dtype=kv_dtype,
                                           page_size=16, seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                                           resp_lens=wl.resp_lens, resp_block_table=wl.resp_block_table)
    _check_bits(_bits(b.q), qb, "q")
    kp, vp, ks, vs = pool
    ref_out, ref_lse = oracle.decode_attention(k_pages=kp, v_pages=vp, k_scale=ks, v_scale=vs, kv_dtype=kv_dtype,
                                               page_size=16, seq_to_group=wl.seq_to_group,
                                               prefix_lens=wl.prefix_lens, prefix_block_table=wl.prefix_block_table,
                                               resp_lens=wl.resp_lens + 1, resp_block_table=wl.resp_block_table,
                                               q=qb, softmax_scale=wl.softmax_scale)
    out = b.out.float().cpu().numpy().astype(np.float64)
    lse = b.lse.cpu().numpy().astype(np.float64)
    compare(out, lse, ref_out, ref_lse, kv_dtype, label=f"decode step {kv_dtype}")


FUSED = [
    # name, seq_to_group, prefix_lens, response lengths (seeded draw), Hq, Hkv, d, kv dtype
    ("frontier-2x8", np.repeat([0, 1], 8), [512, 300], (0, 6017), 16, 8, 128, "bf16"),
    ("fp8-5", [0, 0, 1, 1, 1], [33, 200], (0, 700), 16, 8, 128, "fp8"),
    ("d64-64-seqs", np.arange(64) % 5, [16, 0, 77, 130, 3], (0, 900), 8, 2, 64, "bf16"),
    ("two-launches-100", np.arange(100) // 10, [100] * 10, (0, 1200), 16, 8, 128, "bf16"),
]


@pytest.mark.parametrize("case", FUSED, ids=[c[0] for c in FUSED])
def test_prep_plan_call_equals_prep_then_plan(case):
    """rp_decode_qk_prep_plan (one launch up to 64 sequences) leaves the same q, pool bytes and plan as
    rp_decode_qk_prep followed by rp_plan over the advanced lengths; attention on that plan matches the
    pure oracle's decode step."""
    name, s2g, P, (lo, hi), Hq, Hkv, d, dt = case
    _say(f"prep+plan {name}")
    rng = np.random.default_rng(len(name))
    R = rng.integers(lo, hi, len(s2g))
    wl, x, ref = _setup(s2g, P, R, Hq, Hkv, d, dt, seed=len(name) * 3)
    import paper_2606_26997_amd as rp
    one = rp.DeviceBatch.from_workload(wl)
    for b in (ref, one):
        b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w, keep_k=True)
    ref.qk_prep()
    ref.plan()
    one.workspace.fill_(255)
    one.qk_prep_plan()
    torch.cuda.synchronize()
    assert np.array_equal(_bits(one.q), _bits(ref.q)) and np.array_equal(_bits(one.k_out), _bits(ref.k_out))
    for g, r in zip(_pool_bytes(one, dt), _pool_bytes(ref, dt)):
        assert np.array_equal(g, r), name
    p1, p2 = one.plan_contents(), ref.plan_contents()
    assert np.array_equal(p1["hdr"][:4], p2["hdr"][:4]), name          # the header's used slots
    for key in ("grp_off", "prefix_items", "seq_parts"):
        assert np.array_equal(p1[key], p2[key]), (name, key)
    # Members within a group, and last pieces of equal size, may come in any order (the plan contract).
    off = p1["grp_off"]
    for g in range(len(off) - 1):
        assert sorted(p1["grp_members"][off[g]:off[g + 1]]) == sorted(p2["grp_members"][off[g]:off[g + 1]])
    nb = int(p1["hdr"][2])
    assert np.array_equal(p1["resp_items"][:nb], p2["resp_items"][:nb]), name
    assert sorted(map(tuple, p1["resp_items"][nb:])) == sorted(map(tuple, p2["resp_items"][nb:])), name
    for b in (ref, one):
        b.attn_parts()
        b.combine_parts()
    torch.cuda.synchronize()
    # Same pieces, so the same partial results and the same merge: bit for bit.
    assert torch.equal(one.out.view(torch.int16), ref.out.view(torch.int16))
    assert torch.equal(one.lse.view(torch.int32), ref.lse.view(torch.int32))
    qb, _, pool = oracle.decode_step_prep(q_in=x.q_in, k_in=x.k_in, v_in=x.v_in, q_norm_w=x.q_norm_w,
                                          k_norm_w=x.k_norm_w, k_pages=wl.k_pages, v_pages=wl.v_pages,
                                          k_scale=wl.k_scale, v_scale=wl.v_scale, kv_dtype=dt, page_size=16,
                                          seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                                          resp_lens=wl.resp_lens, resp_block_table=wl.resp_block_table)
    kp, vp, ks, vs = pool
    ref_out, ref_lse = oracle.decode_attention(k_pages=kp, v_pages=vp, k_scale=ks, v_scale=vs, kv_dtype=dt,
                                               page_size=16, seq_to_group=wl.seq_to_group,
                                               prefix_lens=wl.prefix_lens, prefix_block_table=wl.prefix_block_table,
                                               resp_lens=wl.resp_lens + 1, resp_block_table=wl.resp_block_table,
                                               q=qb, softmax_scale=wl.softmax_scale)
    out = one.out.float().cpu().numpy().astype(np.float64)
    lse = one.lse.cpu().numpy().astype(np.float64)
    compare(out, lse, ref_out, ref_lse, dt, label=f"prep+plan {name}")
