"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Inputs are seeded and synthetic; every case prints its name before running.
"""
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import compare, run_hip, run_oracle, run_oracle_all, to_host_out
from tests.paged import bf16_bits, paged_from_dense, random_dense
from workloads import CONFIGS, make_config_workload, make_workload

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def test_config1_full():
    _say("config1 full")
    wl = make_config_workload(CONFIGS[1])
    _, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle(wl)
    compare(out, lse, ref_out, ref_lse, "bf16", "config1")


RAGGED = [
    # (name, Hq, Hkv, d, seq_to_group, prefix_lens, resp_lens, kv_dtype)
    ("edges-d128", 16, 8, 128, [0, 0, 0, 1, 1, 2, 2, 2, 2], [17, 64, 130],
     [0, 1, 15, 16, 17, 255, 256, 257, 600], "bf16"),
    ("edges-d64", 4, 2, 64, [0, 1, 1, 0, 2], [1, 16, 33], [31, 0, 513, 16, 2], "bf16"),
    ("mha", 4, 4, 64, [0, 0, 1], [40, 3], [5, 70, 0], "bf16"),
    ("nrep4", 8, 2, 128, [0, 0, 0, 1], [48, 80], [10, 300, 0, 47], "bf16"),
    ("nrep8", 8, 1, 128, [0, 1, 0], [20, 70], [9, 129, 1], "bf16"),
    ("big-group-3-passes", 16, 8, 128, [0] * 20 + [1] * 3, [70, 18], list(range(0, 230, 10)), "bf16"),
    ("empty-keys", 4, 2, 64, [0, 1, 1], [0, 5], [0, 0, 3], "bf16"),
    ("no-prefix", 4, 2, 128, [0, 0], [0], [40, 1], "bf16"),
    ("fp8-edges", 16, 8, 128, [0, 0, 1, 1, 1], [33, 200], [0, 16, 17, 300, 513], "fp8"),
    ("fp8-d64-nrep4", 8, 2, 64, [0, 1, 0], [64, 9], [100, 31, 0], "fp8"),
    # Response lengths on both sides of 32-page piece boundaries.
    ("piece-edges-short", 4, 2, 64, [0] * 5 + [1] * 4, [20, 0],
     [497, 500, 511, 512, 513, 1008, 1009, 1023, 1024], "bf16"),
    # Lengths at the edges of 64-page multiples (32-page pieces: the batch is small).
    ("piece-edges-long", 4, 2, 64, [0, 0, 0, 1, 1, 1, 1], [100, 16],
     [4090, 4096, 4097, 8191, 8192, 1000, 12000], "bf16"),
]


@pytest.mark.parametrize("case", RAGGED, ids=[c[0] for c in RAGGED])
def test_ragged_shapes(case):
    name, Hq, Hkv, d, s2g, P, L, dt = case
    _say(name)
    wl = make_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, seq_to_group=s2g,
                       prefix_lens=P, resp_lens=L, seed=zlib.crc32(name.encode()) % 1000, kv_dtype=dt)
    _, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle(wl)
    compare(out, lse, ref_out, ref_lse, dt, name)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_random_group_map_many_groups(kv_dtype):
    _say(f"random map {kv_dtype}")
    rng = np.random.default_rng(77)
    G = 37
    s2g = rng.integers(0, G, size=150)
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=s2g,
                       prefix_lens=rng.integers(0, 300, size=G), resp_lens=rng.integers(0, 700, size=150),
                       seed=5, kv_dtype=kv_dtype)
    _, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle(wl)
    compare(out, lse, ref_out, ref_lse, kv_dtype, "random-map")


def test_more_sequences_than_the_planner_caches():
    # The planner keeps 8192 sequences' lengths in LDS and rereads the rest.
    _say("8500 sequences")
    rng = np.random.default_rng(91)
    S, G = 8500, 300
    s2g = rng.integers(0, G, size=S)
    wl = make_workload(num_q_heads=2, num_kv_heads=1, head_dim=64, seq_to_group=s2g,
                       prefix_lens=rng.integers(0, 40, size=G), resp_lens=rng.integers(0, 80, size=S),
                       seed=6)
    _, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle(wl)
    compare(out, lse, ref_out, ref_lse, "bf16", "8500-seqs")


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_append_bytes_match_oracle_then_attention(kv_dtype):
    _say(f"append {kv_dtype}")
    rng = np.random.default_rng(11)
    S = 40
    L = rng.integers(0, 200, size=S)
    L[:6] = [0, 15, 16, 31, 32, 47]
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.arange(S) // 8,
                       prefix_lens=[64, 100, 7, 16, 33], resp_lens=L, seed=9, append=True,
                       kv_dtype=kv_dtype)
    if kv_dtype == "fp8":  # make some appends grow the page scale (requantise path)
        wl.k_new[::3] = bf16_bits(oracle.bf16_to_f32(wl.k_new[::3]) * np.float32(40.0))
    batch, out, lse = run_hip(wl)
    ref_out, ref_lse, pool = run_oracle(wl)
    kp, vp, ks, vs = pool
    torch.cuda.synchronize()
    if kv_dtype == "fp8":
        assert np.array_equal(batch.k_pages.cpu().numpy(), kp)
        assert np.array_equal(batch.v_pages.cpu().numpy(), vp)
        assert np.array_equal(batch.k_scale.cpu().numpy(), ks)
        assert np.array_equal(batch.v_scale.cpu().numpy(), vs)
    else:
        assert np.array_equal(batch.k_pages.view(torch.int16).cpu().numpy().view(np.uint16), kp)
        assert np.array_equal(batch.v_pages.view(torch.int16).cpu().numpy().view(np.uint16), vp)
    compare(out, lse, ref_out, ref_lse, kv_dtype, f"append-{kv_dtype}")
    # The append is idempotent: a second step changes nothing.
    batch.step()
    out2, lse2 = to_host_out(batch)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_fp8_append_nan_element_takes_the_saturated_code():
    """A NaN element of an appended token does not enter the page scale's amax and is stored as the
    saturated code with its sign (the documented rule). Expected bytes: the oracle's append of the
    same token with those elements set to 0 (which never raises amax), then the saturated codes."""
    import paper_2606_26997_amd as rp
    _say("fp8 append with NaN elements")
    S = 8
    wl = make_workload(num_q_heads=4, num_kv_heads=2, head_dim=128, seq_to_group=np.zeros(S, int),
                       prefix_lens=[20], resp_lens=[0, 1, 5, 16, 17, 31, 40, 47], seed=13, append=True,
                       kv_dtype="fp8")
    nan_at = [(0, 0, 3, 0x7FC0), (2, 1, 100, 0xFFC0), (5, 0, 0, 0x7FC0), (6, 1, 127, 0xFFC0)]
    k_new = wl.k_new.copy()
    clean = wl.k_new.copy()
    for s_, h, c, bits in nan_at:
        k_new[s_, h, c] = bits
        clean[s_, h, c] = 0
    wl.k_new = k_new
    b = rp.DeviceBatch.from_workload(wl)
    b.kv_append()
    torch.cuda.synchronize()
    kp, _, ks, _ = oracle.kv_append(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale,
                                    v_scale=wl.v_scale, kv_dtype="fp8", page_size=16, resp_lens=wl.resp_lens,
                                    resp_block_table=wl.resp_block_table, k_new=clean, v_new=wl.v_new)
    for s_, h, c, bits in nan_at:
        t = int(wl.resp_lens[s_])
        kp[wl.resp_block_table[s_, t // 16], h, t % 16, c] = 0xFE if bits & 0x8000 else 0x7E
    assert np.array_equal(b.k_pages.cpu().numpy(), kp)
    assert np.array_equal(b.k_scale.cpu().numpy(), ks)


def test_zero_query_gives_log_key_count():
    """q = 0: lse = ln N exactly up to fp32, which pins the number of keys read."""
    _say("q=0 key count")
    rng = np.random.default_rng(3)
    S = 24
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.arange(S) // 8,
                       prefix_lens=[100, 255, 17], resp_lens=rng.integers(0, 3000, size=S), seed=1)
    wl.q[:] = 0
    _, out, lse = run_hip(wl)
    N = np.array([wl.prefix_lens[wl.seq_to_group[s]] + wl.resp_lens[s] for s in range(S)])
    np.testing.assert_allclose(lse, np.log(N)[:, None].repeat(16, 1), rtol=0, atol=2e-5)
    ref_out, ref_lse, _ = run_oracle(wl)
    compare(out, lse, ref_out, ref_lse, "bf16", "q=0")


def test_dominant_key_sweep_every_slot():
    """One key per sequence dominates; sweeping it over every prefix and response slot
    checks that each slot is read, with its own value row."""
    _say("dominant key sweep")
    d, P, L = 128, 40, 37
    rng = np.random.default_rng(4)
    pk, pv, rk, rv, s2g, _ = random_dense(rng, S=1, G=1, Hq=2, Hkv=1, d=d, prefix_lens=[P], resp_lens=[L])
    # One sequence per slot: all share the prefix, each has its own response copy.
    N = P + L
    S = N
    zero = bf16_bits(np.zeros((1, 1, d)))
    one = bf16_bits(np.full((1, d), 1.0))
    rks = []
    seq_group = []
    groups_pk, groups_pv = [], []
    for t in range(N):
        kp_ = np.repeat(zero, P, 0).copy()
        kr_ = np.repeat(zero, L, 0).copy()
        if t < P:
            kp_[t, 0] = one
        else:
            kr_[t - P, 0] = one
        groups_pk.append(kp_)
        groups_pv.append(pv[0])
        rks.append(kr_)
        seq_group.append(t)
    q = bf16_bits(np.full((S, 2, d), 1.0))      # score of the hot key: 128 / sqrt(128) = 11.3
    wl = paged_from_dense(groups_pk, groups_pv, rks, [rv[0]] * S, np.array(seq_group), q,
                          num_kv_heads=1, seed=2)
    _, out, lse = run_hip(wl)
    ref_out, ref_lse = oracle.attention_for_workload(wl)
    compare(out, lse, ref_out, ref_lse, "bf16", "dominant-key")


def test_physical_page_permutation_bitwise_and_determinism():
    _say("page permutation")
    rng = np.random.default_rng(8)
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=12, G=3, Hq=16, Hkv=8, d=128,
                                          prefix_lens=[70, 33, 160],
                                          resp_lens=list(rng.integers(0, 400, size=12)))
    wl1 = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=8, seed=1)
    wl2 = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=8, seed=2, pad_pages=7)
    b1, o1, l1 = run_hip(wl1)
    _, o2, l2 = run_hip(wl2)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    b1.step()
    o3, l3 = to_host_out(b1)
    assert np.array_equal(o1, o3) and np.array_equal(l1, l3)


def test_shared_prefix_equals_duplicated_prefix_on_gpu():
    _say("shared vs duplicated prefix")
    rng = np.random.default_rng(12)
    S, G = 16, 2
    P, L = [100, 45], list(rng.integers(0, 300, size=S))
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=16, Hkv=8, d=128, prefix_lens=P,
                                          resp_lens=L, seq_to_group=np.arange(S) % G)
    shared = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=8, seed=3)
    empty = [pk[0][:0]] * S
    dup = paged_from_dense(empty, empty, [np.concatenate([pk[s2g[s]], rk[s]]) for s in range(S)],
                           [np.concatenate([pv[s2g[s]], rv[s]]) for s in range(S)], np.arange(S), q,
                           num_kv_heads=8, seed=4)
    _, o1, l1 = run_hip(shared)
    _, o2, l2 = run_hip(dup)
    # Different split points and MFMA vs VALU arithmetic: equal within rounding.
    assert np.abs(o1 - o2).max() <= 1e-2
    assert np.abs(l1 - l2).max() <= 1e-4


def test_logical_key_order_permutation_within_tolerance():
    # Attention over a set of keys does not depend on their order: the same
    # keys in another logical order (prefix and response rows shuffled, so
    # pieces, chunks and page boundaries all change) give the same result up
    # to rounding.
    _say("logical key order permutation")
    rng = np.random.default_rng(21)
    S, G = 12, 3
    P, L = [90, 33, 160], list(rng.integers(1, 700, size=S))
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=16, Hkv=8, d=128, prefix_lens=P, resp_lens=L)
    perm_p = [rng.permutation(len(x)) for x in pk]
    perm_r = [rng.permutation(len(x)) for x in rk]
    wl1 = paged_from_dense(pk, pv, rk, rv, s2g, q, num_kv_heads=8, seed=5)
    wl2 = paged_from_dense([x[i] for x, i in zip(pk, perm_p)], [x[i] for x, i in zip(pv, perm_p)],
                           [x[i] for x, i in zip(rk, perm_r)], [x[i] for x, i in zip(rv, perm_r)],
                           s2g, q, num_kv_heads=8, seed=6)
    _, o1, l1 = run_hip(wl1)
    _, o2, l2 = run_hip(wl2)
    assert np.abs(o1 - o2).max() <= 1e-2
    assert np.abs(l1 - l2).max() <= 1e-4
    ref_out, ref_lse = oracle.attention_for_workload(wl1)
    compare(o2, l2, ref_out, ref_lse, "bf16", "permuted keys")


def test_gqa_mapping_value_in_one_kv_head():
    # V nonzero in kv-head 3 only: exactly query heads 6 and 7 (n_rep = 2,
    # q-head j reads kv-head j // 2) have a nonzero output; every other
    # head's output is exactly zero.
    _say("GQA mapping, V in one kv-head")
    rng = np.random.default_rng(22)
    S, G, h = 8, 2, 3
    P, L = [40, 77], list(rng.integers(0, 300, size=S))
    pk, pv, rk, rv, s2g, q = random_dense(rng, S=S, G=G, Hq=16, Hkv=8, d=128, prefix_lens=P, resp_lens=L)
    keep = lambda x: np.where((np.arange(8) == h)[None, :, None], x, np.uint16(0))
    wl = paged_from_dense(pk, [keep(x) for x in pv], rk, [keep(x) for x in rv], s2g, q, num_kv_heads=8, seed=7)
    _, out, lse = run_hip(wl)
    others = [j for j in range(16) if j // 2 != h]
    assert np.all(out[:, others] == 0)
    assert np.all(np.abs(out[:, [2 * h, 2 * h + 1]]).max(axis=2) > 0)
    ref_out, ref_lse = oracle.attention_for_workload(wl)
    compare(out, lse, ref_out, ref_lse, "bf16", "one kv-head")


def test_fp8_all_codes_decode_like_the_oracle():
    """A single key: out = decoded V codes * v_scale exactly (bf16 holds every e4m3 value)."""
    _say("fp8 256 codes")
    codes = np.arange(256, dtype=np.uint8)
    codes[codes == 0x7F] = 0x7E      # NaN codes are not attention inputs
    codes[codes == 0xFF] = 0xFE
    wl = make_workload(num_q_heads=2, num_kv_heads=1, head_dim=128, seq_to_group=[0, 0],
                       prefix_lens=[0], resp_lens=[1, 1], seed=0, kv_dtype="fp8")
    for s in range(2):
        page = wl.resp_block_table[s, 0]
        wl.v_pages[page, 0, 0, :] = codes[s * 128:(s + 1) * 128]
        wl.v_scale[page, 0] = np.float32(1.0)
        wl.k_scale[page, 0] = np.float32(0.5)
    _, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle(wl)
    want = oracle.e4m3_to_f64(codes).reshape(2, 1, 128)
    assert np.array_equal(out[:, 0:1, :], want) and np.array_equal(out[:, 1:2, :], want)
    assert np.array_equal(ref_out, np.repeat(want, 2, axis=1))
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-5)


def test_lse_combine_abi_against_oracle():
    _say("lse_combine")
    import paper_2606_26997_amd as rp
    rng = np.random.default_rng(5)
    rows, d = 300, 128
    counts = rng.integers(0, 9, size=rows)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    n = int(offs[-1])
    o = rng.standard_normal((n, d)).astype(np.float32)
    l = (rng.standard_normal(n) * 3).astype(np.float32)
    l[rng.random(n) < 0.1] = -np.inf
    o[l == -np.inf] = np.nan           # an empty part's o must not be read into the sum
    ref_out, ref_lse = oracle.lse_combine(o.astype(np.float64), l.astype(np.float64), offs)
    dev = lambda x: torch.from_numpy(x).cuda()
    out = torch.zeros((rows, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros(rows, dtype=torch.float32, device="cuda")
    rp.lse_combine(dev(o), dev(l), dev(offs), rows, d, out, lse)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    gl = lse.cpu().numpy().astype(np.float64)
    fin = np.isfinite(ref_lse)
    assert np.all(gl[~fin] == -np.inf) and np.all(got[~fin] == 0)
    assert np.abs(got - ref_out).max() <= 1e-2
    assert np.abs(gl[fin] - ref_lse[fin]).max() <= 1e-5


def test_validate_layout_reports_bad_page():
    _say("validate_layout")
    import paper_2606_26997_amd as rp
    wl = make_workload(num_q_heads=4, num_kv_heads=2, head_dim=64, seq_to_group=[0, 0],
                       prefix_lens=[20], resp_lens=[5, 40], seed=1)
    batch = rp.DeviceBatch.from_workload(wl)
    batch.validate()
    batch.resp_block_table[1, 2] = wl.num_pages + 5
    with pytest.raises(rp.RpError) as e:
        batch.validate()
    assert e.value.status == rp.RP_ERR_LAYOUT and "resp_block_table" in str(e.value)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_full_config_every_row(cid):
    """Full-size configs in the bench's launch configuration (plan, partial results, combine), every
    sequence compared with the oracle; then the same step again, which must be bitwise identical;
    then q = 0 on every row, where each score is exactly 0 and lse = ln N pins the number of keys
    each row read (one page of 20k keys moves it by 8e-4, the gate is 2e-5)."""
    _say(f"config{cid} full size, every row")
    wl = make_config_workload(CONFIGS[cid])
    _say(f"config{cid} generated: {wl.num_seqs} seqs, {wl.num_pages} pages")
    batch, out, lse = run_hip(wl)
    ref_out, ref_lse, _ = run_oracle_all(wl, label=f"config{cid}")
    stats = compare(out, lse, ref_out, ref_lse, wl.kv_dtype, f"config{cid}")
    _say(f"config{cid} all {wl.num_seqs} rows: {stats}")
    del ref_out, ref_lse

    batch.plan()
    batch.attn_parts()
    batch.combine_parts()
    out2, lse2 = to_host_out(batch)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2), "second run differs"

    batch.q.zero_()
    batch.step()
    out0, lse0 = to_host_out(batch)
    N = wl.prefix_lens[wl.seq_to_group].astype(np.int64) + wl.attn_resp_lens
    err = np.abs(lse0 - np.log(N.astype(np.float64))[:, None])
    _say(f"config{cid} q=0: max |lse - ln N| = {err.max():.2e} over {lse0.size} rows")
    assert err.max() <= 2e-5
    assert np.isfinite(out0).all()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("lo,hi,pages", [(2500, 3500, 64), (3800, 4400, 96)])
def test_frontier_batches_with_longer_pieces(lo, hi, pages):
    """8 groups x 8 live sequences: the planner picks 64- or 96-page pieces on a 256-CU GPU. Lengths
    include the edges of those multiples; every sequence is compared with the oracle."""
    import paper_2606_26997_amd as rp
    _say(f"frontier 64 seqs, responses U[{lo}, {hi}]")
    rng = np.random.default_rng(lo)
    L = rng.integers(lo, hi + 1, 64)
    edges = [pages * 16 * k + e for k in (2, 3) for e in (-1, 0, 1)]
    L[:len(edges)] = edges
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(8), 8),
                       prefix_lens=rng.integers(64, 513, 8), resp_lens=L, seed=lo)
    batch, out, lse = run_hip(wl)
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert int(batch.plan_contents()["hdr"][3]) == pages
    ref_out, ref_lse, _ = run_oracle_all(wl, label=f"frontier-{pages}")
    compare(out, lse, ref_out, ref_lse, "bf16", f"frontier-{pages}")
    assert np.isfinite(out).all() and np.isfinite(lse).all()


def _random_case(seed, big=None):
    """A seeded random batch: head counts, head_dim, kv dtype, group map, lengths and the append all drawn;
    the response lengths scaled so the pool stays near 150 MB. `big` = (kv dtype, sequences, longest
    response) fixes Hkv 8, d 64 and enough response pages for 64- or 96-page pieces on a 256-CU GPU."""
    rng = np.random.default_rng(seed)
    Hkv = int(rng.choice([1, 2, 4, 8]))
    nrep = int(rng.choice([1, 2, 4, 8] if Hkv <= 4 else [1, 2, 4]))
    d = int(rng.choice([64, 128]))
    dt = str(rng.choice(["bf16", "fp8"]))
    S = int(rng.integers(4, 260))
    if big is not None:
        Hkv, d, (dt, S, _) = 8, 64, big
    G = int(rng.integers(1, S + 1))
    s2g = rng.integers(0, G, S)
    P = rng.integers(0, 700, G)
    per_token = Hkv * d * 2 * (1 if dt == "fp8" else 2)
    Lmax = int(max(16, min(20000, 150e6 / per_token / S * 2))) if big is None else big[2]
    L = rng.integers(0, Lmax + 1, S)
    return dict(num_q_heads=Hkv * nrep, num_kv_heads=Hkv, head_dim=d, seq_to_group=s2g, prefix_lens=P,
                resp_lens=L, seed=seed, kv_dtype=dt, append=bool(rng.integers(0, 2)))


RANDOM = [(11, None), (22, None), (33, None), (44, None), (55, None), (66, None),
          (77, ("fp8", 120, 4500)), (88, ("bf16", 64, 5000))]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("seed,big", RANDOM, ids=[str(r[0]) for r in RANDOM])
def test_random_batches_every_row(seed, big):
    """Random shapes across the kernel templates (n_rep, head_dim, kv dtype) and piece lengths; every
    sequence is compared with the oracle."""
    kw = _random_case(seed, big)
    wl = make_workload(**kw)
    _say(f"random seed {seed}: S {wl.num_seqs}, G {wl.num_groups}, Hq {wl.num_q_heads}, Hkv {wl.num_kv_heads}, "
         f"d {wl.head_dim}, {wl.kv_dtype}, append {wl.append}, pages {wl.num_pages}")
    batch, out, lse = run_hip(wl)
    _say(f"random seed {seed}: piece length {int(batch.plan_contents()['hdr'][3])} pages")
    ref_out, ref_lse, _ = run_oracle_all(wl, label=f"random-{seed}")
    compare(out, lse, ref_out, ref_lse, wl.kv_dtype, f"random-{seed}")
    assert np.isfinite(out[np.isfinite(lse)]).all()
