"""GPU parity of the shared-prefix prefill through the C ABI against the fp64 oracle.

The page write is compared byte for byte (bf16 copies and fp8 codes with their
scales); causal attention element by element at the decode path's tolerances,
the max-abs bound widened by half a bf16 ulp of each exact value (the output
format's rounding).
An end-to-end case decodes each prompt's last token over the pages the prefill
wrote and checks it against the prefill's own last row.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import TOL
from workloads import make_prefill_workload

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _run(w):
    import paper_2606_26997_amd as rp
    b = rp.PrefillBatch.from_workload(w)
    b.step()
    torch.cuda.synchronize()
    return b


def _check_pages(b, w, label):
    kp, vp, ks, vs = oracle.prefill_kv_write(k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale,
                                             v_scale=w.v_scale, kv_dtype=w.kv_dtype, page_size=16,
                                             prefix_block_table=w.prefix_block_table, prefix_offs=w.prefix_offs,
                                             k=w.k, v=w.v)
    view = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) if w.kv_dtype == "bf16" else \
        (lambda t: t.cpu().numpy())
    np.testing.assert_array_equal(view(b.k_pages), kp, err_msg=label)
    np.testing.assert_array_equal(view(b.v_pages), vp, err_msg=label)
    if w.kv_dtype == "fp8":
        np.testing.assert_array_equal(b.k_scale.cpu().numpy(), ks, err_msg=label)
        np.testing.assert_array_equal(b.v_scale.cpu().numpy(), vs, err_msg=label)


def _check_attn(b, w, label, rows=None):
    ref_out, ref_lse = oracle.prefill_attention(w.q, w.k, w.v, w.prefix_offs, w.softmax_scale)
    out = b.out.float().cpu().numpy().astype(np.float64)
    lse = b.lse.cpu().numpy().astype(np.float64)
    if rows is not None:
        out, lse, ref_out, ref_lse = out[rows], lse[rows], ref_out[rows], ref_lse[rows]
    tol = TOL["bf16"]
    # The output is bf16: the bound covers the computation plus the format's
    # own rounding, half a bf16 ulp of the exact value. Early prompt tokens
    # attend few keys and reach |out| ~ 4, where that half-ulp alone is 0.0078.
    half_ulp = np.ldexp(1.0, np.frexp(np.abs(ref_out))[1] - 9)
    diff = np.abs(out - ref_out)
    err = np.maximum(diff - half_ulp, 0.0)
    rel = np.sqrt((diff ** 2).sum() / max((ref_out ** 2).sum(), 1e-300))
    dl = np.abs(lse - ref_lse)
    msg = f"{label}: max_abs={err.max():.3e} rel_l2={rel:.3e} max_dlse={dl.max():.3e}"
    assert err.max() <= tol["max_abs"], msg
    assert rel <= tol["rel_l2"], msg
    assert dl.max() <= tol["lse_tight"], msg


CASES = [
    # name, prompt lengths, Hq, Hkv, d, kv dtype
    ("ragged-d128", [1, 15, 16, 17, 33, 0, 200], 16, 8, 128, "bf16"),
    ("ragged-d64", [5, 64, 65, 1], 4, 2, 64, "bf16"),
    ("mha", [31, 7], 4, 4, 64, "bf16"),
    ("nrep4", [40, 3, 18], 8, 2, 128, "bf16"),
    ("nrep8", [25, 9], 8, 1, 128, "bf16"),
    ("fp8-pages", [1, 16, 17, 100], 16, 8, 128, "fp8"),
    ("fp8-d64", [48, 2], 4, 2, 64, "fp8"),
    # Prompts averaging 384+ tokens take two 16-row tiles per wave.
    ("long-two-tiles-d128", [400, 700, 513, 385], 16, 8, 128, "bf16"),
    ("long-two-tiles-d64-nrep4", [450, 390, 1], 8, 2, 64, "bf16"),
    ("long-two-tiles-nrep8", [600, 255], 8, 1, 128, "bf16"),
    ("long-two-tiles-mha", [420, 401, 17], 4, 4, 64, "bf16"),
    ("long-two-tiles-fp8", [520, 333], 16, 8, 128, "fp8"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_prefill_pages_and_attention(case):
    name, P, Hq, Hkv, d, dt = case
    _say(f"prefill {name}")
    w = make_prefill_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, prefix_lens=P, seed=len(name),
                              kv_dtype=dt)
    b = _run(w)
    _check_pages(b, w, name)
    _check_attn(b, w, name)


@pytest.mark.parametrize("one_call", [False, True], ids=["two-calls", "rp_prefill"])
def test_qwen_layer_prompts_full(one_call):
    # The decode benchmark's prompts: 32 groups, prefix U[64, 512], Hq=16, Hkv=8, d=128, K x 0.5,
    # through the two calls and through rp_prefill (the launch the prefill bench times).
    import paper_2606_26997_amd as rp
    _say(f"prefill 32 groups x U[64,512], {'rp_prefill' if one_call else 'two calls'}")
    rng = np.random.default_rng(1002)
    w = make_prefill_workload(num_q_heads=16, num_kv_heads=8, head_dim=128,
                              prefix_lens=rng.integers(64, 513, 32), seed=1002, k_mult=0.5)
    if one_call:
        b = rp.PrefillBatch.from_workload(w)
        b.prefill()
        torch.cuda.synchronize()
    else:
        b = _run(w)
    _check_pages(b, w, "qwen-prompts")
    _check_attn(b, w, "qwen-prompts")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("one_call", [False, True], ids=["two-calls", "rp_prefill"])
def test_1024_token_prompts_full(one_call):
    # The prefill bench's long case: 32 groups of 1024-token prompts (two
    # row tiles per wave; rp_prefill copies each workgroup's own rows into the
    # pages in its prologue), every row against the oracle.
    import paper_2606_26997_amd as rp
    _say(f"prefill 32 groups x 1024 tokens, {'rp_prefill' if one_call else 'two calls'}")
    w = make_prefill_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, prefix_lens=[1024] * 32, seed=1024)
    if one_call:
        b = rp.PrefillBatch.from_workload(w)
        b.prefill()
        torch.cuda.synchronize()
    else:
        b = _run(w)
    _check_pages(b, w, "1024-token prompts")
    _check_attn(b, w, "1024-token prompts")


def test_long_prompts():
    # Largest prompts of the tests: a 4096-token prompt (256 prefix pages) and a
    # ragged 2200-token one; 128 key blocks for the last rows.
    _say("prefill 4096 + 2200 tokens")
    w = make_prefill_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, prefix_lens=[4096, 2200], seed=4096)
    b = _run(w)
    _check_pages(b, w, "long-prompts")
    _check_attn(b, w, "long-prompts")


def test_decode_over_prefilled_pages_matches_last_prompt_row():
    import paper_2606_26997_amd as rp
    _say("prefill then decode the last prompt tokens")
    rng = np.random.default_rng(5)
    P = rng.integers(20, 300, 6)
    w = make_prefill_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, prefix_lens=P, seed=5)
    b = _run(w)
    G = len(P)
    last = w.prefix_offs[1:] - 1
    dev = torch.device("cuda")
    dec = rp.DeviceBatch(k_pages=b.k_pages, v_pages=b.v_pages, k_scale=None, v_scale=None,
                         seq_to_group=np.arange(G, dtype=np.int32), prefix_lens=P.astype(np.int32),
                         prefix_block_table=w.prefix_block_table, resp_lens=np.zeros(G, np.int32),
                         resp_block_table=np.zeros((G, 1), np.int32), q=b.q[torch.as_tensor(last, device=dev)],
                         num_q_heads=16, softmax_scale=w.softmax_scale)
    dec.step()
    torch.cuda.synchronize()
    o_dec = dec.out.float().cpu().numpy()
    o_pre = b.out[torch.as_tensor(last, device=dev)].float().cpu().numpy()
    assert np.abs(o_dec - o_pre).max() <= 1e-2
    np.testing.assert_allclose(dec.lse.cpu().numpy(), b.lse[torch.as_tensor(last, device=dev)].cpu().numpy(),
                               rtol=0, atol=1e-4)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_one_call_prefill_matches_the_two_calls(case):
    """rp_prefill (one launch for bf16 pools: the attention kernel also writes the pages) gives the same page
    bytes, scales, out and lse as rp_prefill_kv_write then rp_prefill_attn, and matches the oracle."""
    import paper_2606_26997_amd as rp
    name, P, Hq, Hkv, d, dt = case
    _say(f"one-call prefill {name}")
    w = make_prefill_workload(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, prefix_lens=P, seed=len(name),
                              kv_dtype=dt)
    two = _run(w)
    one = rp.PrefillBatch.from_workload(w)
    one.prefill()
    torch.cuda.synchronize()
    assert torch.equal(one.k_pages.view(torch.uint8), two.k_pages.view(torch.uint8)), name
    assert torch.equal(one.v_pages.view(torch.uint8), two.v_pages.view(torch.uint8)), name
    if dt == "fp8":
        assert torch.equal(one.k_scale, two.k_scale) and torch.equal(one.v_scale, two.v_scale), name
    assert torch.equal(one.out.view(torch.int16), two.out.view(torch.int16)), name
    assert torch.equal(one.lse.view(torch.int32), two.lse.view(torch.int32)), name
    _check_pages(one, w, name)
    _check_attn(one, w, name)
