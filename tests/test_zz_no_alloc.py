"""rp_group_decode_attn_noalloc (the library's static scratch, no workspace) against
rp_group_decode_attn on a caller workspace, through the C ABI: two calls in a row on one GPU,
the second with a smaller batch, each bit for bit equal to the workspace call and within the
oracle tolerances. The scratch keeps the first call's contents, so a read of anything the
second call did not write would show."""
import sys

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import compare, run_oracle
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _both(wl):
    import paper_2606_26997_amd as rp
    b = rp.DeviceBatch.from_workload(wl)
    if wl.append:
        b.kv_append()
    # Workspace call on a workspace filled with garbage (every byte 0xFF).
    b.workspace.fill_(255)
    b.attention()
    torch.cuda.synchronize()
    ref = (b.out.clone(), b.lse.clone())
    b.out.zero_()
    b.lse.zero_()
    rp.group_decode_attn_noalloc(b.kv, b.attn_layout, b.q, b.softmax_scale, b.out, b.lse)
    torch.cuda.synchronize()
    return b, ref


def test_noalloc_two_calls_match_the_workspace_call():
    import paper_2606_26997_amd as rp
    rng = np.random.default_rng(2027)
    first = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(12), 8),
                          prefix_lens=rng.integers(64, 513, 12), resp_lens=rng.integers(0, 4097, 96), seed=31)
    second = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=[0, 0, 0, 1, 1, 2],
                           prefix_lens=[100, 7, 300], resp_lens=[0, 15, 700, 33, 2000, 129], seed=32,
                           kv_dtype="fp8", append=True)
    for name, wl in (("first, 96 sequences, bf16", first), ("second, 6 sequences, fp8 with append", second)):
        _say(f"noalloc {name}")
        b, (ref_out, ref_lse) = _both(wl)
        _say(f"noalloc {name}: workspace {b.workspace.numel()} bytes of {rp.RP_NOALLOC_SCRATCH_BYTES}")
        assert b.workspace.numel() <= rp.RP_NOALLOC_SCRATCH_BYTES
        assert torch.equal(b.out.view(torch.int16), ref_out.view(torch.int16)), name
        assert torch.equal(b.lse.view(torch.int32), ref_lse.view(torch.int32)), name
        out = b.out.float().cpu().numpy().astype(np.float64)
        lse = b.lse.cpu().numpy().astype(np.float64)
        o_ref, l_ref, _ = run_oracle(wl)
        compare(out, lse, o_ref, l_ref, wl.kv_dtype, f"noalloc {name}")


def test_noalloc_refuses_a_layout_beyond_the_scratch():
    import paper_2606_26997_amd as rp
    _say("noalloc: layout beyond the scratch")
    # 64 sequences with room for 8000 response pages each: a 127 MB workspace.
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.zeros(64, int),
                       prefix_lens=[16], resp_lens=np.arange(64), seed=3, max_resp_pages=8000)
    b = rp.DeviceBatch.from_workload(wl)
    assert b.workspace.numel() > rp.RP_NOALLOC_SCRATCH_BYTES
    with pytest.raises(rp.RpError) as e:
        rp.group_decode_attn_noalloc(b.kv, b.attn_layout, b.q, b.softmax_scale, b.out, b.lse)
    assert e.value.status == rp.RP_ERR_WORKSPACE and "static scratch" in str(e.value)
