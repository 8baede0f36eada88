"""A decode step captured in a HIP graph replays to the eager result, bit for bit.

The decode path launches kernels only (no allocation, memset, copy or host
synchronisation inside a step), so a serving loop can capture a whole step
once and replay it. Each case captures the step with torch.cuda.graph on a
side stream, then replays it three times with eager work between replays
(outputs overwritten with NaN, an eager step, synchronisations) and compares
every replay with the eager step's outputs and pool bytes. The steps are
idempotent: the append writes the slot at resp_lens[s] again with the same
values.
"""
import sys

import numpy as np
import pytest
import torch

from workloads import make_qkprep_inputs, make_workload

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.uint8) if t.element_size() == 1 \
        else t.view(torch.int32)


def _snapshot(b):
    xs = [b.out, b.lse, b.k_pages, b.v_pages]
    xs += [t for t in (b.k_scale, b.v_scale) if t is not None]
    return [x.clone() for x in xs]


def _check_replays(b, step, label):
    step()
    torch.cuda.synchronize()
    ref = _snapshot(b)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for i in range(3):
        b.out.fill_(float("nan"))
        b.lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, x, r in zip(("out", "lse", "k_pages", "v_pages", "k_scale", "v_scale"), _snapshot(b), ref):
            assert torch.equal(_bits(x), _bits(r)), f"{label}: replay {i}: {name}"
        step()  # eager work between replays
        torch.cuda.synchronize()


def test_frontier_step_prep_plan_parts_combine():
    import paper_2606_26997_amd as rp
    _say("graph: frontier step, 2 groups x 8, prep+plan, parts, combine")
    rng = np.random.default_rng(77)
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(2), 8),
                       prefix_lens=[512, 300], resp_lens=rng.integers(0, 3000, 16), seed=77, append=True,
                       k_mult=0.5, rng=rng)
    x = make_qkprep_inputs(num_seqs=16, num_q_heads=16, num_kv_heads=8, head_dim=128, seed=78)
    b = rp.DeviceBatch.from_workload(wl)
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w)

    def step():
        b.qk_prep_plan()
        b.attn_parts()
        b.combine_parts()
    _check_replays(b, step, "frontier step")


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_append_and_attention_one_call(kv_dtype):
    import paper_2606_26997_amd as rp
    _say(f"graph: append + rp_group_decode_attn, 96 sequences, {kv_dtype}")
    rng = np.random.default_rng(5)
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(12), 8),
                       prefix_lens=rng.integers(64, 513, 12), resp_lens=rng.integers(0, 2049, 96), seed=6,
                       append=True, kv_dtype=kv_dtype, rng=rng)
    b = rp.DeviceBatch.from_workload(wl)
    _check_replays(b, b.step, f"append + attention {kv_dtype}")


def test_noalloc_attention():
    import paper_2606_26997_amd as rp
    _say("graph: rp_group_decode_attn_noalloc, 48 sequences")
    rng = np.random.default_rng(9)
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(6), 8),
                       prefix_lens=rng.integers(64, 513, 6), resp_lens=rng.integers(0, 2049, 48), seed=10, rng=rng)
    b = rp.DeviceBatch.from_workload(wl)

    def step():
        rp.group_decode_attn_noalloc(b.kv, b.attn_layout, b.q, b.softmax_scale, b.out, b.lse)
    _check_replays(b, step, "noalloc attention")
