"""Host-side pieces of bench.py: the one-GPU guard and the algorithmic byte model."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import make_workload  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_byte_model_counts_a_shared_prefix_once_per_group():
    # 3 groups (one without live members), Hq 4, Hkv 2, d 64, bf16: K+V per token = 2*64*2*2 = 512 B.
    s2g = [0, 0, 0, 2]
    wl = make_workload(num_q_heads=4, num_kv_heads=2, head_dim=64, seq_to_group=s2g, prefix_lens=[20, 7, 33],
                       resp_lens=[5, 0, 17, 40], seed=3)
    bm = bench.byte_model(wl)
    tok = 2 * 64 * 2 * 2
    assert bm["prefix_kv"] == (20 + 33) * tok          # group 1 has no live member
    assert bm["resp_kv"] == (5 + 0 + 17 + 40) * tok
    assert bm["q"] == bm["out"] == 4 * 4 * 64 * 2
    assert bm["lse"] == 4 * 4 * 4
    assert bm["total"] == sum(bm[k] for k in ("prefix_kv", "resp_kv", "q", "out", "lse", "scales", "append"))
    assert bm["parts_kernel"] == bm["prefix_kv"] + bm["resp_kv"] + bm["q"]
    # Prefix tile rows: 3 * 2 rows (group 0) and 1 * 2 (group 2), in 16-row tiles.
    assert bm["prefix_tile_rows"] == 8
    assert np.isclose(bm["prefix_tile_padded_frac"], 1 - 8 / 32)


def test_byte_model_fp8_scales_and_append():
    wl = make_workload(num_q_heads=4, num_kv_heads=2, head_dim=64, seq_to_group=[0, 0], prefix_lens=[16],
                       resp_lens=[15, 16], seed=4, kv_dtype="fp8", append=True)
    bm = bench.byte_model(wl)
    tok = 2 * 64 * 2 * 1
    L = np.asarray(wl.attn_resp_lens)
    assert bm["resp_kv"] == int(L.sum()) * tok
    pages = 1 + int(((L + 15) // 16).sum())
    assert bm["scales"] == pages * 2 * 8                  # k and v scale per (page, kv-head)
    # new k and v read as bf16, written as fp8: S * Hkv * d * 2 tensors * (2 + 1) bytes
    assert bm["append"] == 2 * 2 * 64 * 2 * (2 + 1)
