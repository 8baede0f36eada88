"""GPU parity of the GRPO group advantages (Eq. 1) through the C ABI against the fp64 oracle.

The kernel computes in fp64 and rounds each output once, like the oracle;
the summation orders differ, so outputs must agree to one fp32 ulp, and in
practice bit for bit (required for at least 99.9% of elements, and for every
element of the binary-reward groups, whose sums are exact).
"""
import sys

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _ulps(a, b):
    ia = a.view(np.int32).astype(np.int64)
    ib = b.view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    return np.abs(ia - ib)


def _run(r, eps=1e-6, ddof=1, offset=0, inplace=False):
    import paper_2606_26997_amd as rp
    R, K = r.shape
    buf = torch.zeros(R * K + offset + 4, dtype=torch.float32, device="cuda")
    rd = buf[offset:offset + R * K].view(R, K)
    rd.copy_(torch.from_numpy(r))
    adv = rd if inplace else torch.empty_like(rd)
    mu = torch.empty(R, dtype=torch.float32, device="cuda")
    sd = torch.empty(R, dtype=torch.float32, device="cuda")
    rp.grpo_advantage(rd, adv, mu, sd, eps_std=eps, ddof=ddof)
    torch.cuda.synchronize()
    return adv.cpu().numpy(), mu.cpu().numpy(), sd.cpu().numpy()


def _check(got, ref, label, exact_frac=0.999):
    for g, e, what in zip(got, ref, ("advantages", "mean", "std")):
        d = _ulps(np.ascontiguousarray(g), np.ascontiguousarray(e))
        assert d.max(initial=0) <= 1, f"{label} {what}: max ulp {d.max()}"
        frac = float((d == 0).mean()) if d.size else 1.0
        assert frac >= exact_frac, f"{label} {what}: {frac:.5f} bit-identical"


CASES = [  # name, R, K, ddof, eps, offset (floats), in place
    ("K8", 1000, 8, 1, 1e-6, 0, False), ("K8-ddof0", 777, 8, 0, 1e-6, 0, False), ("K4", 513, 4, 1, 1e-6, 0, False),
    ("K16", 300, 16, 1, 1e-4, 0, False), ("K5-generic", 401, 5, 1, 1e-6, 0, False),
    ("K8-unaligned", 257, 8, 1, 1e-6, 1, False), ("K8-in-place", 300, 8, 1, 1e-6, 0, True),
    ("K1", 100, 1, 1, 1e-6, 0, False), ("K1-ddof0", 100, 1, 0, 1e-6, 0, False), ("K64", 50, 64, 1, 1e-6, 0, False),
    ("eps0", 200, 8, 0, 0.0, 0, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_grpo_advantage_matches_oracle(case):
    name, R, K, ddof, eps, off, inplace = case
    _say(f"grpo {name}")
    r = (np.random.default_rng(R + K).standard_normal((R, K)) * 2.0 + 0.5).astype(np.float32)
    got = _run(r, eps=eps, ddof=ddof, offset=off, inplace=inplace)
    _check(got, oracle.advantage_f32(r, eps_std=eps, ddof=ddof), name)
    if K > 1:
        assert np.abs(got[0].astype(np.float64).sum(axis=1)).max() < 1e-4


@pytest.mark.parametrize("K", [8, 16])
def test_binary_rewards_bitwise(K):
    # Exact-match rewards (Section 5.1): 0/1 per response, per-group pass rates.
    _say(f"grpo binary K={K}")
    rng = np.random.default_rng(K)
    p = rng.uniform(0, 1, 4096)
    r = (rng.uniform(0, 1, (4096, K)) < p[:, None]).astype(np.float32)
    got = _run(r)
    ref = oracle.advantage_f32(r)
    for g, e in zip(got, ref):
        assert np.array_equal(g, e)
    # All-correct and all-wrong groups carry no signal.
    same = (r.min(axis=1) == r.max(axis=1))
    assert same.any() and np.all(got[0][same] == 0.0)


def test_large_batch_every_group():
    _say("grpo 2^20 groups")
    R, K = 1 << 20, 8
    r = np.random.default_rng(5).standard_normal((R, K)).astype(np.float32)
    adv, mu, sd = _run(r)
    _check((adv, mu, sd), oracle.advantage_f32(r), "2^20 groups")
