"""The native scheduling simulation (rp_sched_simulate) against the step-by-step oracle (CPU only).

Both evaluate the same documented IEEE expressions in the same order, so every
time, the FIFO order, the update timeline and the step count must agree bit
for bit, across the three modes, engine capacities from one request to all of
them, frontier widths from one group to all of them, and edge cases (one
sample per group, one update per round, empty prompts, zero costs). One round
runs at the paper's scale (R = 96 groups of K = 8, B = 16 so U = 2, F_w = 2,
responses of about 3.3k tokens).
"""
import ctypes
import itertools

import numpy as np
import pytest

import oracle
import paper_2606_26997_amd as rp
from paper_2606_26997_amd import _binding as B
from workloads import make_rollout_workload

KEYS = ("serve_done", "frontier_enter", "trainable", "fifo", "update_start", "update_end", "steps", "t_first_u",
        "t_complete", "t_start", "delta_cgp", "t_train_end", "compute", "wait", "w_train", "wait_ratio")

COSTS = dict(step_base=1.1e-3, step_per_seq=7.8e-8, step_per_ctx_token=1.94e-11, prefill_per_token=3.4e-7,
             mat_base=0.05, mat_per_token=2e-6, train_base=0.3, train_per_token=1.9e-4, opt_step=0.8)


def _same(a, b, label):
    for k in KEYS:
        assert a[k] == b[k], f"{label}: {k} differs"


@pytest.mark.parametrize("mode,cap,fw,U", [
    (m, c, f, u) for m, c, f, u in itertools.product(("slime", "cgp", "cgp_fgd"), (1, 7, 24, 10 ** 6), (1, 2, 5),
                                                       (1, 2, 4))
    if not (m != "cgp_fgd" and f != 1)])
def test_native_matches_oracle_bitwise(mode, cap, fw, U):
    P, L = make_rollout_workload(num_groups=16, group_size=4, seed=cap + 10 * fw + U, resp_median=40, resp_cap=120)
    kw = dict(group_size=4, update_groups=U, prompt_lens=P, resp_lens=L, max_running=cap, frontier_width=fw, **COSTS)
    _same(rp.sched_simulate(mode=mode, **kw), oracle.simulate_schedule(mode=mode, **kw), f"{mode}/{cap}/{fw}/{U}")


@pytest.mark.parametrize("case", ["one-sample-groups", "one-update", "frontier-all", "empty-prompts", "zero-costs",
                                  "unit-lengths"])
def test_native_matches_oracle_edge_cases(case):
    rng = np.random.default_rng(len(case))
    R, K, U, fw, cap = 8, 4, 2, 2, 9
    P = rng.integers(0, 50, R)
    L = rng.integers(1, 30, R * K)
    costs = dict(COSTS)
    if case == "one-sample-groups":
        K, L = 1, rng.integers(1, 30, R)
    elif case == "one-update":
        U = R
    elif case == "frontier-all":
        fw = R + 3
    elif case == "empty-prompts":
        P = np.zeros(R, np.int32)
    elif case == "zero-costs":
        costs = {k: 0.0 for k in costs}
    elif case == "unit-lengths":
        L = np.ones(R * K, np.int32)
    for mode in ("slime", "cgp", "cgp_fgd"):
        kw = dict(group_size=K, update_groups=U, prompt_lens=P, resp_lens=L, max_running=cap, frontier_width=fw,
                  **costs)
        _same(rp.sched_simulate(mode=mode, **kw), oracle.simulate_schedule(mode=mode, **kw), f"{case}/{mode}")


@pytest.mark.parametrize("mode", ["slime", "cgp", "cgp_fgd"])
def test_paper_scale_round(mode):
    P, L = make_rollout_workload(num_groups=96, group_size=8, seed=96)
    kw = dict(group_size=8, update_groups=2, prompt_lens=P, resp_lens=L, max_running=256, frontier_width=2, **COSTS)
    a = rp.sched_simulate(mode=mode, **kw)
    b = oracle.simulate_schedule(mode=mode, **kw)
    _same(a, b, mode)
    assert a["steps"] > 8000


def test_invalid_arguments_rejected():
    lib = rp.load()
    P = np.array([3, 4], np.int32)
    L = np.ones(4, np.int32)
    summ = B.RpSchedSummary()

    def run(cfg, p=P, l=L):
        return lib.rp_sched_simulate(ctypes.byref(cfg), p.ctypes.data_as(ctypes.c_void_p),
                                     l.ctypes.data_as(ctypes.c_void_p), ctypes.byref(summ),
                                     None, None, None, None, None, None)

    def cfg(**kw):
        d = dict(mode=1, R=2, K=2, U=1, fw=0, cap=4, costs=[0.0] * 9)
        d.update(kw)
        return B.RpSchedConfig(d["mode"], d["R"], d["K"], d["U"], d["fw"], d["cap"], *d["costs"])
    assert run(cfg()) == rp.RP_OK
    assert run(cfg(U=3)) == rp.RP_ERR_INVALID_ARG and "update_groups" in rp.last_error()
    assert run(cfg(cap=0)) == rp.RP_ERR_INVALID_ARG
    assert run(cfg(mode=7)) == rp.RP_ERR_INVALID_ARG and "mode" in rp.last_error()
    assert run(cfg(mode=2)) == rp.RP_ERR_INVALID_ARG and "frontier_width" in rp.last_error()
    assert run(cfg(costs=[0.0] * 8 + [-1.0])) == rp.RP_ERR_INVALID_ARG and "cost" in rp.last_error()
    assert run(cfg(costs=[float("nan")] + [0.0] * 8)) == rp.RP_ERR_INVALID_ARG
    assert run(cfg(), l=np.array([1, 0, 1, 1], np.int32)) == rp.RP_ERR_INVALID_ARG
    assert run(cfg(), p=np.array([-1, 2], np.int32)) == rp.RP_ERR_INVALID_ARG
    assert lib.rp_sched_simulate(None, None, None, None, None, None, None, None, None, None) == rp.RP_ERR_INVALID_ARG
