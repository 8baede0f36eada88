"""Pins for the oracle's CGP / FGD scheduling simulation (CPU only).

The worked example of Section 3.3 (frontier width 2 over six groups, U = 2) is
checked from a fixture; the rollout is checked against closed forms (all
requests running at a constant step time, one frontier group at a time, one
request at a time, the context-dependent step cost of a single request); the
trainer against Eq. 2 (Slime starts at rollout completion, CGP at the first U
trainable groups), Eq. 3 and Eq. 4 recomputed from the update timeline, and
against invariants: FGD with a frontier covering every group is plain FIFO
admission, the frontier never exceeds F_w and is filled in group order, and
every mode does the same training work.
"""
import os

import numpy as np
import pytest

from oracle import simulate_schedule as sim

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fgd_worked_example.txt")


def _fixture():
    out = {}
    for line in open(GOLDEN):
        if line.strip() and not line.startswith("#"):
            k, *v = line.split()
            out[k] = [int(x) for x in v]
    return out


def _rand(R=12, K=4, seed=0, lmax=40):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 30, R).tolist(), rng.integers(1, lmax, R * K).tolist()


def test_section_3_3_worked_example():
    ex = _fixture()
    Fw, U = ex["frontier_width"][0], ex["update_groups"][0]
    R = len(ex["groups"])
    # Lengths chosen so that group 1 finishes first; every step costs 1 s.
    L = [3, 2, 5, 4, 6, 6, 2, 7, 4, 4, 9, 9]
    r = sim(mode="cgp_fgd", group_size=2, update_groups=U, prompt_lens=[8] * R, resp_lens=L, max_running=64,
            frontier_width=Fw, step_base=1.0)
    done, enter = r["serve_done"], r["frontier_enter"]

    def frontier_at(t):  # 1-based group numbers in the frontier just after the cycle at time t
        return sorted(g + 1 for g in range(R) if enter[g] <= t < done[g])
    assert frontier_at(0.0) == ex["initial_frontier"]
    first = min(range(R), key=lambda g: done[g])
    assert first + 1 == 1
    assert frontier_at(done[first]) == ex["after_group_1_completes"]
    # The trainer starts when two groups are trainable; the listed groups are
    # then still in rollout.
    assert r["t_start"] == sorted(r["trainable"])[U - 1]
    still = [g + 1 for g in range(R) if done[g] > r["t_start"]]
    assert still == ex["trainer_starts_while_in_rollout"]


@pytest.mark.parametrize("mode", ["slime", "cgp"])
def test_all_running_constant_step_closed_form(mode):
    P, L = _rand(R=10, K=3, seed=1)
    tau, m = 0.25, 1.5
    r = sim(mode=mode, group_size=3, update_groups=2, prompt_lens=P, resp_lens=L, max_running=10 ** 6,
            step_base=tau, mat_base=m)
    for g in range(10):
        assert r["serve_done"][g] == tau * max(L[3 * g:3 * g + 3])
        assert r["trainable"][g] == r["serve_done"][g] + m
    tr = sorted(r["trainable"])
    assert r["t_first_u"] == tr[1] and r["t_complete"] == tr[-1]
    assert r["delta_cgp"] == tr[-1] - tr[1]                              # Eq. 3
    assert r["steps"] == max(L)


def test_frontier_of_one_runs_groups_back_to_back():
    P, L = _rand(R=7, K=4, seed=2)
    r = sim(mode="cgp_fgd", group_size=4, update_groups=1, prompt_lens=P, resp_lens=L, max_running=10 ** 6,
            frontier_width=1, step_base=0.5)
    acc = 0.0
    for g in range(7):
        assert r["frontier_enter"][g] == acc
        acc += 0.5 * max(L[4 * g:4 * g + 4])
        assert r["serve_done"][g] == pytest.approx(acc, rel=1e-15)
    assert r["fifo"] == list(range(7))


def test_one_request_at_a_time_is_fifo_in_request_order():
    P, L = _rand(R=5, K=2, seed=3)
    r = sim(mode="cgp", group_size=2, update_groups=1, prompt_lens=P, resp_lens=L, max_running=1, step_base=2.0)
    acc = 0.0
    for g in range(5):
        acc += 2.0 * (L[2 * g] + L[2 * g + 1])
        assert r["serve_done"][g] == pytest.approx(acc, rel=1e-15)


def test_step_cost_of_a_single_request():
    # ctx before step j is P + j, so the decode costs s * (l P + l (l - 1) / 2),
    # plus the prompt prefill once and the per-step and per-sequence terms.
    P, l, s, p, b, q = 37, 11, 0.001, 0.01, 0.5, 0.25
    r = sim(mode="cgp", group_size=1, update_groups=1, prompt_lens=[P], resp_lens=[l], max_running=4,
            step_base=b, step_per_seq=q, step_per_ctx_token=s, prefill_per_token=p)
    assert r["serve_done"][0] == pytest.approx(l * (b + q) + s * (l * P + l * (l - 1) / 2) + p * P, rel=1e-13)


def test_prefill_counts_once_per_group():
    # Two groups of 4 requests, one running slot per request: each group's
    # prompt is charged once however many of its requests start.
    r1 = sim(mode="cgp", group_size=4, update_groups=1, prompt_lens=[100, 50], resp_lens=[1] * 8, max_running=8,
             prefill_per_token=1.0)
    assert r1["serve_done"] == [150.0, 150.0]
    r2 = sim(mode="cgp", group_size=4, update_groups=1, prompt_lens=[100, 50], resp_lens=[1] * 8, max_running=4,
             prefill_per_token=1.0)
    assert r2["serve_done"] == [100.0, 150.0]


def test_eq2_trainer_start_and_slime_back_to_back():
    P, L = _rand(R=8, K=4, seed=4)
    kw = dict(group_size=4, update_groups=2, prompt_lens=P, resp_lens=L, max_running=10 ** 6, step_base=0.1,
              mat_base=0.3, mat_per_token=0.01, train_base=2.0, train_per_token=0.002, opt_step=0.7)
    s, c = sim(mode="slime", **kw), sim(mode="cgp", **kw)
    assert s["serve_done"] == c["serve_done"] and s["trainable"] == c["trainable"]
    assert s["t_start"] == s["t_complete"]                               # Eq. 2, Slime
    assert c["t_start"] == c["t_first_u"]                                # Eq. 2, CGP (trainer idle until then)
    # Slime trains back to back from rollout completion.
    comp = [2.0 + 0.002 * (4 * P[g] + sum(L[4 * g:4 * g + 4])) for g in range(8)]
    fifo = s["fifo"]
    t = s["t_complete"]
    for k in range(4):
        assert s["update_start"][k] == pytest.approx(t, rel=1e-15)
        t += sum(comp[g] for g in fifo[2 * k:2 * k + 2]) + 0.7
    assert s["t_train_end"] == pytest.approx(t, rel=1e-14)
    assert c["t_train_end"] <= s["t_train_end"]


@pytest.mark.parametrize("mode", ["slime", "cgp", "cgp_fgd"])
def test_eq4_and_waiting_ratio_from_the_update_timeline(mode):
    P, L = _rand(R=12, K=4, seed=5)
    r = sim(mode=mode, group_size=4, update_groups=3, prompt_lens=P, resp_lens=L, max_running=20, frontier_width=2,
            step_base=0.2, step_per_ctx_token=1e-3, mat_base=1.0, train_base=3.0, train_per_token=0.01, opt_step=1.0)
    st, en = r["update_start"], r["update_end"]
    idle = st[0] + sum(st[k] - en[k - 1] for k in range(1, len(st)))
    busy = sum(e - s for s, e in zip(st, en))
    assert r["w_train"] == pytest.approx(st[0] / en[-1], rel=1e-15)     # Eq. 4
    assert r["wait_ratio"] == pytest.approx(idle / (idle + busy), rel=1e-12)
    assert r["wait_ratio"] >= r["w_train"] - 1e-15                       # the initial wait is part of all waiting
    # Each update consumes the next U FIFO groups after they are all trainable.
    tr = r["trainable"]
    for k, s in enumerate(st):
        batch = r["fifo"][3 * k:3 * k + 3]
        assert s >= max(tr[g] for g in batch) - 1e-12
        assert s >= (r["t_complete"] if mode == "slime" else 0.0)


def test_frontier_covering_every_group_is_fifo_admission():
    P, L = _rand(R=9, K=4, seed=6)
    kw = dict(group_size=4, update_groups=3, prompt_lens=P, resp_lens=L, max_running=11, step_base=0.1,
              step_per_ctx_token=1e-3, prefill_per_token=1e-3, mat_base=0.5, train_base=1.0)
    a, b = sim(mode="cgp", **kw), sim(mode="cgp_fgd", frontier_width=9, **kw)
    for key in ("serve_done", "trainable", "fifo", "update_start", "update_end", "steps"):
        assert a[key] == b[key], key


@pytest.mark.parametrize("Fw", [1, 2, 3])
def test_frontier_bounded_and_filled_in_order(Fw):
    P, L = _rand(R=10, K=4, seed=7 + Fw)
    r = sim(mode="cgp_fgd", group_size=4, update_groups=2, prompt_lens=P, resp_lens=L, max_running=6,
            frontier_width=Fw, step_base=0.1, step_per_ctx_token=1e-3)
    enter, done = r["frontier_enter"], r["serve_done"]
    assert enter == sorted(enter)
    for t in set(enter) | set(done):
        assert sum(1 for g in range(10) if enter[g] <= t < done[g]) <= Fw
    # A slot freed by a completion is refilled at that same scheduling cycle.
    for g in range(Fw, 10):
        assert enter[g] in done


def test_same_training_work_in_every_mode():
    P, L = _rand(R=16, K=4, seed=9)
    kw = dict(group_size=4, update_groups=2, prompt_lens=P, resp_lens=L, max_running=12, frontier_width=2,
              step_base=0.1, step_per_ctx_token=1e-3, train_base=1.0, train_per_token=0.01, opt_step=0.5)
    comps = [sim(mode=m, **kw)["compute"] for m in ("slime", "cgp", "cgp_fgd")]
    assert comps[1] == pytest.approx(comps[0], rel=1e-14) and comps[2] == pytest.approx(comps[0], rel=1e-14)


def test_invalid_inputs_rejected():
    with pytest.raises(ValueError):
        sim(mode="cgp", group_size=2, update_groups=2, prompt_lens=[1, 1, 1], resp_lens=[1] * 6, max_running=4)
    with pytest.raises(ValueError):
        sim(mode="cgp", group_size=2, update_groups=1, prompt_lens=[1], resp_lens=[1, 0], max_running=4)
    with pytest.raises(ValueError):
        sim(mode="cgp_fgd", group_size=2, update_groups=1, prompt_lens=[1], resp_lens=[1, 1], max_running=4)
