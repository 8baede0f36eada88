"""Complete-group pipelining (CGP) and frontier-group dispatch (FGD), simulated step by step.

TEST INFRASTRUCTURE ONLY (see the package docstring). A plain, slow
simulation of one rollout round and its training, written from Sections
3.2-3.3 and Algorithm 1 of the paper; every decode step is taken one at a
time.

Rollout node. R groups of K requests; request ``q = g K + i`` belongs to group
``g`` (submission order = group index) and must generate ``resp_lens[q] >= 1``
tokens after its group's prompt of ``prompt_lens[g]`` tokens. At every
scheduling cycle (a decode-step boundary):

* FGD admission (mode ``cgp_fgd``, Eq. 5-6 and Algorithm 1): while the frontier
  holds fewer than F_w groups and groups remain deferred, the lowest-order
  deferred group joins the frontier and its K requests join the admitted
  queue. Otherwise (``slime``, ``cgp``) all R K requests are in the admitted
  queue from the start, group by group (request-level FIFO).
* The engine moves admitted requests, first come first served, into the
  running set while it holds fewer than ``max_running``. The first request of
  a group to run brings its group's prompt prefill into that step.
* One decode step: every running request generates one token. The step lasts
  ``step_base + step_per_seq * n + step_per_ctx_token * ctx + prefill`` with
  ``n`` running requests, ``ctx`` the sum of their context lengths (prompt plus
  tokens generated so far) before the step, and ``prefill`` the sum of
  ``prefill_per_token * prompt_lens[g]`` over groups started in this cycle.
* Requests that reach their length finish at the end of the step; a group is
  serving-complete when all K have finished, and it leaves the frontier.

Control node. A serving-complete group is trainable-complete after
``mat_base + mat_per_token * (its response tokens)`` (reward, verification,
materialisation) and enters the trainer FIFO; FIFO order is by
trainable-complete time, ties by group order.

Training node. Update ``k`` consumes FIFO entries ``kU .. kU + U - 1``; its
duration is the sum over its groups of ``train_base + train_per_token *
(prompt and response tokens of the group's K samples)``, plus ``opt_step``. It
starts when the trainer is free and its data is there: the U-th group of the
batch has arrived (``cgp``, ``cgp_fgd``; Eq. 2 right), or every group of the
round has (``slime``; Eq. 2 left).

Metrics: ``t_first_u`` (time the first U groups are all trainable, the U-th
FIFO entry), ``t_complete`` (the last group trainable), ``t_start`` (first
update start), ``delta_cgp = t_complete - t_first_u`` (Eq. 3), ``t_train_end``
(end of the last update), ``w_train = (t_start - 0) / (t_train_end - 0)``
(Eq. 4, rollout start at 0), and the trainer-side waiting ratio of the
evaluation, ``wait / (wait + compute)`` with ``compute`` the summed update
durations and ``wait`` the trainer's idle time in ``[0, t_train_end]``.

All times are float64 seconds. Sums are accumulated in the order stated
above, so a faithful implementation reproduces every value bit for bit.
"""
from collections import deque

MODES = ("slime", "cgp", "cgp_fgd")


def simulate(*, mode, group_size, update_groups, prompt_lens, resp_lens, max_running, frontier_width=0,
             step_base=0.0, step_per_seq=0.0, step_per_ctx_token=0.0, prefill_per_token=0.0,
             mat_base=0.0, mat_per_token=0.0, train_base=0.0, train_per_token=0.0, opt_step=0.0):
    if mode not in MODES:
        raise ValueError(f"mode {mode!r}")
    K, U = int(group_size), int(update_groups)
    P = [int(x) for x in prompt_lens]
    L = [int(x) for x in resp_lens]
    R = len(P)
    if K < 1 or U < 1 or R < 1 or len(L) != R * K or R % U or max_running < 1 or min(L) < 1 or min(P) < 0:
        raise ValueError("invalid simulation inputs")
    if mode == "cgp_fgd" and frontier_width < 1:
        raise ValueError("frontier_width must be >= 1 for cgp_fgd")

    # ---- rollout node -------------------------------------------------------
    admitted = deque(range(R * K)) if mode != "cgp_fgd" else deque()
    deferred = deque(range(R))                 # FGD: groups not yet in the frontier, by order
    frontier = set()
    frontier_enter = [0.0] * R
    running = []                               # request ids in admission order
    generated = [0] * (R * K)
    started = [False] * R
    left = [K] * R                             # unfinished requests per group
    serve_done = [None] * R
    t = 0.0
    steps = 0
    while True:
        if mode == "cgp_fgd":
            while len(frontier) < frontier_width and deferred:
                g = deferred.popleft()
                frontier.add(g)
                frontier_enter[g] = t
                admitted.extend(g * K + i for i in range(K))
        prefill = 0.0
        while len(running) < max_running and admitted:
            q = admitted.popleft()
            running.append(q)
            g = q // K
            if not started[g]:
                started[g] = True
                prefill += prefill_per_token * P[g]
        if not running:
            break
        n = len(running)
        ctx = sum(P[q // K] + generated[q] for q in running)
        t += step_base + step_per_seq * n + step_per_ctx_token * ctx + prefill
        steps += 1
        still = []
        for q in running:
            generated[q] += 1
            if generated[q] < L[q]:
                still.append(q)
                continue
            g = q // K
            left[g] -= 1
            if left[g] == 0:
                serve_done[g] = t
                frontier.discard(g)
        running = still

    # ---- control node -------------------------------------------------------
    resp_tok = [sum(L[g * K:(g + 1) * K]) for g in range(R)]
    trainable = [serve_done[g] + (mat_base + mat_per_token * resp_tok[g]) for g in range(R)]
    fifo = sorted(range(R), key=lambda g: (trainable[g], g))

    # ---- training node ------------------------------------------------------
    comp = [train_base + train_per_token * (K * P[g] + resp_tok[g]) for g in range(R)]
    t_complete = max(trainable)
    free = 0.0
    starts, ends = [], []
    compute = 0.0
    for k in range(R // U):
        batch = fifo[k * U:(k + 1) * U]
        avail = t_complete if mode == "slime" else trainable[batch[-1]]
        start = max(free, avail)
        dur = 0.0
        for g in batch:
            dur += comp[g]
        dur += opt_step
        free = start + dur
        compute += dur
        starts.append(start)
        ends.append(free)
    t_first_u = trainable[fifo[U - 1]]
    t_train_end = free
    wait = t_train_end - compute
    return dict(serve_done=serve_done, frontier_enter=frontier_enter if mode == "cgp_fgd" else [0.0] * R,
                trainable=trainable, fifo=fifo, update_start=starts, update_end=ends, steps=steps,
                t_first_u=t_first_u, t_complete=t_complete, t_start=starts[0], delta_cgp=t_complete - t_first_u,
                t_train_end=t_train_end, compute=compute, wait=wait,
                w_train=starts[0] / t_train_end if t_train_end > 0 else 0.0,
                wait_ratio=wait / t_train_end if t_train_end > 0 else 0.0)
