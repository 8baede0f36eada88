#!/usr/bin/env python3
"""Benchmark: group decode attention over a paged, group-shared KV cache on one MI355X.

One step = one decode-attention pass of one layer over the whole batch: the KV
append (for workloads that carry new tokens), the work plan, the group-prefix
and response partial results (one kernel) and the LSE combine, each launched
through the C ABI on torch's current stream. The wall clock over K steps
(synchronised on both sides) gives ms_per_step; inside the timed steps only
the partial-attention kernel is bracketed by HIP events (its duration feeds
the roofline). A second, untimed pass with events between every launch gives
the per-kernel breakdown. Inputs are seeded synthetic data resident in HBM
before the timed region starts.

value = algorithmic bytes per step / step time (GB/s). Algorithmic bytes: each
group's prompt-prefix K/V once (for groups with live members), every
sequence's response K/V (including an appended token), q, out and lse, plus for
an append the new k/v read and written, plus 8 bytes of fp8 scales per
(page, kv-head) read. Plan, partial results and block tables are overhead.

Other modes, each printing its own JSON line: --prefill (the shared-prefix
prefill of the workload's prompts), --fgd (the whole decode step from the
raw projections, q/k prep included, at the frontier operating point of 2
groups x 8 live samples), --sim (rollout rounds under Slime, CGP and
CGP+FGD, simulated with decode-step costs measured on the GPU) and --grpo (the
GRPO group advantages of Eq. 1).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode-attn achieved HBM GB/s (% of MI355X peak) + seq-steps/s per layer"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, vendor figure
# Stored HBM counter summaries of the partial-attention kernel, one file per workload.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_attn_parts_{workload}.json")
# What the partial-attention kernel is built from: its source, the device helpers it includes and
# its argument structs (the counters stay valid while none of these change).
KERNEL_SOURCES = ["paper_2606_26997_amd/csrc/rp_attn.hip", "paper_2606_26997_amd/csrc/rp_device.h"]
KERNEL_STRUCTS = ("paper_2606_26997_amd/csrc/rp_internal.h", "struct AttnArgs {")


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--config", type=int, default=None,
                   help="workload number 1-5 (default: configs 3, 4, 5 on stderr, then config 2, the headline)")
    p.add_argument("--seed", type=int, default=None)
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="wall-clock budget of the oracle CPU baseline sample (0 disables it)")
    p.add_argument("--read-ceiling", action="store_true",
                   help="time plain torch streaming kernels (4 GiB sum, 1 GiB copy) as roofline context")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run only a plain device copy of known size (for HBM counter scaling)")
    p.add_argument("--prefill", action="store_true",
                   help="time the shared-prefix prefill (one prompt per group: K/V page write + causal "
                        "attention) on the workload's prompts instead of the decode step")
    p.add_argument("--prefill-len", type=int, default=None,
                   help="with --prefill: every prompt this many tokens instead of the workload's lengths")
    p.add_argument("--fgd", action="store_true",
                   help="time the whole decode step (q/k norm + rotary + append, plan, attention, combine) at "
                        "the frontier operating point: 2 groups x 8 live samples")
    p.add_argument("--sim", action="store_true",
                   help="simulate rollout rounds under Slime, CGP and CGP+FGD with decode-step costs measured "
                        "on this GPU")
    p.add_argument("--grpo", action="store_true",
                   help="time the GRPO group advantages (Eq. 1) for a paper-size round and a large batch")
    p.add_argument("--traffic-from", metavar="DIR", default=None,
                   help="summarise rocprofv3 --pmc runs under DIR (pmc_fetch, pmc_write, pmc_copy_fetch, "
                        "pmc_copy_write) into the stored HBM traffic of the partial-attention kernel")
    return p.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    path, head = KERNEL_STRUCTS
    text = open(os.path.join(ROOT, path)).read()
    i = text.index(head)
    h.update(text[i:text.index("};", i) + 2].encode())
    return h.hexdigest()[:16]


def byte_model(wl):
    """Algorithmic bytes per step, split by the kernel that moves them."""
    import numpy as np
    S, Hq, Hkv, d = wl.num_seqs, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    eb = wl.kv_elem_bytes
    tok = Hkv * d * 2 * eb                       # K + V bytes of one token, all kv-heads
    live = np.bincount(wl.seq_to_group, minlength=wl.num_groups) > 0
    P = wl.prefix_lens.astype(np.int64)
    L = wl.attn_resp_lens.astype(np.int64)
    prefix_tokens = int(P[live].sum())
    resp_tokens = int(L.sum())
    q_bytes = S * Hq * d * 2
    scale_bytes = 0
    prefix_scale = resp_scale = 0
    if wl.kv_dtype == "fp8":
        prefix_scale = int(((P[live] + 15) // 16).sum()) * Hkv * 8
        resp_scale = int(((L + 15) // 16).sum()) * Hkv * 8
        scale_bytes = prefix_scale + resp_scale
    append = 0
    if wl.append:
        append = S * Hkv * d * 2 * 2 + S * Hkv * d * 2 * eb
    out = dict(prefix_kv=prefix_tokens * tok, resp_kv=resp_tokens * tok, q=q_bytes, out=S * Hq * d * 2,
               lse=S * Hq * 4, scales=scale_bytes, append=append)
    out["total"] = sum(out.values())
    # The partial-attention kernel reads every K/V page once, their scales and q.
    out["parts_kernel"] = out["prefix_kv"] + out["resp_kv"] + scale_bytes + q_bytes
    out["prefix_tokens"], out["resp_tokens"] = prefix_tokens, resp_tokens
    # The group-prefix MFMA tile: live(g) * n_rep query rows per (group, kv-head), in 16-row tiles.
    rows = np.bincount(wl.seq_to_group, minlength=wl.num_groups)[live] * (Hq // Hkv)
    tile_rows = 16 * ((rows + 15) // 16)
    out["prefix_tile_rows"] = int(rows.sum())
    out["prefix_tile_padded_frac"] = float(1.0 - rows.sum() / tile_rows.sum()) if tile_rows.sum() else 0.0
    return out


def load_traffic(workload):
    """HBM traffic of the partial-attention kernel from stored rocprofv3 counter runs, if they
    were taken on this workload with the current kernel sources."""
    path = TRAFFIC_FILE.format(workload=workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("traffic_bytes_per_launch")


def host_cores():
    """Host cores this process may use: its CPU affinity, capped by OMP_NUM_THREADS when that is set
    (a one-GPU machine grants a share of the host's cores and sets it to that share)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp and omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(1, n)


# The forked oracle workers read the workload (and the post-append pool) that the
# parent holds; fork shares those pages, so nothing is copied or pickled.
_CPU_STATE = {}


def _oracle_worker(job):
    """One worker of the CPU baseline: the oracle on its own sequences, in order, until the budget.
    The caller has limited BLAS to one thread (a forked worker inherits that setting; it must not
    query the loaded libraries itself, which can block on a loader lock held at the fork)."""
    import oracle
    order, budget_s = job
    wl, pool = _CPU_STATE["wl"], _CPU_STATE["pool"]
    done = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        oracle.attention_for_workload(wl, seqs=[int(order[done % len(order)])], pool=pool)
        done += 1
    return done, time.perf_counter() - t0


def cpu_baseline(wl, budget_s, bytes_per_step):
    """The oracle as it stands, timed on the host: on every core this process may use (one forked
    worker per core, each on its own share of the sequences in a random order, BLAS at one thread)
    and on one core, each for a bounded wall-clock sample. Must run before the process touches the
    GPU, so that the workers are forks of a process without a device context."""
    if budget_s <= 0:
        return None
    if any(k.startswith("ROCPROF") for k in os.environ) or "rocprof" in os.environ.get("LD_PRELOAD", ""):
        # Under a profiler the preloaded library has already opened the device: no forks.
        print("[bench] under a profiler: CPU baseline skipped", file=sys.stderr, flush=True)
        return None
    import multiprocessing as mp
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle.append import append_for_workload

    pool, t_app = None, 0.0
    if wl.append:
        t0 = time.perf_counter()
        pool = append_for_workload(wl)
        t_app = time.perf_counter() - t0
    _CPU_STATE.update(wl=wl, pool=pool)
    order = np.random.default_rng(0).permutation(wl.num_seqs)
    n = min(host_cores(), wl.num_seqs)
    share = budget_s * 0.6
    with threadpool_limits(limits=1):
        with mp.get_context("fork").Pool(n) as workers:
            res = workers.map(_oracle_worker, [(order[i::n], share) for i in range(n)])
        done_one, el_one = _oracle_worker((order, budget_s - share))
    done_all = sum(r[0] for r in res)
    el_all = max(r[1] for r in res)
    _CPU_STATE.clear()
    # The append runs once per step over the whole pool; charge it per sequence-step.
    rate = lambda done, el: done / (el + t_app * done / wl.num_seqs)
    all_rate, one_rate = rate(done_all, el_all), rate(done_one, el_one)
    per_seq = bytes_per_step / wl.num_seqs
    app = ", plus the append on the whole pool" if wl.append else ""
    return {"value": round(per_seq * all_rate / 1e9, 4), "unit": "GB/s", "cores": n, "kind": "oracle",
            "sample": f"fp64 numpy oracle on {n} forked workers (one per host core, BLAS at one thread each), "
                      f"{done_all} sequence-steps in {el_all:.1f} s over the {wl.num_seqs} sequences of the "
                      f"workload in random order{app}; scaled by the step's algorithmic bytes per sequence",
            "seq_steps_per_s": round(all_rate, 3),
            "one_core": {"value": round(per_seq * one_rate / 1e9, 4), "unit": "GB/s", "cores": 1,
                         "seq_steps_per_s": round(one_rate, 3),
                         "sample": f"{done_one} sequence-steps in {el_one:.1f} s, one thread{app}"},
            "host_cores_visible": os.cpu_count()}


def _pmc_kib_per_dispatch(csv_path, kernel_substr, counter):
    import csv
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(csv_path))
            if kernel_substr in r["Kernel_Name"] and r["Counter_Name"] == counter]
    if not vals:
        raise SystemExit(f"no {counter} rows for {kernel_substr} in {csv_path}")
    return sum(vals) / len(vals), len(vals)


def summarise_traffic(root, workload):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the partial-attention kernel, scaled by the
    same counters' reading for a plain 1 GiB device copy (1 GiB read + 1 GiB written)."""
    f = lambda sub: os.path.join(root, sub, "pmc_counter_collection.csv")
    fetch, n1 = _pmc_kib_per_dispatch(f("pmc_fetch"), "attn_parts_kernel", "FETCH_SIZE")
    write, n2 = _pmc_kib_per_dispatch(f("pmc_write"), "attn_parts_kernel", "WRITE_SIZE")
    cfetch, _ = _pmc_kib_per_dispatch(f("pmc_copy_fetch"), "copyBuffer", "FETCH_SIZE")
    cwrite, _ = _pmc_kib_per_dispatch(f("pmc_copy_write"), "copyBuffer", "WRITE_SIZE")
    gib_kib = float(1 << 20)
    kf, kw = gib_kib / cfetch, gib_kib / cwrite       # true bytes per counted byte
    fetch_b, write_b = fetch * 1024 * kf, write * 1024 * kw
    out = {"kernel": "attn_parts_kernel", "workload": workload, "source_hash": kernel_source_hash(),
           "fetch_kib_per_dispatch": round(fetch, 1), "write_kib_per_dispatch": round(write, 1),
           "dispatches": [n1, n2], "copy_fetch_kib_per_GiB": round(cfetch, 1),
           "copy_write_kib_per_GiB": round(cwrite, 1), "fetch_scale": round(kf, 4), "write_scale": round(kw, 4),
           "read_bytes_per_launch": int(fetch_b), "write_bytes_per_launch": int(write_b),
           "traffic_bytes_per_launch": int(fetch_b + write_b)}
    print(json.dumps(out, indent=1))
    return out


def copy_calibration(steps):
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        b.copy_(a)
    torch.cuda.synchronize()
    el = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "ms": el * 1e3,
                      "GBps_read_plus_write": 2 * n / el / 1e9}), flush=True)


def read_ceiling(steps):
    """Context for the roofline, median over steps: the library's streaming-read probe (plain and
    non-temporal loads) and torch's own streaming kernels on this GPU. A 4 GiB read and sum, and
    a 1 GiB copy (read + write); all exceed the 256 MB last-level cache."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    x = torch.ones(1 << 31, dtype=torch.bfloat16, device="cuda")      # 4 GiB
    a = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    sink = torch.zeros(rp.RP_STREAM_READ_SINK_WORDS, dtype=torch.int32, device="cuda")
    xb = x.numel() * 2
    res = {}
    for name, fn, nbytes in (("rp_stream_read", lambda: rp.stream_read(x, xb, sink), xb),
                             ("rp_stream_read_nontemporal", lambda: rp.stream_read(x, xb, sink, nontemporal=True), xb),
                             ("sum_read", lambda: x.sum(dtype=torch.float32), xb),
                             ("copy_read_write", lambda: b.copy_(a), 2 * a.numel())):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for e0, e1 in ev:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))
        res[name] = {"bytes": nbytes, "ms": round(ms, 4), "GBps": round(nbytes / ms / 1e6, 1),
                     "frac_of_8TBps": round(nbytes / ms / 1e6 / HBM_PEAK_GBPS, 4)}
    print(json.dumps({"read_ceiling": res}), flush=True)


def stream_read_ceiling(steps=10):
    """The practical HBM read rate on this GPU: the library's streaming-read probe (non-temporal
    16-byte loads, one contiguous chunk per workgroup) over a 4 GiB buffer, median of steps."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    nbytes = 1 << 32
    x = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    sink = torch.zeros(rp.RP_STREAM_READ_SINK_WORDS, dtype=torch.int32, device="cuda")
    for _ in range(2):
        rp.stream_read(x, nbytes, sink, nontemporal=True)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in ev:
        e0.record()
        rp.stream_read(x, nbytes, sink, nontemporal=True)
        e1.record()
    torch.cuda.synchronize()
    ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))
    del x, sink
    torch.cuda.empty_cache()
    return round(nbytes / ms / 1e6, 1)


def prefill_bench(args):
    """Shared-prefix prefill: per step, every group's prompt K/V written once and causal attention."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    from workloads import CONFIGS, make_prefill_workload

    cfg = CONFIGS[args.config or 2]
    rng = np.random.default_rng(cfg.seed if args.seed is None else args.seed)
    if args.prefill_len is not None:
        P = np.full(cfg.groups, args.prefill_len)
    elif cfg.prefix[0] == "fixed":
        P = np.full(cfg.groups, cfg.prefix[1])
    else:
        P = rng.integers(cfg.prefix[1], cfg.prefix[2] + 1, cfg.groups)
    w = make_prefill_workload(num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, head_dim=cfg.head_dim,
                              prefix_lens=P, seed=cfg.seed, kv_dtype=cfg.kv_dtype, k_mult=cfg.k_mult)
    torch.cuda.set_device(0)
    b = rp.PrefillBatch.from_workload(w, device="cuda:0")
    T, Hq, Hkv, d = w.num_tokens, w.num_q_heads, w.num_kv_heads, w.head_dim
    eb = 1 if w.kv_dtype == "fp8" else 2
    P64 = P.astype(np.int64)
    # Algorithmic bytes: q, k, v read once, out written, K/V pages written (+ fp8 scales), lse.
    nbytes = T * (Hq + 2 * Hkv + Hq) * d * 2 + T * Hkv * d * 2 * eb + T * Hq * 4
    if w.kv_dtype == "fp8":
        nbytes += int(((P64 + 15) // 16).sum()) * Hkv * 8
    # Causal attention flops: QK and PV over the u <= t pairs (2 flops per multiply-add).
    flops = int((P64 * (P64 + 1) // 2).sum()) * Hq * d * 4
    # One step is rp_prefill: for a bf16 pool a single launch of the attention
    # kernel that also writes the pages; for fp8 the page-write kernel first.
    for _ in range(args.warmup):
        b.prefill()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        ev[k][0].record()
        b.prefill()
        ev[k][1].record()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    attn_us = float(np.mean([a.elapsed_time(c) for a, c in ev])) * 1e3
    # The timed call's bytes: q, k, v read, out and lse written, and the pages
    # written (bf16: by the attention launch itself; fp8: by the page-write
    # kernel that runs first, which reads k and v once more and writes the
    # codes and the per-(page, kv-head) scales).
    attn_bytes = T * (Hq + 2 * Hkv + Hq) * d * 2 + T * Hq * 4 + T * Hkv * d * 2 * eb
    if eb == 1:
        attn_bytes += T * Hkv * d * 2 * 2 + int(((P64 + 15) // 16).sum()) * Hkv * 8
    # Below the bf16 ridge (about 310 flop/B) the kernel is priced against HBM
    # bandwidth, above it against the dense bf16 MFMA peak.
    gbps_attn = attn_bytes / (attn_us * 1e-6) / 1e9
    tflops_attn = flops / (attn_us * 1e-6) / 1e12
    kname = "prefill_attn_kernel" if eb == 2 else "prefill_kv_write_kernel + prefill_attn_kernel"
    if flops / attn_bytes < 310:
        roof = {"kernel": kname, "bound": "hbm", "achieved": round(gbps_attn, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps_attn / HBM_PEAK_GBPS, 4)}
    else:
        roof = {"kernel": kname, "bound": "mfma", "achieved": round(tflops_attn, 1),
                "peak": 2500.0, "unit": "TFLOP/s", "frac": round(tflops_attn / 2500.0, 4)}
    roof.update({"traffic": None, "algorithmic_bytes_per_launch": int(attn_bytes), "flops_per_launch": flops,
                 "mfma_frac": round(tflops_attn / 2500.0, 4)})
    line = {
        "metric": "shared-prefix prefill: prompt tokens/s and achieved HBM GB/s (one prompt per group)",
        "value": round(T / (ms * 1e-3), 1), "unit": "prompt tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.kv_dtype, "data": "synthetic",
        "config": {"workload": f"config{cfg.cid} prompts" + (f" of {args.prefill_len} tokens" if args.prefill_len else ""),
                   "groups": int(cfg.groups), "prompt_tokens": T, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
                   "kv_dtype": w.kv_dtype},
        "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1), "attn_tflops": round(flops / (attn_us * 1e-6) / 1e12, 2),
        "attn_us": round(attn_us, 2),
        "roofline": roof,
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def _model_step_ms(b, steps, layers=None, min_bytes=2e9):
    """One decode step of a model: one plan (the lengths are shared by all layers), then per layer
    q/k prep, partial attention and combine. Layers cycle through enough copies of the K/V pool
    (same page layout) that the K/V read per step exceeds `min_bytes`, so that, unlike one layer
    repeated, they come from HBM rather than the 256 MB last-level cache."""
    import torch
    import paper_2606_26997_amd as rp
    layers = QWEN3_LAYERS if layers is None else layers
    pool_bytes = 2 * b.k_pages.numel() * b.k_pages.element_size()
    copies = int(min(layers, max(1, -(-min_bytes // pool_bytes))))
    pools = [(b.k_pages, b.v_pages)] + [(b.k_pages.clone(), b.v_pages.clone()) for _ in range(copies - 1)]
    kvs = [rp.paged_kv(kp, vp) for kp, vp in pools]

    def model_step():
        # The first layer's prep also plans the step (one launch for small batches).
        for l in range(layers):
            kv = kvs[l % copies]
            if l == 0:
                rp.decode_qk_prep_plan(kv, b.append_layout, b.q_in, b.k_in, b.v_in, b.q_norm_w, b.k_norm_w, b.q,
                                       None, b.workspace)
            else:
                rp.decode_qk_prep(kv, b.append_layout, b.q_in, b.k_in, b.v_in, b.q_norm_w, b.k_norm_w, b.q, None)
            rp.attn_parts(kv, b.attn_layout, b.q, b.softmax_scale, b.workspace)
            rp.combine_parts(kv, b.attn_layout, b.out, b.lse, b.workspace)

    for _ in range(2):
        model_step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        model_step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps * 1e3, copies


FGD_GROUPS, FGD_LIVE, FGD_PREFIX, FGD_RESP_MAX = 2, 8, 512, 6016


def fgd_bench(args):
    """One decode step of one layer at the frontier operating point.

    Frontier-group dispatch keeps F_w = 2 groups of K = 8 samples in flight, so
    the live batch is 16 sequences. Each group has a 512-token prompt; the
    responses are uniform in [0, 6016], about 3.5k tokens of context per
    sequence on average. Qwen3-1.7B layer shape, bf16 KV. A step starts from
    the raw projections: q/k RMS norm and rotary embedding with the k/v append
    and the plan (one launch), then the partial results and the combine.
    """
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    from workloads import make_qkprep_inputs, make_workload

    seed = 2026 if args.seed is None else args.seed
    rng = np.random.default_rng(seed)
    S = FGD_GROUPS * FGD_LIVE
    resp = rng.integers(0, FGD_RESP_MAX + 1, S)
    wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.repeat(np.arange(FGD_GROUPS), FGD_LIVE),
                       prefix_lens=np.full(FGD_GROUPS, FGD_PREFIX), resp_lens=resp, seed=seed, append=True,
                       k_mult=0.5, rng=rng)
    x = make_qkprep_inputs(num_seqs=S, num_q_heads=16, num_kv_heads=8, head_dim=128, seed=seed + 1)
    torch.cuda.set_device(0)
    b = rp.DeviceBatch.from_workload(wl, device="cuda:0")
    b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w)
    bm = byte_model(wl)
    prep_extra = 2 * S * wl.num_q_heads * wl.head_dim * 2      # raw q read and prepared q written
    total = bm["total"] + prep_extra
    # rp_decode_qk_prep_plan: the prep and the plan of the step in one launch.
    stages = ["prep+plan", "parts", "combine"]
    calls = {"prep+plan": b.qk_prep_plan, "parts": b.attn_parts, "combine": b.combine_parts}

    def step(evs=None):
        for i, name in enumerate(stages):
            if evs is not None:
                evs[i].record()
            calls[name]()
        if evs is not None:
            evs[len(stages)].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(args.steps)]
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    per = {name: float(np.mean([events[k][i].elapsed_time(events[k][i + 1]) for k in range(args.steps)])) * 1e3
           for i, name in enumerate(stages)}
    parts_us = per["parts"]
    achieved = bm["parts_kernel"] / (parts_us * 1e-6) / 1e9

    # A whole model step (see _model_step_ms): K/V from HBM, one plan per step.
    model_ms, copies = _model_step_ms(b, max(args.steps // 10, 5))
    layer_bytes = total

    # The prep kernel alone on a large batch (4096 sequences, one response page
    # each): q read and written, k and v read and appended.
    S2 = 4096
    wl2 = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.arange(S2) // 8,
                        prefix_lens=np.full(S2 // 8, 16), resp_lens=rng.integers(0, 15, S2), seed=seed + 2,
                        append=True, rng=rng)
    x2 = make_qkprep_inputs(num_seqs=S2, num_q_heads=16, num_kv_heads=8, head_dim=128, seed=seed + 3)
    b2 = rp.DeviceBatch.from_workload(wl2, device="cuda:0")
    b2.set_projections(x2.q_in, x2.k_in, x2.v_in, x2.q_norm_w, x2.k_norm_w)
    for _ in range(args.warmup):
        b2.qk_prep()
    ev2 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, c in ev2:
        a.record()
        b2.qk_prep()
        c.record()
    torch.cuda.synchronize()
    prep_us = float(np.mean([a.elapsed_time(c) for a, c in ev2])) * 1e3
    prep_bytes = S2 * (2 * 16 + 4 * 8) * 128 * 2
    line = {
        "metric": "decode step at the frontier operating point: seq-steps/s per layer and achieved HBM GB/s",
        "value": round(S / (ms * 1e-3), 1), "unit": "seq-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"frontier batch: {FGD_GROUPS} groups x {FGD_LIVE} live samples, prompt "
                               f"{FGD_PREFIX}, responses uniform [0, {FGD_RESP_MAX}]",
                   "seqs": S, "q_heads": 16, "kv_heads": 8, "head_dim": 128, "kv_dtype": "bf16",
                   "prefix_tokens": bm["prefix_tokens"], "resp_tokens": bm["resp_tokens"], "seed": seed},
        "GBps": round(total / (ms * 1e-3) / 1e9, 1), "algorithmic_bytes_per_step": int(total),
        "kernel_us": {k: round(v, 2) for k, v in per.items()},
        "model_step": {"layers": QWEN3_LAYERS, "kv_pool_copies": copies, "ms": round(model_ms, 4),
                       "per_layer_us": round(model_ms * 1e3 / QWEN3_LAYERS, 2),
                       "seq_steps_per_s": round(S / (model_ms * 1e-3), 1),
                       "GBps": round(QWEN3_LAYERS * layer_bytes / (model_ms * 1e-3) / 1e9, 1)},
        "prep_4096_seqs": {"us": round(prep_us, 2), "bytes": prep_bytes,
                           "GBps": round(prep_bytes / (prep_us * 1e-6) / 1e9, 1)},
        "roofline": {"kernel": "attn_parts_kernel", "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": None, "algorithmic_bytes_per_launch": int(bm["parts_kernel"])},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


# Qwen3-1.7B: 28 layers, 8 kv-heads of 128 channels; 1.7e9 parameters.
QWEN3_LAYERS, QWEN3_PARAMS = 28, 1.7e9
KV_BYTES_PER_TOKEN = QWEN3_LAYERS * 8 * 128 * 2 * 2       # bf16 K and V of one token, all layers
GEMM_FLOPS = 0.5 * 2.5e15                                  # assumed: projections and MLP at half the bf16 peak
PAPER_TRAIN_R96 = 587.4                                    # trainer compute, LSAT-AR, R = 96, Slime (Table 1)
PAPER_ROLLOUT_R96 = 525.0                                  # mid-range of Slime's first dispatch at R = 96 (509-543 s)


def _measure_decode_step(args, rng):
    """Attention part of a whole-model decode step (one plan, then per layer q/k prep, partial
    attention and combine; K/V from HBM) at several batch shapes, fitted as
    a + b * sequences + c * context tokens (context counted per sequence, prompt included)."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    from workloads import make_qkprep_inputs, make_workload
    rows, times = [], []
    for S, rmax in ((16, 6016), (64, 6016), (256, 6016), (64, 2000), (256, 12000)):
        resp = rng.integers(0, rmax + 1, S)
        wl = make_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, seq_to_group=np.arange(S) // 8,
                           prefix_lens=np.full(S // 8, 512), resp_lens=resp, seed=int(S + rmax), append=True,
                           k_mult=0.5, rng=rng)
        x = make_qkprep_inputs(num_seqs=S, num_q_heads=16, num_kv_heads=8, head_dim=128, seed=S)
        b = rp.DeviceBatch.from_workload(wl, device="cuda:0")
        b.set_projections(x.q_in, x.k_in, x.v_in, x.q_norm_w, x.k_norm_w)
        ms, _ = _model_step_ms(b, 5)
        times.append(ms * 1e-3)
        rows.append([1.0, S, float(512 * S + resp.sum() + S)])
        del b
        torch.cuda.empty_cache()
    coef, *_ = np.linalg.lstsq(np.array(rows), np.array(times), rcond=None)
    return [float(c) for c in coef], [dict(seqs=int(r[1]), ctx_tokens=int(r[2]), ms=round(t * 1e3, 4))
                                      for r, t in zip(rows, times)]


def _measure_prefill_token():
    """Per-layer prefill time per prompt token (page write + causal attention), 32 prompts of 600 tokens."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    from workloads import make_prefill_workload
    w = make_prefill_workload(num_q_heads=16, num_kv_heads=8, head_dim=128, prefix_lens=[600] * 32, seed=5)
    b = rp.PrefillBatch.from_workload(w, device="cuda:0")
    for _ in range(5):
        b.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(20):
        b.step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / 20 / w.num_tokens


def _measure_weight_read():
    """Time to read the model's weight bytes once from HBM (what a small-batch decode step pays)."""
    import torch
    w = torch.ones(int(QWEN3_PARAMS), dtype=torch.bfloat16, device="cuda:0")
    for _ in range(3):
        w.sum()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(10):
        w.sum()
    torch.cuda.synchronize()
    el = (time.perf_counter() - t0) / 10
    del w
    return el


def sim_bench(args):
    """Rollout rounds of R groups x K = 8 under Slime, CGP and CGP+FGD (U = 2, F_w = 2), simulated by
    rp_sched_simulate with decode-step costs measured on this GPU."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp
    import oracle
    from workloads import make_rollout_workload

    torch.cuda.set_device(0)
    rng = np.random.default_rng(77 if args.seed is None else args.seed)
    (a, b, c), points = _measure_decode_step(args, rng)
    pre_tok = _measure_prefill_token()
    t_w = _measure_weight_read()
    per_tok_gemm = 2 * QWEN3_PARAMS / GEMM_FLOPS
    cost = dict(step_base=max(a, 0.0) + t_w, step_per_seq=max(b, 0.0) + per_tok_gemm,
                step_per_ctx_token=max(c, 0.0), prefill_per_token=QWEN3_LAYERS * pre_tok + per_tok_gemm)
    K, U, Fw, P_MAX, CAP = 8, 2, 2, 1024, 8192

    # Concurrency from the KV memory left after the weights, at the average context of a request
    # (prompt plus response), as a serving engine admits against current usage.
    P96, L96 = make_rollout_workload(num_groups=96, group_size=K, seed=96, prompt_max=P_MAX, resp_cap=CAP)
    avg_ctx = float(P96.mean() + L96.mean())

    def capacity(hbm_bytes):
        return int((0.9 * hbm_bytes - 2 * QWEN3_PARAMS) // (KV_BYTES_PER_TOKEN * avg_ctx))

    def rounds(scale, cap):
        out = {}
        for R in (32, 64, 96):
            P, L = make_rollout_workload(num_groups=R, group_size=K, seed=R, prompt_max=P_MAX, resp_cap=CAP)
            # Trainer speed from the paper's trainer compute at R = 96, per trained token.
            P96, L96 = make_rollout_workload(num_groups=96, group_size=K, seed=96, prompt_max=P_MAX, resp_cap=CAP)
            tpt = PAPER_TRAIN_R96 / float(K * P96.astype(np.int64).sum() + L96.astype(np.int64).sum())
            kw = dict(group_size=K, update_groups=U, prompt_lens=P, resp_lens=L, max_running=cap, frontier_width=Fw,
                      mat_base=1.0, train_per_token=tpt, **{k: v * scale for k, v in cost.items()})
            res = {m: rp.sched_simulate(mode=m, **kw) for m in ("slime", "cgp", "cgp_fgd")}
            sl = res["slime"]["t_train_end"]
            out[f"R{R}"] = {m: dict(train_end_s=round(r["t_train_end"], 2),
                                    reduction_vs_slime_pct=round(100 * (1 - r["t_train_end"] / sl), 2),
                                    first_dispatch_s=round(r["t_start"], 2), rollout_s=round(r["t_complete"], 2),
                                    w_train=round(r["w_train"], 4), wait_ratio=round(r["wait_ratio"], 4))
                            for m, r in res.items()}
            out[f"R{R}"]["fgd_gain_over_cgp_pct"] = round(
                100 * (1 - res["cgp_fgd"]["t_train_end"] / res["cgp"]["t_train_end"]), 2)
        return out

    cap_mi355x, cap_a100 = capacity(288e9), capacity(2 * 40e9)
    mi = rounds(1.0, cap_mi355x)
    # The paper's rollout regime: the same cost model slowed down until Slime's R = 96 rollout
    # ends where the paper's first dispatch does, with the KV capacity of 2 x A100 40 GB.
    base = rp.sched_simulate(mode="slime", group_size=K, update_groups=U, prompt_lens=P96, resp_lens=L96,
                             max_running=cap_a100, **cost)
    alpha = PAPER_ROLLOUT_R96 / max(base["serve_done"])
    paper = rounds(alpha, cap_a100)

    # Frontier width against the trainer's supply, R = 96, both regimes.
    tpt96 = PAPER_TRAIN_R96 / float(K * P96.astype(np.int64).sum() + L96.astype(np.int64).sum())
    sweep = {}
    for name, scale, cap in (("mi355x_rollout", 1.0, cap_mi355x), ("paper_regime", alpha, cap_a100)):
        sweep[name] = {}
        for fw in (2, 4, 8, 16):
            r = rp.sched_simulate(mode="cgp_fgd", group_size=K, update_groups=U, prompt_lens=P96, resp_lens=L96,
                                  max_running=cap, frontier_width=fw, mat_base=1.0, train_per_token=tpt96,
                                  **{k: v * scale for k, v in cost.items()})
            sweep[name][f"Fw{fw}"] = dict(train_end_s=round(r["t_train_end"], 2), first_dispatch_s=round(r["t_start"], 2),
                                         rollout_s=round(r["t_complete"], 2), wait_ratio=round(r["wait_ratio"], 4))

    # Speed of the native simulation against the step-by-step oracle, same round.
    kw = dict(group_size=K, update_groups=U, prompt_lens=P96, resp_lens=L96, max_running=cap_a100, frontier_width=Fw,
              **{k: v * alpha for k, v in cost.items()})
    t0 = time.perf_counter()
    for _ in range(20):
        rp.sched_simulate(mode="cgp_fgd", **kw)
    native_s = (time.perf_counter() - t0) / 20
    t0 = time.perf_counter()
    ref = oracle.simulate_schedule(mode="cgp_fgd", **kw)
    oracle_s = time.perf_counter() - t0
    assert ref["t_train_end"] == rp.sched_simulate(mode="cgp_fgd", **kw)["t_train_end"]

    val = mi["R96"]["cgp_fgd"]["reduction_vs_slime_pct"]
    line = {
        "metric": "simulated rollout-to-train-end reduction of CGP+FGD vs Slime (R=96, K=8, U=2, F_w=2), "
                  "decode-step costs measured on MI355X",
        "value": val, "unit": "%", "n_gpus": 1, "steps": None, "warmup": None, "ms_per_step": None,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "rollout rounds of R = 32/64/96 groups x 8 samples, prompts U[128, 1024], "
                               "responses lognormal (median 3000; group sigma 0.5, sample sigma 0.3; cap 8192)",
                   "max_running_mi355x": cap_mi355x, "max_running_2xA100": cap_a100},
        "cost_model": {k: float(f"{v:.6g}") for k, v in cost.items()},
        "measured": {"decode_step_fit_us": {"base": round(a * 1e6, 3), "per_seq": round(b * 1e6, 5),
                                            "per_ctx_token": round(c * 1e6, 8)},
                     "decode_step_points": points, "prefill_layer_us_per_token": round(pre_tok * 1e6, 5),
                     "weight_read_ms": round(t_w * 1e3, 4)},
        "assumed": {"gemm_flops": GEMM_FLOPS, "materialise_s_per_group": 1.0,
                    "trainer_s_per_token_from_paper_R96": PAPER_TRAIN_R96},
        "mi355x_rollout": mi,
        "paper_regime": {"rollout_slowdown": round(alpha, 3), **paper},
        "frontier_width_sweep_R96": sweep,
        "paper_context": {"reduction_vs_slime_pct_R96": [39.8, 42.3], "first_dispatch_s_R96_cgp": [46, 90],
                          "first_dispatch_s_R96_cgp_fgd": [52, 61], "wait_ratio_R96_pct": [13.8, 15.0],
                          "fgd_gain_over_cgp_pct": [2.5, 11.4]},
        "simulator_s_per_round": round(native_s, 6),
        "cpu_baseline": {"value": round(oracle_s, 3), "unit": "s per round", "cores": 1, "kind": "oracle",
                         "sample": "the same R = 96 CGP+FGD round, simulated one decode step at a time"},
    }
    print(json.dumps(line), flush=True)


def grpo_bench(args):
    """GRPO advantages (Eq. 1): one round of the paper (R = 96 groups of K = 8) and 2^22 groups of 8."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp

    torch.cuda.set_device(0)
    res = {}
    for name, R in (("round_R96", 96), ("batch_2^22", 1 << 22)):
        K = 8
        r = torch.from_numpy(np.random.default_rng(R).standard_normal((R, K)).astype(np.float32)).cuda()
        adv = torch.empty_like(r)
        mu = torch.empty(R, dtype=torch.float32, device="cuda")
        sd = torch.empty(R, dtype=torch.float32, device="cuda")
        for _ in range(args.warmup):
            rp.grpo_advantage(r, adv, mu, sd)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for a, b in ev:
            a.record()
            rp.grpo_advantage(r, adv, mu, sd)
            b.record()
        torch.cuda.synchronize()
        us = float(np.mean([a.elapsed_time(b) for a, b in ev])) * 1e3
        nbytes = R * K * 4 * 2 + R * 8          # rewards read, advantages written, mean and std written
        res[name] = dict(groups=R, group_size=K, us=round(us, 2), bytes=nbytes,
                         GBps=round(nbytes / (us * 1e-6) / 1e9, 1))
    big = res["batch_2^22"]
    line = {
        "metric": "GRPO group advantages (Eq. 1): achieved HBM GB/s on 2^22 groups of 8",
        "value": big["GBps"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(big["us"] / 1e3, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": "rewards N(0, 1) in groups of 8: 2^22 groups, and one round of 96 groups"},
        "runs": res,
        "roofline": {"kernel": "grpo_fixed_kernel<8>", "bound": "hbm", "achieved": big["GBps"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(big["GBps"] / HBM_PEAK_GBPS, 4), "traffic": None,
                     "algorithmic_bytes_per_launch": big["bytes"]},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU; --gpus {args.gpus} is not supported "
              f"(the attention shards exchange-free by whole groups, see the design notes).",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if args.copy_calibration:
        copy_calibration(args.steps)
        return
    if args.read_ceiling:
        read_ceiling(args.steps)
        return
    if args.traffic_from:
        summarise_traffic(args.traffic_from, f"config{args.config or 2}")
        return
    if args.prefill:
        prefill_bench(args)
        return
    if args.fgd:
        fgd_bench(args)
        return
    if args.sim:
        sim_bench(args)
        return
    if args.grpo:
        grpo_bench(args)
        return

    from workloads import CONFIGS, make_config_workload

    # Phase 1, host only: every workload and its oracle CPU baseline, before anything touches the
    # GPU (the baseline forks its workers). The headline workload is config 2, the Qwen3-1.7B
    # layer shape; the default run also reports configs 3-5 (one line each on stderr, first).
    cids = [args.config] if args.config is not None else [3, 4, 5, 2]
    prepared = []
    for cid in cids:
        cfg = CONFIGS[cid]
        t0 = time.perf_counter()
        wl = make_config_workload(cfg, seed=args.seed)
        print(f"[bench] config{cid} generated in {time.perf_counter() - t0:.1f}s: {wl.num_seqs} seqs, "
              f"{wl.num_pages} pages", file=sys.stderr, flush=True)
        cpu = None
        if args.cpu_seconds > 0:
            budget = args.cpu_seconds if cid == cids[-1] else args.cpu_seconds / 2
            t0 = time.perf_counter()
            cpu = cpu_baseline(wl, budget, byte_model(wl)["total"])
            if cpu is not None:
                print(f"[bench] config{cid} oracle CPU baseline: {cpu['value']} GB/s on {cpu['cores']} cores "
                      f"({time.perf_counter() - t0:.1f}s)", file=sys.stderr, flush=True)
        prepared.append((cfg, wl, cpu))

    # Phase 2: the GPU, one workload at a time, after the practical read ceiling.
    args.read_ceiling_gbps = stream_read_ceiling()
    print(f"[bench] streaming-read ceiling: {args.read_ceiling_gbps} GB/s", file=sys.stderr, flush=True)
    for i, (cfg, wl, cpu) in enumerate(prepared):
        line = decode_bench(cfg, wl, cpu, args)
        prepared[i] = None
        del wl
        last = i == len(prepared) - 1
        print(json.dumps(line), file=sys.stdout if last else sys.stderr, flush=True)


def decode_bench(cfg, wl, cpu, args):
    """One workload's decode-attention step on the GPU: timed steps, per-kernel breakdown, roofline."""
    import numpy as np
    import torch
    import paper_2606_26997_amd as rp

    torch.cuda.set_device(0)
    batch = rp.DeviceBatch.from_workload(wl, device="cuda:0")
    bm = byte_model(wl)

    stages = (["append"] if wl.append else []) + ["plan", "parts", "combine"]
    calls = {"append": batch.kv_append, "plan": batch.plan, "parts": batch.attn_parts,
             "combine": batch.combine_parts}

    def step(evs=None, only_parts=False):
        for i, name in enumerate(stages):
            if evs is not None and (not only_parts or name == "parts"):
                evs[i].record()
            calls[name]()
            if evs is not None and only_parts and name == "parts":
                evs[i + 1].record()
        if evs is not None and not only_parts:
            evs[len(stages)].record()

    def new_events():
        return [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
                for _ in range(args.steps)]

    ip = stages.index("parts")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = new_events()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k], only_parts=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall / args.steps * 1e3
    parts_samples = np.array([events[k][ip].elapsed_time(events[k][ip + 1]) for k in range(args.steps)]) * 1e3
    parts_us = float(parts_samples.mean())

    # Untimed breakdown pass: events between every launch.
    events = new_events()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    samples = {name: np.array([events[k][i].elapsed_time(events[k][i + 1]) for k in range(args.steps)]) * 1e3
               for i, name in enumerate(stages)}      # microseconds
    samples["step"] = np.array([events[k][0].elapsed_time(events[k][-1]) for k in range(args.steps)]) * 1e3
    per_kernel = {name: float(samples[name].mean()) for name in stages}
    event_step_us = float(samples["step"].mean())
    samples["parts_timed"] = parts_samples
    spread = {name: {"median": round(float(np.median(v)), 2), "p10": round(float(np.percentile(v, 10)), 2),
                     "p90": round(float(np.percentile(v, 90)), 2)} for name, v in samples.items()}
    del batch
    torch.cuda.empty_cache()

    gbps = bm["total"] / (ms_per_step * 1e-3) / 1e9
    achieved = bm["parts_kernel"] / (parts_us * 1e-6) / 1e9
    traffic = load_traffic(f"config{cfg.cid}") if args.seed is None else None
    rc = getattr(args, "read_ceiling_gbps", None)
    # Context, not the roofline's peak: the kernel's rate against what a plain streaming read reaches.
    ceiling = {"GBps": rc, "frac": round(achieved / rc, 4), "probe": "rp_stream_read, 4 GiB, non-temporal loads"} \
        if rc else None
    return {
        "metric": METRIC,
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.kv_dtype,
        "data": "synthetic",
        "config": {"workload": f"config{cfg.cid}: {cfg.name}", "seqs": wl.num_seqs,
                   "groups": wl.num_groups, "q_heads": wl.num_q_heads, "kv_heads": wl.num_kv_heads,
                   "head_dim": wl.head_dim, "page_size": wl.page_size, "kv_dtype": wl.kv_dtype,
                   "append": wl.append, "prefix_tokens": bm["prefix_tokens"],
                   "resp_tokens": bm["resp_tokens"], "seed": cfg.seed if args.seed is None else args.seed},
        "pct_of_hbm_peak": round(100.0 * gbps / HBM_PEAK_GBPS, 2),
        "seq_steps_per_s": round(wl.num_seqs / (ms_per_step * 1e-3), 1),
        "algorithmic_bytes_per_step": int(bm["total"]),
        "prefix_tile_padded_rows_frac": round(bm["prefix_tile_padded_frac"], 4),
        "kernel_us": {k: round(v, 2) for k, v in per_kernel.items()},
        "event_step_us": round(event_step_us, 2),
        "parts_kernel_us_timed": round(parts_us, 2),
        "kernel_us_spread": spread,
        "roofline": {"kernel": "attn_parts_kernel", "bound": "hbm", "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "algorithmic_bytes_per_launch": int(bm["parts_kernel"]),
                     "read_ceiling": ceiling},
        "cpu_baseline": cpu,
    }


if __name__ == "__main__":
    main()
