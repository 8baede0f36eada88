"""Shared helpers for GPU parity tests: run the HIP path, run the oracle, compare."""
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
from oracle.append import append_for_workload

# Contract tolerances for the bf16 output / natural-log lse, and tighter internal
# gates (relative L2 of the output, lse) that catch a skipped page even where the
# max-abs contract is loose for long key sets.
TOL = {"bf16": dict(max_abs=1e-2, lse=1e-3, rel_l2=5e-3, lse_tight=1e-4),
       "fp8": dict(max_abs=3e-2, lse=1e-3, rel_l2=5e-3, lse_tight=1e-4)}


def gpu_available():
    return torch.cuda.is_available()


def to_host_out(batch):
    torch.cuda.synchronize()
    out = batch.out.float().cpu().numpy().astype(np.float64)
    lse = batch.lse.cpu().numpy().astype(np.float64)
    return out, lse


def run_hip(wl, batch=None):
    import paper_2606_26997_amd as rp
    if batch is None:
        batch = rp.DeviceBatch.from_workload(wl)
    batch.step()
    out, lse = to_host_out(batch)
    return batch, out, lse


def run_oracle(wl, seqs=None):
    pool = append_for_workload(wl) if wl.append else None
    out, lse = oracle.attention_for_workload(wl, seqs=seqs, pool=pool)
    return out, lse, pool


def oracle_threads():
    """Oracle worker threads: the host's CPU share (16 on a one-GPU machine), at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n, int(os.environ.get("OMP_NUM_THREADS", n))))


def run_oracle_all(wl, pool=None, chunk=16, label=""):
    """Oracle result for every sequence of ``wl``, computed in chunks of sequences by a thread pool
    over the one host copy of the pool (numpy's gathers and BLAS calls release the GIL for part of
    the work). Prints a progress line per quarter so that a long comparison is visibly alive."""
    from threadpoolctl import threadpool_limits
    if wl.append and pool is None:
        pool = append_for_workload(wl)
    S = wl.num_seqs
    chunks = [list(range(i, min(S, i + chunk))) for i in range(0, S, chunk)]
    out = np.zeros((S, wl.num_q_heads, wl.head_dim))
    lse = np.full((S, wl.num_q_heads), -np.inf)
    t0 = time.perf_counter()
    done = 0
    with threadpool_limits(limits=1), ThreadPoolExecutor(oracle_threads()) as ex:
        futs = [(c, ex.submit(oracle.attention_for_workload, wl, seqs=c, pool=pool)) for c in chunks]
        for i, (c, f) in enumerate(futs):
            o, l = f.result()
            out[c[0]:c[-1] + 1], lse[c[0]:c[-1] + 1] = o, l
            done += len(c)
            if (i + 1) % max(1, len(futs) // 4) == 0 or i + 1 == len(futs):
                print(f"[oracle] {label} {done}/{S} sequences, {time.perf_counter() - t0:.1f} s", flush=True)
                sys.stdout.flush()
    return out, lse, pool


def compare(out, lse, ref_out, ref_lse, kv_dtype, label=""):
    tol = TOL[kv_dtype]
    assert out.shape == ref_out.shape, (out.shape, ref_out.shape)
    fin = np.isfinite(ref_lse)
    # Empty key sets: out = 0, lse = -inf exactly.
    assert np.all(out[~fin] == 0), label
    assert np.all(lse[~fin] == -np.inf), label
    err = np.abs(out - ref_out)
    max_abs = float(err.max()) if err.size else 0.0
    dl = np.abs(lse[fin] - ref_lse[fin])
    max_dl = float(dl.max()) if dl.size else 0.0
    num = np.sqrt(((out - ref_out) ** 2).sum())
    den = np.sqrt((ref_out ** 2).sum())
    rel = float(num / den) if den > 0 else 0.0
    msg = f"{label}: max_abs={max_abs:.3e} max_dlse={max_dl:.3e} rel_l2={rel:.3e}"
    assert max_abs <= tol["max_abs"], msg
    assert max_dl <= tol["lse"], msg
    assert rel <= tol["rel_l2"], msg
    assert max_dl <= tol["lse_tight"], msg
    return dict(max_abs=max_abs, max_dlse=max_dl, rel_l2=rel)
