"""ctypes binding for librp.so: argument marshalling only.

Every computation runs in the HIP library. torch is imported first so that the
library's HIP runtime dependency resolves to the runtime torch already loaded;
tensors are passed by ``data_ptr()`` and streams by their raw HIP handle.
If the library is missing or cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch  # noqa: F401  (loads torch's HIP runtime before librp.so)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librp.so")

RP_OK = 0
RP_ERR_INVALID_ARG = 1
RP_ERR_UNSUPPORTED = 2
RP_ERR_WORKSPACE = 3
RP_ERR_HIP = 4
RP_ERR_LAYOUT = 5
RP_KV_BF16 = 0
RP_KV_FP8_E4M3 = 1
RP_NOALLOC_SCRATCH_BYTES = 64 << 20   # include/rp.h: static scratch of rp_group_decode_attn_noalloc

EXPORTED = ("rp_status_string", "rp_last_error", "rp_kv_append",
            "rp_group_decode_attn_workspace_size", "rp_group_decode_attn", "rp_lse_combine",
            "rp_plan", "rp_attn_parts", "rp_combine_parts", "rp_plan_layout", "rp_validate_layout",
            "rp_prefill_kv_write", "rp_prefill_attn", "rp_decode_qk_prep", "rp_sched_simulate",
            "rp_grpo_advantage", "rp_prefill", "rp_group_decode_attn_noalloc", "rp_decode_qk_prep_plan",
            "rp_selftest_mfma", "rp_stream_read")
RP_STREAM_READ_SINK_WORDS = 2048 * 4   # include/rp.h
# include/rp.h rp_selftest_shape: name -> (code, M, N, K)
RP_SELFTEST_SHAPES = {"16x16x32": (0, 16, 16, 32), "16x16x16": (1, 16, 16, 16), "16x16x32_lds_tr": (2, 16, 16, 32)}
RP_SCHED_MODES = {"slime": 0, "cgp": 1, "cgp_fgd": 2}


class RpPagedKV(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("num_pages", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32)]


class RpGroupLayout(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_groups", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32),
                ("seq_to_group", ctypes.c_void_p), ("prefix_lens", ctypes.c_void_p),
                ("prefix_block_table", ctypes.c_void_p), ("max_prefix_pages", ctypes.c_int32),
                ("resp_lens", ctypes.c_void_p), ("resp_block_table", ctypes.c_void_p),
                ("max_resp_pages", ctypes.c_int32)]


class RpPrefillLayout(ctypes.Structure):
    _fields_ = [("num_groups", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("prompt_offs", ctypes.c_void_p), ("prefix_block_table", ctypes.c_void_p),
                ("max_prefix_pages", ctypes.c_int32)]


class RpPlanInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("hdr", "grp_off", "grp_members", "prefix_items", "resp_items",
                                                 "seq_parts", "part_o", "part_lse")] + \
               [(n, ctypes.c_int32) for n in ("max_prefix_items", "max_resp_items", "parts_per_row", "max_parts")]


class RpSchedConfig(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("num_groups", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("update_groups", ctypes.c_int32), ("frontier_width", ctypes.c_int32),
                ("max_running", ctypes.c_int32)] + \
               [(n, ctypes.c_double) for n in ("step_base", "step_per_seq", "step_per_ctx_token", "prefill_per_token",
                                                "mat_base", "mat_per_token", "train_base", "train_per_token",
                                                "opt_step")]


class RpSchedSummary(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("t_first_u", "t_complete", "t_start", "delta_cgp", "t_train_end",
                                                "compute", "wait", "w_train", "wait_ratio")] + \
               [("steps", ctypes.c_int64)]


class RpError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: {status_string(status)}: {detail}")


_lib = None


def load() -> ctypes.CDLL:
    """Load librp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "rp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "rp_last_error": (ctypes.c_char_p, []),
        "rp_kv_append": (ctypes.c_int, [P, P, P, P, P]),
        "rp_group_decode_attn_workspace_size": (ctypes.c_int, [P, P, ctypes.POINTER(ctypes.c_size_t)]),
        "rp_group_decode_attn": (ctypes.c_int, [P, P, P, F32, P, P, P, ctypes.c_size_t, P]),
        "rp_group_decode_attn_noalloc": (ctypes.c_int, [P, P, P, F32, P, P, P]),
        "rp_lse_combine": (ctypes.c_int, [P, P, P, I32, I32, P, P, P]),
        "rp_plan": (ctypes.c_int, [P, P, P, ctypes.c_size_t, P]),
        "rp_attn_parts": (ctypes.c_int, [P, P, P, F32, P, ctypes.c_size_t, P]),
        "rp_combine_parts": (ctypes.c_int, [P, P, P, P, P, ctypes.c_size_t, P]),
        "rp_plan_layout": (ctypes.c_int, [P, P, P]),
        "rp_validate_layout": (ctypes.c_int, [P, P, P]),
        "rp_prefill_kv_write": (ctypes.c_int, [P, P, P, P, P]),
        "rp_prefill_attn": (ctypes.c_int, [P, P, P, P, P, F32, P, P, P]),
        "rp_prefill": (ctypes.c_int, [P, P, P, P, P, F32, P, P, P]),
        "rp_decode_qk_prep": (ctypes.c_int, [P, P, P, P, P, P, P, ctypes.c_double, ctypes.c_double, P, P, P]),
        "rp_decode_qk_prep_plan": (ctypes.c_int, [P, P, P, P, P, P, P, ctypes.c_double, ctypes.c_double, P, P, P,
                                                   ctypes.c_size_t, P]),
        "rp_sched_simulate": (ctypes.c_int, [P, P, P, P, P, P, P, P, P, P]),
        "rp_grpo_advantage": (ctypes.c_int, [P, I32, I32, ctypes.c_double, I32, P, P, P, P]),
        "rp_selftest_mfma": (ctypes.c_int, [I32, P, P, P, P]),
        "rp_stream_read": (ctypes.c_int, [P, ctypes.c_uint64, P, I32, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().rp_status_string(int(status)).decode()


def last_error() -> str:
    return load().rp_last_error().decode()


def _check(status: int, func: str) -> None:
    if status != RP_OK:
        raise RpError(status, func, last_error())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def paged_kv(k_pages, v_pages, k_scale=None, v_scale=None, *, num_pages=None, num_kv_heads=None,
             page_size=16, head_dim=None, kv_dtype=None) -> RpPagedKV:
    """Describe a pool of tensors shaped [num_pages][Hkv][page_size][head_dim]."""
    shape = tuple(k_pages.shape) if hasattr(k_pages, "shape") else None
    if kv_dtype is None:
        kv_dtype = RP_KV_FP8_E4M3 if k_scale is not None else RP_KV_BF16
    return RpPagedKV(_ptr(k_pages), _ptr(v_pages), _ptr(k_scale), _ptr(v_scale),
                     num_pages if num_pages is not None else shape[0],
                     num_kv_heads if num_kv_heads is not None else shape[1],
                     page_size, head_dim if head_dim is not None else shape[3], kv_dtype)


def group_layout(seq_to_group, prefix_lens, prefix_block_table, resp_lens, resp_block_table, *,
                 num_q_heads, num_seqs=None, num_groups=None, max_prefix_pages=None,
                 max_resp_pages=None) -> RpGroupLayout:
    return RpGroupLayout(
        num_seqs if num_seqs is not None else seq_to_group.shape[0],
        num_groups if num_groups is not None else prefix_lens.shape[0],
        num_q_heads, _ptr(seq_to_group), _ptr(prefix_lens), _ptr(prefix_block_table),
        max_prefix_pages if max_prefix_pages is not None else prefix_block_table.shape[1],
        _ptr(resp_lens), _ptr(resp_block_table),
        max_resp_pages if max_resp_pages is not None else resp_block_table.shape[1])


def kv_append(kv: RpPagedKV, layout: RpGroupLayout, k_new, v_new, stream=None) -> None:
    _check(load().rp_kv_append(ctypes.byref(kv), ctypes.byref(layout), _ptr(k_new), _ptr(v_new),
                               _stream(stream)), "rp_kv_append")


def decode_qk_prep(kv, layout, q_in, k_in, v_in, q_norm_w, k_norm_w, q_out, k_out=None, *,
                   rms_eps=1e-6, rope_theta=1e6, stream=None) -> None:
    _check(load().rp_decode_qk_prep(ctypes.byref(kv), ctypes.byref(layout), _ptr(q_in), _ptr(k_in), _ptr(v_in),
                                    _ptr(q_norm_w), _ptr(k_norm_w), float(rms_eps), float(rope_theta),
                                    _ptr(q_out), _ptr(k_out), _stream(stream)),
           "rp_decode_qk_prep")


def decode_qk_prep_plan(kv, layout, q_in, k_in, v_in, q_norm_w, k_norm_w, q_out, k_out, workspace, *,
                        rms_eps=1e-6, rope_theta=1e6, stream=None) -> None:
    """q/k prep with the append (``layout``: pre-append lengths) and the plan of the attention over the
    advanced lengths, in ``workspace``."""
    _check(load().rp_decode_qk_prep_plan(ctypes.byref(kv), ctypes.byref(layout), _ptr(q_in), _ptr(k_in),
                                         _ptr(v_in), _ptr(q_norm_w), _ptr(k_norm_w), float(rms_eps),
                                         float(rope_theta), _ptr(q_out), _ptr(k_out), _ptr(workspace),
                                         _ws_bytes(workspace), _stream(stream)),
           "rp_decode_qk_prep_plan")


def grpo_advantage(rewards, advantages, group_mean=None, group_std=None, *, eps_std=1e-6, ddof=1,
                   stream=None) -> None:
    """rewards, advantages: fp32 device tensors [R][K]; group_mean, group_std: [R] or None."""
    R, K = int(rewards.shape[0]), int(rewards.shape[1])
    _check(load().rp_grpo_advantage(_ptr(rewards), R, K, float(eps_std), int(ddof), _ptr(advantages),
                                    _ptr(group_mean), _ptr(group_std), _stream(stream)), "rp_grpo_advantage")


def group_decode_attn_workspace_size(kv: RpPagedKV, layout: RpGroupLayout) -> int:
    n = ctypes.c_size_t(0)
    _check(load().rp_group_decode_attn_workspace_size(ctypes.byref(kv), ctypes.byref(layout),
                                                      ctypes.byref(n)),
           "rp_group_decode_attn_workspace_size")
    return int(n.value)


def _ws_bytes(workspace) -> int:
    if workspace is None:
        return 0
    return workspace.numel() * workspace.element_size()


def group_decode_attn(kv, layout, q, softmax_scale, out, lse, workspace, stream=None) -> None:
    _check(load().rp_group_decode_attn(ctypes.byref(kv), ctypes.byref(layout), _ptr(q),
                                       float(softmax_scale), _ptr(out), _ptr(lse), _ptr(workspace),
                                       _ws_bytes(workspace), _stream(stream)),
           "rp_group_decode_attn")


def group_decode_attn_noalloc(kv, layout, q, softmax_scale, out, lse, stream=None) -> None:
    """rp_group_decode_attn on the library's static scratch (no workspace, nothing allocated)."""
    _check(load().rp_group_decode_attn_noalloc(ctypes.byref(kv), ctypes.byref(layout), _ptr(q),
                                               float(softmax_scale), _ptr(out), _ptr(lse), _stream(stream)),
           "rp_group_decode_attn_noalloc")


def plan(kv, layout, workspace, stream=None) -> None:
    _check(load().rp_plan(ctypes.byref(kv), ctypes.byref(layout), _ptr(workspace),
                          _ws_bytes(workspace), _stream(stream)), "rp_plan")


def attn_parts(kv, layout, q, softmax_scale, workspace, stream=None) -> None:
    _check(load().rp_attn_parts(ctypes.byref(kv), ctypes.byref(layout), _ptr(q), float(softmax_scale),
                                _ptr(workspace), _ws_bytes(workspace), _stream(stream)),
           "rp_attn_parts")


def combine_parts(kv, layout, out, lse, workspace, stream=None) -> None:
    _check(load().rp_combine_parts(ctypes.byref(kv), ctypes.byref(layout), _ptr(out), _ptr(lse),
                                   _ptr(workspace), _ws_bytes(workspace), _stream(stream)),
           "rp_combine_parts")


def selftest_mfma(shape, a, b, c, stream=None) -> None:
    """One MFMA in the kernels' lane layouts: c (fp32 [M][N]) = a (bf16 [M][K]) b (bf16 [K][N]).

    shape: a key of RP_SELFTEST_SHAPES or its integer code."""
    code = RP_SELFTEST_SHAPES[shape][0] if isinstance(shape, str) else int(shape)
    _check(load().rp_selftest_mfma(code, _ptr(a), _ptr(b), _ptr(c), _stream(stream)), "rp_selftest_mfma")


def stream_read(src, nbytes, sink, nontemporal=False, stream=None) -> None:
    """Read nbytes of device tensor src once (16-byte loads); sink: int32/uint32 [RP_STREAM_READ_SINK_WORDS]."""
    _check(load().rp_stream_read(_ptr(src), int(nbytes), _ptr(sink), int(bool(nontemporal)), _stream(stream)),
           "rp_stream_read")


def lse_combine(o_parts, lse_parts, row_part_offsets, num_rows, head_dim, out, lse_out,
                stream=None) -> None:
    _check(load().rp_lse_combine(_ptr(o_parts), _ptr(lse_parts), _ptr(row_part_offsets),
                                 int(num_rows), int(head_dim), _ptr(out), _ptr(lse_out),
                                 _stream(stream)), "rp_lse_combine")


def plan_layout(kv, layout) -> RpPlanInfo:
    info = RpPlanInfo()
    _check(load().rp_plan_layout(ctypes.byref(kv), ctypes.byref(layout), ctypes.byref(info)), "rp_plan_layout")
    return info


def validate_layout(kv, layout, stream=None) -> None:
    _check(load().rp_validate_layout(ctypes.byref(kv), ctypes.byref(layout), _stream(stream)),
           "rp_validate_layout")


def prefill_layout(prompt_offs, prefix_block_table, *, num_q_heads, num_tokens) -> RpPrefillLayout:
    """Describe packed prompts: group g owns rows prompt_offs[g] .. prompt_offs[g+1]-1."""
    return RpPrefillLayout(int(prompt_offs.shape[0]) - 1, int(num_q_heads), int(num_tokens), _ptr(prompt_offs),
                           _ptr(prefix_block_table), int(prefix_block_table.shape[1]))


def prefill_kv_write(kv, layout, k, v, stream=None) -> None:
    _check(load().rp_prefill_kv_write(ctypes.byref(kv), ctypes.byref(layout), _ptr(k), _ptr(v), _stream(stream)),
           "rp_prefill_kv_write")


def prefill_attn(kv, layout, q, k, v, softmax_scale, out, lse, stream=None) -> None:
    _check(load().rp_prefill_attn(ctypes.byref(kv), ctypes.byref(layout), _ptr(q), _ptr(k), _ptr(v),
                                  float(softmax_scale), _ptr(out), _ptr(lse), _stream(stream)), "rp_prefill_attn")


def prefill(kv, layout, q, k, v, softmax_scale, out, lse, stream=None) -> None:
    _check(load().rp_prefill(ctypes.byref(kv), ctypes.byref(layout), _ptr(q), _ptr(k), _ptr(v),
                             float(softmax_scale), _ptr(out), _ptr(lse), _stream(stream)), "rp_prefill")


def sched_simulate(*, mode, group_size, update_groups, prompt_lens, resp_lens, max_running, frontier_width=0,
                   step_base=0.0, step_per_seq=0.0, step_per_ctx_token=0.0, prefill_per_token=0.0,
                   mat_base=0.0, mat_per_token=0.0, train_base=0.0, train_per_token=0.0, opt_step=0.0) -> dict:
    """Run rp_sched_simulate on host arrays; returns the summary and the per-group timelines."""
    import numpy as np
    prompt = np.ascontiguousarray(prompt_lens, dtype=np.int32)
    resp = np.ascontiguousarray(resp_lens, dtype=np.int32)
    R = int(prompt.shape[0])
    U = max(int(update_groups), 1)
    cfg = RpSchedConfig(RP_SCHED_MODES[mode], R, int(group_size), int(update_groups), int(frontier_width),
                        int(max_running), step_base, step_per_seq, step_per_ctx_token, prefill_per_token,
                        mat_base, mat_per_token, train_base, train_per_token, opt_step)
    summ = RpSchedSummary()
    f64 = [np.zeros(R, np.float64) for _ in range(3)]
    fifo = np.zeros(R, np.int32)
    upd = [np.zeros(max(R // U, 1), np.float64) for _ in range(2)]
    dp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    _check(load().rp_sched_simulate(ctypes.byref(cfg), dp(prompt), dp(resp), ctypes.byref(summ), dp(f64[0]),
                                    dp(f64[1]), dp(f64[2]), dp(fifo), dp(upd[0]), dp(upd[1])),
           "rp_sched_simulate")
    out = {n: getattr(summ, n) for n, _ in RpSchedSummary._fields_}
    out.update(serve_done=f64[0].tolist(), frontier_enter=f64[1].tolist(), trainable=f64[2].tolist(),
               fifo=fifo.tolist(), update_start=upd[0][:R // U].tolist(), update_end=upd[1][:R // U].tolist())
    return out
