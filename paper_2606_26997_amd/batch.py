"""Device-resident decode batch: torch tensors plus the C-ABI descriptors.

Host arrays (numpy or torch) are copied to the device once; the descriptors
point at those tensors. This is marshalling only: attention, append and
combine all run in librp.so.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _binding as B


def _dev(x, device, dtype=None):
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        if x.dtype == np.uint16:
            t = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16)
        elif x.dtype == np.uint8:
            t = torch.from_numpy(x)
        else:
            t = torch.from_numpy(np.ascontiguousarray(x))
    else:
        t = x
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device).contiguous()


class DeviceBatch:
    """One decode step's inputs on the device.

    ``resp_lens`` are the response tokens already cached. With ``append`` the
    new token goes to slot ``resp_lens[s]`` and attention then reads
    ``resp_lens + 1`` (the caller's length advance, done here once).
    """

    def __init__(self, *, k_pages, v_pages, k_scale, v_scale, seq_to_group, prefix_lens,
                 prefix_block_table, resp_lens, resp_block_table, q, num_q_heads, softmax_scale,
                 k_new=None, v_new=None, append=False, device="cuda"):
        self.device = torch.device(device)
        d = self.device
        self.k_pages = _dev(k_pages, d)
        self.v_pages = _dev(v_pages, d)
        self.k_scale = _dev(k_scale, d, torch.float32)
        self.v_scale = _dev(v_scale, d, torch.float32)
        self.seq_to_group = _dev(seq_to_group, d, torch.int32)
        self.prefix_lens = _dev(prefix_lens, d, torch.int32)
        self.prefix_block_table = _dev(prefix_block_table, d, torch.int32)
        self.resp_lens = _dev(resp_lens, d, torch.int32)
        self.resp_block_table = _dev(resp_block_table, d, torch.int32)
        self.q = _dev(q, d)
        self.k_new = _dev(k_new, d)
        self.v_new = _dev(v_new, d)
        self.append = bool(append)
        self.attn_resp_lens = self.resp_lens + 1 if self.append else self.resp_lens
        self.num_q_heads = int(num_q_heads)
        self.softmax_scale = float(softmax_scale)
        S = self.seq_to_group.shape[0]
        D = self.k_pages.shape[3]
        self.out = torch.zeros((S, self.num_q_heads, D), dtype=torch.bfloat16, device=d)
        self.lse = torch.zeros((S, self.num_q_heads), dtype=torch.float32, device=d)
        self.kv = B.paged_kv(self.k_pages, self.v_pages, self.k_scale, self.v_scale)
        self.append_layout = self._layout(self.resp_lens)
        self.attn_layout = self._layout(self.attn_resp_lens)
        ws = B.group_decode_attn_workspace_size(self.kv, self.attn_layout)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=d)

    @classmethod
    def from_workload(cls, wl, device="cuda"):
        return cls(k_pages=wl.k_pages, v_pages=wl.v_pages, k_scale=wl.k_scale, v_scale=wl.v_scale,
                   seq_to_group=wl.seq_to_group, prefix_lens=wl.prefix_lens,
                   prefix_block_table=wl.prefix_block_table, resp_lens=wl.resp_lens,
                   resp_block_table=wl.resp_block_table, q=wl.q, num_q_heads=wl.num_q_heads,
                   softmax_scale=wl.softmax_scale, k_new=wl.k_new, v_new=wl.v_new,
                   append=wl.append, device=device)

    def _layout(self, resp_lens):
        return B.group_layout(self.seq_to_group, self.prefix_lens, self.prefix_block_table, resp_lens,
                              self.resp_block_table, num_q_heads=self.num_q_heads)

    # -- the decode step ------------------------------------------------------
    def kv_append(self, stream=None):
        B.kv_append(self.kv, self.append_layout, self.k_new, self.v_new, stream)

    def attention(self, stream=None):
        B.group_decode_attn(self.kv, self.attn_layout, self.q, self.softmax_scale, self.out, self.lse,
                            self.workspace, stream)

    def step(self, stream=None):
        """Append (if the batch carries new tokens) and attention."""
        if self.append:
            self.kv_append(stream)
        self.attention(stream)

    # -- decode step from the raw projections ---------------------------------
    def set_projections(self, q_in, k_in, v_in, q_norm_w, k_norm_w, *, rms_eps=1e-6, rope_theta=1e6,
                        keep_k=False):
        """Raw (pre-norm) projections of the new token; ``decode_step`` then builds q and the appended k/v."""
        if not self.append:
            raise ValueError("set_projections needs a batch built with append=True")
        d = self.device
        self.q_in, self.k_in, self.v_in = _dev(q_in, d), _dev(k_in, d), _dev(v_in, d)
        self.q_norm_w, self.k_norm_w = _dev(q_norm_w, d), _dev(k_norm_w, d)
        self.rms_eps, self.rope_theta = float(rms_eps), float(rope_theta)
        self.k_out = torch.empty_like(self.k_in) if keep_k else None

    def qk_prep(self, stream=None):
        """RMS norm + rotary embedding of q (into ``self.q``) and k, and the append of k and v."""
        B.decode_qk_prep(self.kv, self.append_layout, self.q_in, self.k_in, self.v_in, self.q_norm_w,
                         self.k_norm_w, self.q, self.k_out, rms_eps=self.rms_eps, rope_theta=self.rope_theta,
                         stream=stream)

    def decode_step(self, stream=None):
        """Pre-attention prep (with the append), then attention over the advanced lengths."""
        self.qk_prep(stream)
        self.attention(stream)

    def qk_prep_plan(self, stream=None):
        """``qk_prep`` and the plan of the attention over the advanced lengths (one launch for small
        batches); ``attn_parts`` and ``combine_parts`` then finish the step."""
        B.decode_qk_prep_plan(self.kv, self.append_layout, self.q_in, self.k_in, self.v_in, self.q_norm_w,
                              self.k_norm_w, self.q, self.k_out, self.workspace, rms_eps=self.rms_eps,
                              rope_theta=self.rope_theta, stream=stream)

    # -- staged form ------------------------------------------------------------
    def plan(self, stream=None):
        B.plan(self.kv, self.attn_layout, self.workspace, stream)

    def attn_parts(self, stream=None):
        B.attn_parts(self.kv, self.attn_layout, self.q, self.softmax_scale, self.workspace, stream)

    def combine_parts(self, stream=None):
        B.combine_parts(self.kv, self.attn_layout, self.out, self.lse, self.workspace, stream)

    def plan_contents(self):
        """The planned workspace read back to the host (numpy int32 arrays)."""
        info = B.plan_layout(self.kv, self.attn_layout)
        torch.cuda.synchronize()
        ws = self.workspace.cpu().numpy()
        S, G = self.seq_to_group.shape[0], self.prefix_lens.shape[0]

        def arr(off, count, width=1):
            return ws[off:off + 4 * count * width].view(np.int32).reshape(-1, width) if width > 1 else \
                ws[off:off + 4 * count].view(np.int32)
        hdr = arr(info.hdr, 16)
        return dict(hdr=hdr, grp_off=arr(info.grp_off, G + 1), grp_members=arr(info.grp_members, S),
                    prefix_items=arr(info.prefix_items, int(hdr[0]), 2),
                    resp_items=arr(info.resp_items, int(hdr[1]), 4),
                    seq_parts=arr(info.seq_parts, S), parts_per_row=info.parts_per_row)

    def validate(self, stream=None):
        B.validate_layout(self.kv, self.attn_layout, stream)


class PrefillBatch:
    """Packed prompts of several groups on the device, for the shared-prefix prefill."""

    def __init__(self, *, q, k, v, prompt_offs, prefix_block_table, k_pages, v_pages, k_scale=None, v_scale=None,
                 num_q_heads, softmax_scale, device="cuda"):
        d = self.device = torch.device(device)
        self.q, self.k, self.v = _dev(q, d), _dev(k, d), _dev(v, d)
        self.prompt_offs = _dev(prompt_offs, d, torch.int32)
        self.prefix_block_table = _dev(prefix_block_table, d, torch.int32)
        self.k_pages, self.v_pages = _dev(k_pages, d), _dev(v_pages, d)
        self.k_scale = _dev(k_scale, d, torch.float32)
        self.v_scale = _dev(v_scale, d, torch.float32)
        self.softmax_scale = float(softmax_scale)
        T = int(self.q.shape[0])
        self.out = torch.zeros((T, int(num_q_heads), int(self.q.shape[2])), dtype=torch.bfloat16, device=d)
        self.lse = torch.zeros((T, int(num_q_heads)), dtype=torch.float32, device=d)
        self.kv = B.paged_kv(self.k_pages, self.v_pages, self.k_scale, self.v_scale)
        self.layout = B.prefill_layout(self.prompt_offs, self.prefix_block_table, num_q_heads=num_q_heads,
                                       num_tokens=T)

    @classmethod
    def from_workload(cls, w, device="cuda"):
        return cls(q=w.q, k=w.k, v=w.v, prompt_offs=w.prefix_offs, prefix_block_table=w.prefix_block_table,
                   k_pages=w.k_pages, v_pages=w.v_pages, k_scale=w.k_scale, v_scale=w.v_scale,
                   num_q_heads=w.num_q_heads, softmax_scale=w.softmax_scale, device=device)

    def kv_write(self, stream=None):
        B.prefill_kv_write(self.kv, self.layout, self.k, self.v, stream)

    def attention(self, stream=None):
        B.prefill_attn(self.kv, self.layout, self.q, self.k, self.v, self.softmax_scale, self.out, self.lse, stream)

    def step(self, stream=None):
        """Write the prompts' K/V pages, then attend within each prompt (two calls)."""
        self.kv_write(stream)
        self.attention(stream)

    def prefill(self, stream=None):
        """The same results as ``step`` through rp_prefill (one launch for a bf16 pool)."""
        B.prefill(self.kv, self.layout, self.q, self.k, self.v, self.softmax_scale, self.out, self.lse, stream)
