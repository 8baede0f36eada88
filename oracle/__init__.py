"""CPU oracle for group decode attention over a paged KV cache.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or call anything in this package;
the library's product path never does. It shares no code with the HIP library.

Everything is computed in float64 from the plain definitions:

* attention per sequence: ``out = softmax(sigma * q K^T) V`` over the keys of the
  sequence's group prefix followed by its own response (the GRPO group shares one
  prompt, Section 2.1 of the paper; the key order is irrelevant mathematically);
* the log-sum-exp merge of partial results over disjoint key subsets;
* the KV append (bf16 copy, or OCP e4m3fn quantisation with a per-(page, head)
  scale);
* the shared-prefix prefill: causal attention over each group's prompt and
  the one-time write of its K/V pages;
* the pre-attention side of a decode step: RMS norm and rotary embedding of
  q and k, then the append;
* one rollout round under Slime, CGP and CGP+FGD scheduling, simulated one
  decode step at a time (``sched``);
* GRPO group statistics and advantages (Eq. 1, ``grpo``);
* bf16 and OCP e4m3fn decoding from the formats' bit definitions.

Every function here is pinned by ``-m "not gpu"`` tests against library
routines, closed forms, invariants and brute force; none is "parity unpinned".
"""
from .formats import bf16_to_f64, bf16_to_f32, e4m3_to_f64, e4m3_encode, E4M3_MAX
from .attention import decode_attention, key_slots, attention_for_workload
from .combine import lse_combine
from .append import kv_append, append_for_workload
from .prefill import prefill_attention, prefill_kv_write
from .qkprep import decode_positions, decode_step_prep, qk_prep, rms_norm, rope
from .sched import simulate as simulate_schedule
from .grpo import advantage, advantage_f32, group_stats

__all__ = ["bf16_to_f64", "bf16_to_f32", "e4m3_to_f64", "e4m3_encode", "E4M3_MAX",
           "decode_attention", "key_slots", "attention_for_workload",
           "lse_combine", "kv_append", "append_for_workload", "prefill_attention", "prefill_kv_write",
           "decode_positions", "decode_step_prep", "qk_prep", "rms_norm", "rope",
           "simulate_schedule", "advantage", "advantage_f32", "group_stats"]
