// Host/device interface between the C-ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rp_device.h"
#include "rp_host.h"

namespace rp {

// Lengths and group ids are clamped into the table/pool bounds before use, so
// an invalid layout gives wrong numbers but never an out-of-bounds access.
__host__ __device__ inline int clamp_group(int g, int G) { return g < 0 ? 0 : (g >= G ? G - 1 : g); }
__host__ __device__ inline int clamp_len(int len, int max_pages) {
  const int cap = max_pages * kPage;
  return len < 0 ? 0 : (len > cap ? cap : len);
}
__host__ __device__ inline int prefix_chunks(int P, int max_prefix_pages, int max_chunks) {
  const int n = cdiv(cdiv(clamp_len(P, max_prefix_pages), kPage), kPrefixChunkPages);
  return n > max_chunks ? max_chunks : n;
}
__device__ inline int clamp_page(int p, int num_pages) {
  return (unsigned)p < (unsigned)num_pages ? p : 0;
}

struct PlanArgs {
  int num_seqs, num_groups, num_q_heads, num_kv_heads;
  int num_cus;  // compute units of the device the batch runs on (sets the piece length)
  const int* seq_to_group;
  const int* prefix_lens;
  const int* resp_lens;
  int len_add;  // the plan is for resp_lens[s] + len_add response tokens (1: after this step's append)
  int max_prefix_pages, max_resp_pages;
  PlanView view;
};

struct AttnArgs {
  const void* k_pages;
  const void* v_pages;
  const float* k_scale;
  const float* v_scale;
  int num_pages, num_kv_heads;
  int num_seqs, num_groups, num_q_heads;
  const int* seq_to_group;
  const int* prefix_lens;
  const int* prefix_block_table;
  int max_prefix_pages;
  const int* resp_lens;
  const int* resp_block_table;
  int max_resp_pages;
  const void* q;     // bf16 [S][Hq][D]
  float qk_scale;    // softmax_scale * log2(e)
  PlanView view;
};

// Combine input: either an explicit CSR (row_offs != null) or the planned
// fixed slots, whose part counts follow from the lengths.
struct CombineArgs {
  const float* o_parts;
  const float* lse_parts;
  const int* row_offs;   // CSR [num_rows + 1], or null for planned slots
  int num_rows;
  void* out;             // bf16 [rows][D]
  float* lse;            // [rows] or null
  // planned slots only: parts per query row of each sequence, from the plan
  const int* seq_parts;
  int num_q_heads, parts_per_row;
};

struct AppendArgs {
  void* k_pages;
  void* v_pages;
  float* k_scale;
  float* v_scale;
  int num_pages, num_kv_heads, num_seqs;
  const int* resp_lens;
  const int* resp_block_table;
  int max_resp_pages;
  const void* k_new;  // bf16 [S][Hkv][D]
  const void* v_new;
};

// GRPO advantages: rewards [num_groups][group_size] fp32.
struct GrpoArgs {
  const float* rewards;
  int num_groups, group_size, ddof;
  double eps_std;
  float* advantages;  // [num_groups][group_size]
  float* mean;        // [num_groups] or null
  float* stdev;       // [num_groups] or null
  bool vector_ok;     // rewards and advantages 16-byte aligned (group_size 4, 8 or 16 then loads float4)
};

constexpr int kMaxHeadDim = 128;

// Pre-attention side of a decode step: q/k RMS norm + rotary embedding,
// q written out, k and v appended at response slot resp_lens[s].
struct QkPrepArgs {
  void* k_pages;
  void* v_pages;
  float* k_scale;
  float* v_scale;
  int num_pages, num_kv_heads, num_q_heads, num_seqs, num_groups;
  const int* seq_to_group;
  const int* prefix_lens;
  const int* resp_lens;
  const int* resp_block_table;
  int max_resp_pages;
  const uint16_t* q_in;      // bf16 [S][Hq][D]
  const uint16_t* k_in;      // bf16 [S][Hkv][D]
  const uint16_t* v_in;
  const uint16_t* q_norm_w;  // bf16 [D]
  const uint16_t* k_norm_w;
  double rms_eps;
  double inv_freq[kMaxHeadDim / 2];  // rotary frequency of pair i: theta^(-2i/D)
  uint16_t* q_out;           // bf16 [S][Hq][D]
  uint16_t* k_out;           // bf16 [S][Hkv][D] or null
  int blocks_per_seq;        // set by the launcher
};

// Shared-prefix prefill: packed prompt tokens of every group (group g owns
// rows prompt_offs[g] .. prompt_offs[g+1]-1 of q/k/v/out), K/V written once
// into the group's prefix pages.
struct PrefillArgs {
  void* k_pages;
  void* v_pages;
  float* k_scale;
  float* v_scale;
  int num_pages, num_kv_heads, num_groups, num_q_heads, num_tokens;
  const int* prompt_offs;
  const int* prefix_block_table;
  int max_prefix_pages;
  const void* q;  // bf16 [T][Hq][D]
  const void* k;  // bf16 [T][Hkv][D]
  const void* v;
  float qk_scale;  // softmax_scale * log2(e)
  void* out;       // bf16 [T][Hq][D]
  float* lse;      // [T][Hq] or null
  int write_pages;  // attention kernel also writes the bf16 K/V pages (one launch for the whole prefill)
};

struct ValidateArgs {
  int num_pages, num_seqs, num_groups;
  const int* seq_to_group;
  const int* prefix_lens;
  const int* prefix_block_table;
  int max_prefix_pages;
  const int* resp_lens;
  const int* resp_block_table;
  int max_resp_pages;
  int* result;       // [4]: error count, first bad kind, first bad index, value
};

hipError_t launch_plan(const PlanArgs& a, hipStream_t stream);
// q/k prep and the plan of the attention after its append in one launch
// (batches of at most 64 sequences; the plan's len_add is 1).
hipError_t launch_qk_prep_plan(QkPrepArgs a, const PlanArgs& p, int head_dim, bool fp8, hipStream_t stream);
// Grid sizes are upper bounds from host scalars; idle waves exit at once.
hipError_t launch_attn_parts(const AttnArgs& a, int head_dim, int n_rep, bool fp8, long long max_prefix_items,
                             long long max_resp_items, hipStream_t stream);
hipError_t launch_combine(const CombineArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_append(const AppendArgs& a, int head_dim, bool fp8, hipStream_t stream);
hipError_t launch_prefill_kv_write(const PrefillArgs& a, int head_dim, bool fp8, hipStream_t stream);
hipError_t launch_prefill_attn(const PrefillArgs& a, int head_dim, int n_rep, hipStream_t stream);
hipError_t launch_qk_prep(QkPrepArgs a, int head_dim, bool fp8, hipStream_t stream);
hipError_t launch_grpo(const GrpoArgs& a, hipStream_t stream);
hipError_t launch_validate(const ValidateArgs& a, hipStream_t stream);
hipError_t launch_selftest_mfma(int shape, const void* a, const void* b, float* c, hipStream_t stream);
hipError_t launch_stream_read(const void* src, uint64_t bytes, uint32_t* sink, bool nontemporal,
                              hipStream_t stream);

}  // namespace rp
