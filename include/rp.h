/*
 * rp.h - group decode attention over a paged, group-shared KV cache (gfx950).
 *
 * The operation is the attention step of autoregressive rollout decoding. In
 * GRPO rollouts every prompt is sampled K times and the K responses of a prompt
 * form a group (paper, Section 2.1 and Section 5.1 with K = 8); the decode
 * workers of the serving engine generate all of them under fixed weights
 * (Section 4, rollout node). Here a group's prompt-prefix KV is stored once and
 * every response of the group adds its own ragged response KV.
 *
 * For sequence s in group g = seq_to_group[s] and query head j the result is
 * the plain softmax attention over the concatenated keys
 *     prefix tokens t < prefix_lens[g]  at page prefix_block_table[g][t / ps], row t % ps
 *     response tokens t < resp_lens[s]  at page resp_block_table[s][t / ps],   row t % ps
 * namely, with sigma = softmax_scale and kv-head h = j / (Hq / Hkv):
 *     s_t = sigma * <q[s][j], k_t[h]>,  lse = ln sum_t exp(s_t),
 *     out[s][j] = sum_t exp(s_t - lse) * v_t[h].
 * An empty key set yields out = 0 and lse = -inf.
 *
 * Conventions for every call:
 *  - Pointers inside rp_paged_kv / rp_group_layout and all array arguments are
 *    DEVICE pointers unless marked "host". The two structs themselves live in
 *    host memory and are read during the call only.
 *  - Calls are asynchronous on `stream` (may be NULL for the default stream),
 *    never synchronise (except rp_validate_layout) and never allocate device
 *    memory (except rp_validate_layout). The caller owns every buffer.
 *  - Scalar/pointer arguments are validated synchronously; a failed check
 *    returns an error before anything is launched. Device array CONTENTS are
 *    not validated on the hot path: out-of-range page ids or lengths beyond the
 *    table widths are undefined behaviour (check them with rp_validate_layout).
 *  - Errors are reported by return code; rp_last_error() gives detail text for
 *    the calling thread.
 */
#ifndef RP_H_
#define RP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t; /* identical to HIP's own typedef */

typedef enum {
  RP_OK = 0,
  RP_ERR_INVALID_ARG = 1,  /* null pointer, misalignment, inconsistent sizes */
  RP_ERR_UNSUPPORTED = 2,  /* valid but not implemented (head_dim, page_size, ratio) */
  RP_ERR_WORKSPACE = 3,    /* workspace missing or smaller than required */
  RP_ERR_HIP = 4,          /* a HIP launch or runtime call failed; see rp_last_error */
  RP_ERR_LAYOUT = 5        /* rp_validate_layout found an out-of-range entry */
} rp_status;

typedef enum {
  RP_KV_BF16 = 0,          /* bf16 K/V elements */
  RP_KV_FP8_E4M3 = 1       /* OCP FP8 e4m3fn codes (max 448, no inf) with fp32 scales */
} rp_kv_dtype;

/* Paged KV pool, caller-owned.
 * k_pages, v_pages: [num_pages][num_kv_heads][page_size][head_dim] elements of
 *   kv_dtype, 16-byte aligned. One (page, kv-head) block is contiguous.
 * k_scale, v_scale: fp32 [num_pages][num_kv_heads]; element value = decoded
 *   code * scale of its (page, kv-head). Must be NULL for RP_KV_BF16 and
 *   non-NULL for RP_KV_FP8_E4M3.
 * Supported: page_size == 16, head_dim in {64, 128}. */
typedef struct {
  void* k_pages;
  void* v_pages;
  float* k_scale;
  float* v_scale;
  int32_t num_pages;
  int32_t num_kv_heads;
  int32_t page_size;
  int32_t head_dim;
  rp_kv_dtype kv_dtype;
} rp_paged_kv;

/* Batch layout: S sequences in num_groups prompt groups, caller-owned int32
 * device arrays.
 * seq_to_group[S]                          group of each sequence, in [0, num_groups)
 * prefix_lens[num_groups]                  shared prompt-prefix tokens per group
 * prefix_block_table[num_groups][max_prefix_pages]
 * resp_lens[S]                             response tokens of each sequence
 * resp_block_table[S][max_resp_pages]
 * Requires num_q_heads % num_kv_heads == 0 with ratio in {1, 2, 4, 8};
 * query head j uses kv-head j / (num_q_heads / num_kv_heads). */
typedef struct {
  int32_t num_seqs;
  int32_t num_groups;
  int32_t num_q_heads;
  const int32_t* seq_to_group;
  const int32_t* prefix_lens;
  const int32_t* prefix_block_table;
  int32_t max_prefix_pages;
  const int32_t* resp_lens;
  const int32_t* resp_block_table;
  int32_t max_resp_pages;
} rp_group_layout;

/* Static description of an error code (never NULL). */
const char* rp_status_string(rp_status status);

/* Detail text of the last error returned on the calling thread ("" if none). */
const char* rp_last_error(void);

/* KV append: write one new token per sequence.
 * k_new, v_new: bf16 [num_seqs][num_kv_heads][head_dim], 16-byte aligned.
 * layout->resp_lens holds the PRE-append lengths L_s; the token goes to
 * response slot L_s (page resp_block_table[s][L_s / 16], row L_s % 16), which
 * the caller must have provided in the table. resp_lens is not modified: the
 * caller advances it. Repeating a call with the same inputs is idempotent.
 * RP_KV_BF16: the bf16 values are copied.
 * RP_KV_FP8_E4M3, per (sequence, kv-head), separately for K and V, in fp32:
 * amax = max|x|; row 0 of a page sets scale = amax / 448 (1 if amax == 0);
 * a later row keeps the scale if amax <= 448 * scale, otherwise sets
 * scale = amax / 448 and requantises rows 0..r-1 from code * old_scale; the
 * row is stored as e4m3(x / scale), round to nearest even, saturated at 448.
 * A NaN element of x does not enter amax and is stored as the saturated code
 * with its sign (0x7E or 0xFE); the NaN code is never written.
 * Two sequences must not append into the same (page, kv-head).
 * Defined by the decode step of the rollout's decode workers (paper,
 * Section 4): every generated token's K and V join its sequence's cache
 * before attention reads them. */
rp_status rp_kv_append(const rp_paged_kv* kv, const rp_group_layout* layout,
                       const void* k_new, const void* v_new, hipStream_t stream);

/* Pre-attention side of one decode step of a Qwen3-style attention layer
 * (the paper's policy model, Section 5.1): RMS norm of every q and k head
 * with the layer's per-channel weights, then the rotary position embedding,
 * then the append of k and v.
 * The new token of sequence s (group g = seq_to_group[s]) is at position
 * p_s = prefix_lens[g] + resp_lens[s]. For a head vector x of head_dim d,
 *   y = x / sqrt(mean(x^2) + rms_eps) * w,
 *   out[i]       = y[i] cos(a_i) - y[i + d/2] sin(a_i),
 *   out[i + d/2] = y[i + d/2] cos(a_i) + y[i] sin(a_i),  a_i = p_s * rope_theta^(-2i/d),
 * for i < d/2, with w = q_norm_w for q heads and k_norm_w for k heads.
 * Computed in fp64 from the bf16 inputs and rounded once to bf16 (nearest
 * even): outputs equal the correctly rounded values except where the exact
 * value lies within a few fp64 ulps of a rounding boundary (then they are
 * one bf16 ulp away). The rotary frequencies theta^(-2i/d) are computed on
 * the host with the C library's pow.
 * q_in: bf16 [S][Hq][d]; k_in, v_in: bf16 [S][Hkv][d]; q_norm_w, k_norm_w:
 * bf16 [d]; q_out: bf16 [S][Hq][d] (the q layout rp_group_decode_attn reads);
 * all 16-byte aligned. q_out may be q_in itself but must not otherwise
 * overlap it. k_out: bf16 [S][Hkv][d] copy of the rotated k, or NULL. The
 * rotated k and the unchanged v are appended exactly as rp_kv_append would
 * append them (same slot, same fp8 rule); a sequence with resp_lens[s]
 * outside [0, max_resp_pages * 16) gets q_out (and k_out) but no append.
 * rms_eps must be finite and >= 0 (Qwen3: 1e-6; with 0, an all-zero head
 * gives NaN), rope_theta finite and > 0 (Qwen3: 1e6). */
rp_status rp_decode_qk_prep(const rp_paged_kv* kv, const rp_group_layout* layout,
                            const void* q_in, const void* k_in, const void* v_in,
                            const void* q_norm_w, const void* k_norm_w,
                            double rms_eps, double rope_theta,
                            void* q_out, void* k_out, hipStream_t stream);

/* rp_decode_qk_prep followed by rp_plan for the attention over the advanced
 * lengths, as one call: the q/k prep and append exactly as rp_decode_qk_prep
 * with `layout` (resp_lens = the tokens already cached), and the work plan
 * of rp_plan for the same batch with resp_lens[s] + 1 response tokens, in
 * `workspace` (at least rp_group_decode_attn_workspace_size bytes of this
 * layout, 256-byte aligned). Then rp_attn_parts and rp_combine_parts with
 * the advanced layout (the same arrays, resp_lens + 1) complete the decode
 * step. Batches of at most 64 sequences (the frontier batches of
 * frontier-group dispatch, Section 3.3: F_w groups of K samples) take one
 * launch, the plan built by one wave beside the prep blocks; larger ones
 * take the two launches. Same arguments, checks and errors as the two calls. */
rp_status rp_decode_qk_prep_plan(const rp_paged_kv* kv, const rp_group_layout* layout,
                                 const void* q_in, const void* k_in, const void* v_in,
                                 const void* q_norm_w, const void* k_norm_w,
                                 double rms_eps, double rope_theta,
                                 void* q_out, void* k_out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes needed by rp_group_decode_attn / rp_plan for this shape.
 * Depends only on host-side scalars (S, num_groups, Hq, Hkv, head_dim,
 * max_prefix_pages, max_resp_pages); *bytes is a host pointer. */
rp_status rp_group_decode_attn_workspace_size(const rp_paged_kv* kv,
                                              const rp_group_layout* layout,
                                              size_t* bytes);

/* Group decode attention (the definition at the top of this file): one
 * decode step of every sequence of the rollout batch (paper, Section 4, the
 * rollout node's decode workers), the K responses of a GRPO group sharing
 * their prompt's KV (Section 2.1; Section 5.1 samples K = 8).
 * q:   bf16 [num_seqs][num_q_heads][head_dim], 16-byte aligned.
 * out: bf16 [num_seqs][num_q_heads][head_dim], 16-byte aligned.
 * lse: fp32 [num_seqs][num_q_heads], natural log; may be NULL.
 * softmax_scale: sigma, normally 1/sqrt(head_dim).
 * workspace: device buffer of at least rp_group_decode_attn_workspace_size
 *   bytes, 256-byte aligned, used for the work plan and partial results;
 *   concurrent calls need distinct workspaces.
 * Equivalent to rp_plan, rp_attn_parts, rp_combine_parts. */
rp_status rp_group_decode_attn(const rp_paged_kv* kv, const rp_group_layout* layout,
                               const void* q, float softmax_scale, void* out, float* lse,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of device scratch behind rp_group_decode_attn_noalloc (64 MiB): a
 * static array in the library, one copy per GPU, held until the process
 * ends. */
#define RP_NOALLOC_SCRATCH_BYTES (64u << 20)

/* rp_group_decode_attn without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops and
 * harnesses that forbid hipMalloc. The plan and the partial results live in
 * the library's static scratch of RP_NOALLOC_SCRATCH_BYTES on the current
 * device (the same kernels and results as rp_group_decode_attn, bit for bit).
 * Nothing is allocated; the first call on a device looks up that device's
 * scratch address once. Layouts whose workspace
 * (rp_group_decode_attn_workspace_size) exceeds the scratch are refused with
 * RP_ERR_WORKSPACE before anything is launched: 256 sequences with 4096-token
 * responses fit (21 MB), 1024 sequences of 8192 do not.
 * All calls on one GPU share its scratch: calls that overlap in time on one
 * GPU (different streams, host threads or processes sharing a context) race
 * and give wrong results; serialise them. Arguments and errors otherwise as
 * rp_group_decode_attn. */
rp_status rp_group_decode_attn_noalloc(const rp_paged_kv* kv, const rp_group_layout* layout,
                                       const void* q, float softmax_scale, void* out, float* lse,
                                       hipStream_t stream);

/* Log-sum-exp merge of partial attention results over disjoint key subsets
 * (the step that makes splitting a sequence's keys exact: attention over a
 * union of disjoint key sets is the lse-weighted mean of the parts; it is
 * how the group-prefix parts of Section 2.1's shared prompt join each
 * response's own parts).
 * o_parts: fp32 [total_parts][head_dim] (16-byte aligned), lse_parts: fp32 [total_parts] (natural
 * log, -inf marks an empty part whose o is ignored); row r owns parts
 * row_part_offsets[r] .. row_part_offsets[r+1]-1 (int32 CSR, [num_rows + 1]).
 *   lse_out[r] = ln sum_i exp(lse_i),  out[r] = sum_i exp(lse_i - lse_out[r]) o_i
 * out: bf16 [num_rows][head_dim] (8-byte aligned); lse_out: fp32 [num_rows] or NULL. A row with
 * no non-empty part gets out = 0, lse = -inf. head_dim in {64, 128}. */
rp_status rp_lse_combine(const float* o_parts, const float* lse_parts,
                         const int32_t* row_part_offsets, int32_t num_rows, int32_t head_dim,
                         void* out, float* lse_out, hipStream_t stream);

/* ---- Shared-prefix prefill ---------------------------------------------
 * Every response of a GRPO group is sampled from the same prompt (paper,
 * Section 2.1), so a prompt is processed once per group, not once per
 * response: its K/V are written once into the group's prefix pages (the pages
 * rp_group_decode_attn reads for every response of the group) and its tokens
 * attend causally within the prompt.
 *
 * Prompt tokens of all groups are packed: group g owns rows
 * prompt_offs[g] .. prompt_offs[g+1]-1 of q [T][Hq][head_dim] and
 * k, v [T][Hkv][head_dim] (bf16), its prompt length being the difference;
 * token t of group g lives at page prefix_block_table[g][t / 16], row t % 16. */
typedef struct {
  int32_t num_groups;                 /* G */
  int32_t num_q_heads;                /* Hq; Hkv and head_dim come from the pool */
  int32_t num_tokens;                 /* T = prompt_offs[G], a host copy */
  const int32_t* prompt_offs;         /* [G + 1], non-decreasing, prompt_offs[0] = 0 */
  const int32_t* prefix_block_table;  /* [G][max_prefix_pages] */
  int32_t max_prefix_pages;           /* every prompt has at most max_prefix_pages * 16 tokens */
} rp_prefill_layout;

/* Write every group's prompt K/V into its prefix pages. bf16 pools copy the
 * rows. fp8 pools give each (page, kv-head) of a prompt, in fp32,
 * scale = amax / 448 over the page's written rows (1.0 when amax = 0) and
 * store e4m3(x / scale) (round to nearest even, saturating at 448; a NaN
 * element does not enter amax and is stored as the saturated code with its
 * sign); rows past a prompt's end are not written. k, v: bf16
 * [T][Hkv][head_dim], 16-byte aligned. Prompts must not share pages. */
rp_status rp_prefill_kv_write(const rp_paged_kv* kv, const rp_prefill_layout* layout,
                              const void* k, const void* v, hipStream_t stream);

/* Causal attention within each prompt: for token t of group g and query head
 * j (kv-head j / (Hq / Hkv)), over the group's tokens u <= t,
 *   s_u = softmax_scale * <q_t[j], k_u>, lse = ln sum_u exp(s_u),
 *   out[t][j] = sum_u exp(s_u - lse) v_u.
 * Reads the bf16 projections q, k, v (not the pool; the pool only supplies
 * Hkv and head_dim). out: bf16 [T][Hq][head_dim], 16-byte aligned; lse: fp32
 * [T][Hq], natural log, may be NULL. softmax_scale must be finite and > 0. */
rp_status rp_prefill_attn(const rp_paged_kv* kv, const rp_prefill_layout* layout,
                          const void* q, const void* k, const void* v, float softmax_scale,
                          void* out, float* lse, hipStream_t stream);

/* The whole prefill of a step: rp_prefill_kv_write and rp_prefill_attn with
 * the same arguments, in that order, with the same results (the same page
 * bytes, out and lse). For a bf16 pool it is one launch: the attention
 * kernel stages every prompt's K/V blocks anyway, and the workgroup whose
 * query rows start a block also copies it into the pages. An fp8 pool takes
 * the page-write kernel first, because each page's scale needs the whole
 * page. Same argument rules and errors as the two calls. */
rp_status rp_prefill(const rp_paged_kv* kv, const rp_prefill_layout* layout,
                     const void* q, const void* k, const void* v, float softmax_scale,
                     void* out, float* lse, hipStream_t stream);

/* ---- Staged form of rp_group_decode_attn -------------------------------
 * A decode step's layout is shared by every layer, so a caller can plan once
 * and run the attention of all layers against the same plan. */

/* Build the work plan in `workspace` from the layout's device arrays: group
 * member lists, prefix work items (16-page chunks of each live group's
 * prefix), response work items (every response cut into pieces of B pages,
 * the B-page pieces first and then each response's shorter last piece by
 * decreasing size), and the number of partial results per query row. B is
 * the multiple of 32 pages nearest to W / (32 * 6 * C), clamped to 32..128,
 * where W is the batch's response pages (ceil(resp_lens[s] / 16) summed over
 * s) times num_kv_heads and C the current device's compute units; it is 16
 * when W < 0.75 * 32 * 6 * C and the layout's response capacity (num_seqs *
 * max_resp_pages * num_kv_heads) is at most 2^17 page-heads, the layouts
 * whose workspace is sized for 16-page pieces.
 * Must be re-run whenever seq_to_group, prefix_lens or resp_lens change.
 * Supports num_groups <= 4096. */
rp_status rp_plan(const rp_paged_kv* kv, const rp_group_layout* layout,
                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/* All partial results for a planned workspace, in one kernel launch:
 * group-prefix parts (each group's prompt prefix read once per kv-head and
 * applied to all query rows of its live members on the matrix cores) and
 * response parts (each sequence's own response pages, one planned piece per
 * unit).
 * q and softmax_scale as in rp_group_decode_attn. */
rp_status rp_attn_parts(const rp_paged_kv* kv, const rp_group_layout* layout,
                        const void* q, float softmax_scale,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Merge the planned workspace's partial results into out / lse (same meaning
 * as in rp_group_decode_attn); runs rp_lse_combine's kernel on them. */
rp_status rp_combine_parts(const rp_paged_kv* kv, const rp_group_layout* layout,
                           void* out, float* lse,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Where rp_plan stores its results inside a workspace, for tests and tools
 * that read a plan back (host-side only; launches nothing). Offsets are in
 * bytes from the workspace start. Contents, all int32:
 *   hdr[16]: [0] prefix items, [1] response items, [2] of those, the B-page
 *            pieces (they come first), [3] B, the piece length in pages;
 *   grp_off[G + 1], grp_members[S]: CSR of each group's live sequences;
 *   prefix_items: (group, chunk of 16 prefix pages) pairs;
 *   resp_items: (sequence, first page index in the sequence's block table,
 *               tokens, partial-result slot) quadruples, in dispatch order;
 *   seq_parts[S]: partial results per query row of each sequence.
 * part_o (fp32 [max_parts][head_dim]) and part_lse (fp32 [max_parts]) hold
 * the partial results of query row r in slots r * parts_per_row + k. */
typedef struct {
  size_t hdr, grp_off, grp_members, prefix_items, resp_items, seq_parts;
  size_t part_o, part_lse;
  int32_t max_prefix_items, max_resp_items, parts_per_row, max_parts;
} rp_plan_info;

rp_status rp_plan_layout(const rp_paged_kv* kv, const rp_group_layout* layout, rp_plan_info* info);

/* Check the layout's device arrays against the pool and table sizes: groups
 * in range, lengths non-negative and within the table widths, every page id
 * that a length makes reachable in [0, num_pages). TEST UTILITY: allocates a
 * small device buffer and synchronises `stream`. Returns RP_OK or
 * RP_ERR_LAYOUT (detail in rp_last_error). */
rp_status rp_validate_layout(const rp_paged_kv* kv, const rp_group_layout* layout,
                             hipStream_t stream);

/* ---- GRPO group statistics (Eq. 1) -----------------------------------
 * For each of num_groups groups of group_size rewards r_1..r_K (fp32,
 * rewards[g][i], device), in fp64:
 *   mu = sum r / K,  sigma = sqrt(sum (r - mu)^2 / (K - ddof))  (0 when K - ddof < 1),
 *   A_i = (r_i - mu) / (sigma + eps_std),
 * each output rounded once to fp32: advantages[g][i], and, unless NULL,
 * group_mean[g] = mu and group_std[g] = sigma. The paper fixes neither the
 * estimator nor eps_std: ddof = 1 is the unbiased estimate (the default of
 * common GRPO implementations), ddof = 0 the population one; eps_std must
 * be finite and >= 0 (1e-6 is the usual choice). A group of equal rewards
 * gets A = 0 when eps_std > 0 (NaN when eps_std = 0). Arrays are fp32 and 4-byte aligned (16-byte alignment of
 * rewards and advantages enables vector loads for K = 4, 8, 16);
 * advantages may alias rewards. */
rp_status rp_grpo_advantage(const float* rewards, int32_t num_groups, int32_t group_size,
                            double eps_std, int32_t ddof, float* advantages,
                            float* group_mean, float* group_std, hipStream_t stream);

/* ---- Scheduling simulation (host) -------------------------------------
 * One rollout round and its training under the paper's schedulers (Sections
 * 3.2-3.3, Eq. 2-6, Algorithm 1). All pointers here are HOST pointers; the
 * call is synchronous and touches no GPU.
 *
 * Rollout node: R groups of K requests; request q = g K + i belongs to group
 * g (submission order = g) and generates resp_lens[q] >= 1 tokens after its
 * group's prompt of prompt_lens[g] >= 0 tokens. At each scheduling cycle (a
 * decode-step boundary): under RP_SCHED_CGP_FGD, while the frontier holds
 * fewer than frontier_width groups, the lowest-order group not yet admitted
 * joins it and its K requests join the admitted queue (Eq. 5-6); under the
 * other modes all R K requests are in that queue from the start, group by
 * group. Then admitted requests enter the running set, first come first
 * served, while it holds fewer than max_running; the first request of a group
 * to run brings the group's prompt prefill into that step. A decode step
 * lasts step_base + step_per_seq n + step_per_ctx_token ctx + prefill, with n
 * running requests, ctx the sum of their prompt plus generated tokens before
 * the step, prefill the sum of prefill_per_token prompt_lens[g] over the
 * groups started in that cycle; every running request generates one token.
 * A group is serving-complete at the end of the step in which its last
 * request finishes, and leaves the frontier.
 * Control node: the group is trainable-complete mat_base + mat_per_token
 * (its response tokens) later and joins the trainer FIFO (by time, ties by
 * group order).
 * Training node: update k consumes FIFO entries kU .. kU+U-1 (U =
 * update_groups, which must divide R) and lasts the sum over its groups of
 * train_base + train_per_token (K prompt + response tokens of the group),
 * plus opt_step. It starts when the trainer is free and the U-th of those
 * groups is trainable (CGP modes) or every group is (RP_SCHED_SLIME), Eq. 2.
 * Sums are accumulated in the order written here, in IEEE double without
 * contraction, so results are reproducible bit for bit.
 * Cost parameters must be finite and >= 0 (seconds). */
typedef enum {
  RP_SCHED_SLIME = 0,    /* train after the whole rollout is trainable */
  RP_SCHED_CGP = 1,      /* complete-group pipelining, request-level FIFO admission */
  RP_SCHED_CGP_FGD = 2   /* complete-group pipelining with frontier-group dispatch */
} rp_sched_mode;

typedef struct {
  rp_sched_mode mode;
  int32_t num_groups;      /* R */
  int32_t group_size;      /* K */
  int32_t update_groups;   /* U = B / K, divides R */
  int32_t frontier_width;  /* F_w (RP_SCHED_CGP_FGD only, >= 1) */
  int32_t max_running;     /* engine concurrency, >= 1 */
  double step_base, step_per_seq, step_per_ctx_token, prefill_per_token;
  double mat_base, mat_per_token;
  double train_base, train_per_token, opt_step;
} rp_sched_config;

typedef struct {
  double t_first_u;    /* the first U groups are all trainable (the U-th FIFO entry) */
  double t_complete;   /* every group trainable */
  double t_start;      /* first update starts (Eq. 2) */
  double delta_cgp;    /* t_complete - t_first_u (Eq. 3) */
  double t_train_end;  /* last update ends; rollout starts at 0 */
  double compute;      /* summed update durations */
  double wait;         /* trainer idle time in [0, t_train_end] */
  double w_train;      /* t_start / t_train_end (Eq. 4) */
  double wait_ratio;   /* wait / (wait + compute), the trainer-side ratio */
  int64_t steps;       /* decode steps of the round */
} rp_sched_summary;

/* prompt_lens[R], resp_lens[R K] (host int32). summary is required; the
 * per-group outputs may be NULL: serve_done[R], frontier_enter[R] (0 unless
 * RP_SCHED_CGP_FGD), trainable[R] (double seconds), fifo[R] (group ids in
 * FIFO order), update_start[R / U], update_end[R / U]. */
rp_status rp_sched_simulate(const rp_sched_config* config, const int32_t* prompt_lens,
                            const int32_t* resp_lens, rp_sched_summary* summary,
                            double* serve_done, double* frontier_enter, double* trainable,
                            int32_t* fifo, double* update_start, double* update_end);

/* ---- Self-test of the matrix-core lane layouts ----
 * Test infrastructure for callers and for this library's own tests. The
 * attention and prefill kernels form MFMA operands and read accumulators in
 * fixed per-lane layouts, and form the V^T operand of P V with gfx950's
 * transposing LDS read; one wave forms the operands of a single MFMA from
 * a (bf16 [M][K], row-major) and b (bf16 [K][N], row-major) in those layouts
 * and writes the accumulator as c (fp32 [M][N], row-major). With small
 * integer inputs the products are exact, so c must equal a b exactly; any
 * other result means the layouts the kernels rely on do not hold on the
 * device. The _LDS_TR shape stages a transposed in LDS and reads it back
 * with the transposing read, in the key order the prefill uses in P V.
 * All pointers are device memory; nothing is allocated. RP_ERR_UNSUPPORTED
 * for an unknown shape, RP_ERR_INVALID_ARG for a NULL or misaligned pointer. */
typedef enum {
  RP_SELFTEST_MFMA_16X16X32 = 0,        /* M = N = 16, K = 32 */
  RP_SELFTEST_MFMA_16X16X16 = 1,        /* M = N = K = 16 */
  RP_SELFTEST_MFMA_16X16X32_LDS_TR = 2  /* M = N = 16, K = 32 */
} rp_selftest_shape;

rp_status rp_selftest_mfma(int32_t shape, const void* a, const void* b, float* c, hipStream_t stream);

/* ---- Streaming-read probe ----
 * Measurement infrastructure: the HBM read rate a plain kernel reaches on
 * this device, the practical ceiling for the memory-bound decode kernels
 * (bench.py --read-ceiling times it). Reads `bytes` bytes at src once with
 * 16-byte vector loads spread over RP_STREAM_READ_BLOCKS workgroups, with the
 * non-temporal load hint when nontemporal != 0 (as the decode kernel's V
 * stream), and writes RP_STREAM_READ_SINK_WORDS folded words to sink so that
 * no load can be dropped. src: device memory, 16-byte aligned, bytes a
 * multiple of 16; sink: device memory, 4-byte aligned. Nothing is allocated.
 * RP_ERR_INVALID_ARG for a NULL or misaligned pointer or a bad size. */
#define RP_STREAM_READ_BLOCKS 2048
#define RP_STREAM_READ_SINK_WORDS (RP_STREAM_READ_BLOCKS * 4)
rp_status rp_stream_read(const void* src, uint64_t bytes, uint32_t* sink, int32_t nontemporal, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RP_H_ */
