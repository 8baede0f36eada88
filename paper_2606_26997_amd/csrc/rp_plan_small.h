// The work plan of a small batch (at most 64 sequences) built by one wave,
// one lane per sequence, with wave-level synchronisation only: the same plan
// contract as the general planner (member lists, prefix items, the piece
// length B, B-page pieces in sequence order, then the ragged last pieces by
// decreasing page count, part counts). Used by rp_plan for small batches and
// by the decode step's fused q/k prep + plan launch, where it runs in one
// workgroup of the prep grid.
#pragma once

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

// Orders this wave's LDS accesses (a single-wave planner needs no more).
__device__ inline void plan_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Inclusive prefix sum over the wave of non-negative v, and the wave total,
// one ballot per bit of the largest v: bit b contributes 2^b times the
// number of lanes at or below this one that have it set (v_mbcnt). No data
// moves between lanes, so each bit costs a few cycles instead of a round
// trip through the LDS crossbar.
__device__ inline int plan_wave_incl_scan(int v, int* total) {
  int incl = 0, tot = 0;
  for (int b = 0; __ballot((v >> b) != 0) != 0; ++b) {
    const unsigned long long m = __ballot((v >> b) & 1);
    const int upto = __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0)) +
                     (int)((v >> b) & 1);
    incl += upto << b;
    tot += __popcll(m) << b;
  }
  *total = tot;
  return incl;
}

// The response length the plan is made for: resp_lens[s] + len_add (the
// decode step plans the attention over the lengths after its append),
// saturating instead of overflowing, then clamped to the table.
__device__ inline int plan_resp_len(const PlanArgs& a, int s) {
  const int L = a.resp_lens[s];
  return clamp_len(L > 0x7FFFFFFF - a.len_add ? 0x7FFFFFFF : L + a.len_add, a.max_resp_pages);
}

// B for a batch with W page-heads of response work (see kRespChunkStep).
__device__ inline int plan_piece_pages(const PlanArgs& a, long long W) {
  const long long unit = (long long)kRespChunkStep * kUnitsPerCu * max(a.num_cus, 1);
  int chunk = kRespChunkStep * (int)min(max((W + unit / 2) / unit, 1ll), (long long)kRespChunkChoices);
  if (4 * W < 3 * unit && a.view.max_resp_chunks >= cdiv(a.max_resp_pages, kRespChunkPagesSmall))
    chunk = kRespChunkPagesSmall;
  return chunk;
}

// Call with the 64 lanes of one wave (and no other wave of the workgroup
// taking part); s_cnt is LDS for kPlanMaxGroups counters. Requires
// num_seqs <= kSmallPlanMaxSeqs and num_groups <= kPlanMaxGroups.
__device__ inline void plan_small(const PlanArgs& a, int* s_cnt) {
  const int lane = threadIdx.x & 63;
  const int S = a.num_seqs, G = a.num_groups;
  const PlanView v = a.view;
  const bool mine = lane < S;  // this lane's sequence exists

  // All loads at once: the sequence's group and length, and the prefix
  // lengths of groups 0..63 (a later group's is loaded when it is needed).
  int g = 0, L = 0, p64 = 0;
  if (mine) {
    g = clamp_group(a.seq_to_group[lane], G);
    L = plan_resp_len(a, lane);
  }
  if (lane < G) p64 = a.prefix_lens[lane];
  for (int i = lane; i < G; i += 64) s_cnt[i] = 0;
  const int P = G <= 64 ? __shfl(p64, g) : (mine ? a.prefix_lens[g] : 0);
  const int gpc = mine ? prefix_chunks(P, a.max_prefix_pages, v.max_prefix_chunks) : 0;
  const int pages = mine ? cdiv(L, kPage) : 0;

  int wpages;
  plan_wave_incl_scan(pages, &wpages);
  const int chunk = plan_piece_pages(a, (long long)wpages * a.num_kv_heads);
  const int nfull = pages / chunk, rem = pages - nfull * chunk;

  // Rank of the sequence among its group's members, then the groups' member
  // offsets and prefix items (groups in order, 64 per step).
  plan_wave_sync();
  const int rank = mine ? atomicAdd(&s_cnt[g], 1) : 0;
  plan_wave_sync();
  int carry_m = 0, carry_i = 0;
  for (int base = 0; base < G; base += 64) {
    const int gg = base + lane;
    const int cnt = gg < G ? s_cnt[gg] : 0;
    int npc = 0;
    if (cnt > 0) npc = prefix_chunks(base == 0 ? p64 : a.prefix_lens[gg], a.max_prefix_pages, v.max_prefix_chunks);
    int tm, ti;
    const int im = plan_wave_incl_scan(cnt, &tm), ii = plan_wave_incl_scan(npc, &ti);
    if (gg < G) {
      const int off = carry_m + im - cnt;
      v.grp_off[gg] = off;
      s_cnt[gg] = off;  // from here on: the group's first member slot
    }
    const int i0 = carry_i + ii - npc;
    for (int c = 0; c < npc; ++c) v.prefix_items[i0 + c] = make_int2(gg, c);
    carry_m += tm;
    carry_i += ti;
  }
  plan_wave_sync();
  if (mine) v.grp_members[s_cnt[g] + rank] = lane;

  // B-page pieces in sequence order, then each ragged last piece at its
  // place among the ragged pieces by decreasing page count (ties by sequence).
  int nbig;
  const int ib = plan_wave_incl_scan(nfull, &nbig);
  for (int c = 0; c < nfull; ++c) {
    const int p0 = c * chunk;
    v.resp_items[ib - nfull + c] = make_int4(lane, p0, min(chunk * kPage, L - p0 * kPage), gpc + c);
  }
  int pos = 0, nrag = 0;
  for (int s2 = 0; s2 < S; ++s2) {
    const int r2 = __builtin_amdgcn_readlane(rem, s2);
    pos += (r2 > rem || (r2 == rem && s2 < lane)) ? 1 : 0;
    nrag += r2 > 0 ? 1 : 0;
  }
  if (mine && rem > 0) {
    const int p0 = nfull * chunk;
    v.resp_items[nbig + pos] = make_int4(lane, p0, L - p0 * kPage, gpc + nfull);
  }
  if (mine) v.seq_parts[lane] = gpc + nfull + (rem > 0 ? 1 : 0);
  if (lane == 0) {
    v.grp_off[G] = carry_m;
    v.hdr[kHdrPrefixItems] = carry_i;
    v.hdr[kHdrRespItems] = nbig + nrag;
    v.hdr[kHdrBigRespItems] = nbig;
    v.hdr[kHdrRespChunkPages] = chunk;
  }
}

}  // namespace rp
