// Work planner (one workgroup): from the group map and the lengths it builds
//  * per-group member lists (CSR over sequences),
//  * prefix work items (group, chunk of kPrefixChunkPages prefix pages) for
//    groups with at least one live member,
//  * the piece length B for this batch (from its total response pages),
//  * the number of partial results per query row of each sequence,
//  * response work items (sequence, first page, tokens, partial-result slot):
//    every B-page piece first, then the ragged last pieces by decreasing size.
// Group counters live in LDS; scans are wavefront scans plus one pass over
// the wave totals.
#include "rp_device.h"
#include "rp_internal.h"
#include "rp_plan_small.h"

namespace rp {
namespace {

// The planner runs as one workgroup: 1024 threads in general, four waves for
// batches of at most kMediumPlanSeqs sequences (fewer waves to meet at each
// barrier, and a smaller launch starts sooner; measured). Batches of at most
// kSmallPlanMaxSeqs sequences take the single-wave planner of
// rp_plan_small.h.
constexpr int kMediumPlanSeqs = 256;

__device__ inline long long wave_incl_scan(long long v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const long long y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  return v;
}

// Exclusive scan across the workgroup; `total` receives the sum. Two packed
// 32-bit counters add independently as long as neither half overflows.
template <int kPlanThreads>
__device__ long long block_excl_scan(long long v, long long* s_tot, long long& total) {
  constexpr int kPlanWaves = kPlanThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long incl = wave_incl_scan(v, lane);
  if (lane == 63) s_tot[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    long long w = lane < kPlanWaves ? s_tot[lane] : 0;
    w = wave_incl_scan(w, lane);
    if (lane < kPlanWaves) s_tot[lane] = w;
  }
  __syncthreads();
  const long long base = wave > 0 ? s_tot[wave - 1] : 0;
  total = s_tot[kPlanWaves - 1];
  __syncthreads();
  return base + incl - v;
}

// Sum over the 64 lanes of a wave (every lane gets the total).
__device__ inline long long wave_sum(long long v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ inline long long pack2(int hi, int lo) { return ((long long)hi << 32) + (long long)(unsigned)lo; }
__device__ inline int hi32(long long v) { return (int)(v >> 32); }
__device__ inline int lo32(long long v) { return (int)(v & 0xFFFFFFFFll); }

// B-sized pieces written per thread per round.
constexpr int kItemBatch = 8;

// kPlanSeqBlock sequences per pass: their group ids, lengths and piece
// offsets stay in LDS (a batch with more sequences takes several passes).
template <int kPlanThreads, int kPlanSeqBlock>
__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  constexpr int kPlanWaves = kPlanThreads / 64;
  constexpr int kSeqPerThread = kPlanSeqBlock / kPlanThreads;
  constexpr int kRoundItems = kItemBatch * kPlanThreads;
  static_assert(kPlanSeqBlock % kPlanThreads == 0, "sequences per thread");
  __shared__ int s_cnt[kPlanMaxGroups];   // members per group, then the group's next member slot
  __shared__ int s_gpc[kPlanMaxGroups];   // prefix chunks per group
  __shared__ int s_sg[kPlanSeqBlock];     // clamped group of each sequence of the pass
  __shared__ int s_sl[kPlanSeqBlock];     // clamped response length of each sequence of the pass
  __shared__ int s_off[kPlanSeqBlock];    // first B-sized piece of each sequence of the pass
  __shared__ int s_own[kRoundItems];      // sequence (of the pass) of each B-sized piece of a round
  __shared__ int s_hist[kRespChunkPagesMax];  // ragged pieces per page count
  __shared__ int s_hoff[kRespChunkPagesMax];  // next item index per ragged page count
  __shared__ int s_nbig;                      // B-sized pieces
  __shared__ long long s_tot[kPlanWaves];
  __shared__ unsigned long long s_pages;
  const int t = threadIdx.x, lane = t & 63;
  const int S = a.num_seqs, G = a.num_groups;
  const PlanView v = a.view;

  for (int g = t; g < G; g += kPlanThreads) s_cnt[g] = 0;
  for (int i = t; i < kRespChunkPagesMax; i += kPlanThreads) s_hist[i] = 0;
  if (t == 0) {
    s_nbig = 0;
    s_pages = 0;
  }
  __syncthreads();

  // First pass over the inputs: group sizes, prefix chunks per group and the
  // total response pages, which set B.
  for (int g = t; g < G; g += kPlanThreads)
    s_gpc[g] = prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks);
  unsigned long long my_pages = 0;
  for (int s = t; s < S; s += kPlanThreads) {
    const int g = clamp_group(a.seq_to_group[s], G);
    const int L = plan_resp_len(a, s);
    if (s < kPlanSeqBlock) {
      s_sg[s] = g;
      s_sl[s] = L;
    }
    atomicAdd(&s_cnt[g], 1);
    my_pages += cdiv(L, kPage);
  }
  // One LDS atomic per wave: same-address atomics from every thread serialise.
  my_pages = (unsigned long long)wave_sum((long long)my_pages);
  if (lane == 0) atomicAdd(&s_pages, my_pages);
  __syncthreads();
  // B: the multiple of kRespChunkStep nearest to W / (kRespChunkStep * target
  // units), W = response pages x kv-heads, clamped to the candidates.
  // Below three quarters of one step, 16-page pieces if every response fits
  // the workspace's partial-result slots at that length.
  const int chunk = plan_piece_pages(a, (long long)s_pages * a.num_kv_heads);

  // Second pass (lengths from LDS where the first pass kept them): B-sized
  // pieces and the ragged pieces per page count.
  int my_big = 0;
  for (int s = t; s < S; s += kPlanThreads) {
    const int L = s < kPlanSeqBlock ? s_sl[s] : plan_resp_len(a, s);
    const int pages = cdiv(L, kPage);
    my_big += pages / chunk;
    if (pages % chunk) atomicAdd(&s_hist[pages % chunk], 1);
  }
  my_big = (int)wave_sum(my_big);
  if (lane == 0) atomicAdd(&s_nbig, my_big);
  __syncthreads();
  const int nbig = s_nbig;

  // Item order: every B-sized piece first, then the ragged pieces by
  // decreasing page count (one wave scans the count bins, largest first, two
  // bins per lane).
  static_assert(kRespChunkPagesMax <= 128, "one wave scans the piece-count bins");
  if (t < 64) {
    const int r1 = chunk - 1 - 2 * lane, r0 = r1 - 1;
    const int h1 = r1 >= 1 ? s_hist[r1] : 0, h0 = r0 >= 1 ? s_hist[r0] : 0;
    const int incl = (int)wave_incl_scan(h1 + h0, lane);
    if (r1 >= 1) s_hoff[r1] = nbig + incl - h1 - h0;
    if (r0 >= 1) s_hoff[r0] = nbig + incl - h0;
    if (lane == 63) {
      v.hdr[kHdrRespItems] = nbig + incl;
      v.hdr[kHdrBigRespItems] = nbig;
      v.hdr[kHdrRespChunkPages] = chunk;
    }
  }

  // Groups: member offsets and prefix items.
  int carry_m = 0, carry_i = 0;
  for (int base = 0; base < G; base += kPlanThreads) {
    const int g = base + t;
    int cnt = 0, npc = 0;
    if (g < G) {
      cnt = s_cnt[g];
      npc = cnt > 0 ? s_gpc[g] : 0;
    }
    long long tot;
    const long long ex = block_excl_scan<kPlanThreads>(pack2(cnt, npc), s_tot, tot);
    if (g < G) {
      const int off = carry_m + hi32(ex);
      v.grp_off[g] = off;
      s_cnt[g] = off;  // from here on: the group's next free member slot
      const int i0 = carry_i + lo32(ex);
      for (int c = 0; c < npc; ++c) v.prefix_items[i0 + c] = make_int2(g, c);
    }
    carry_m += hi32(tot);
    carry_i += lo32(tot);
  }
  if (t == 0) {
    v.grp_off[G] = carry_m;
    v.hdr[kHdrPrefixItems] = carry_i;
  }
  __syncthreads();  // member cursors and ragged-piece cursors are complete

  // Sequences, kPlanSeqBlock per pass: member slots and response items. A
  // sequence's B-sized pieces take items in sequence order after those of the
  // sequences before it; its ragged piece takes the next item of its page
  // count.
  int carry_f = 0;
  for (int base = 0; base < S; base += kPlanSeqBlock) {
    const int n = min(S - base, kPlanSeqBlock);
    if (base > 0) {
      __syncthreads();  // the previous pass is done with the LDS copies
      for (int k = t; k < n; k += kPlanThreads) {
        s_sg[k] = clamp_group(a.seq_to_group[base + k], G);
        s_sl[k] = plan_resp_len(a, base + k);
      }
      __syncthreads();
    }
    int cnt[kSeqPerThread], sum = 0;
#pragma unroll
    for (int j = 0; j < kSeqPerThread; ++j) {
      const int k = t * kSeqPerThread + j;
      cnt[j] = k < n ? cdiv(s_sl[k], kPage) / chunk : 0;
      sum += cnt[j];
    }
    long long tot;
    int off = (int)block_excl_scan<kPlanThreads>(sum, s_tot, tot);
#pragma unroll
    for (int j = 0; j < kSeqPerThread; ++j) {
      const int k = t * kSeqPerThread + j;
      if (k < n) s_off[k] = off;
      off += cnt[j];
    }
    __syncthreads();

    // Rounds of kRoundItems B-sized pieces: the owner of every piece of the
    // round goes into LDS first, then thread t writes pieces t + u *
    // kPlanThreads of the round, plus the member slot and ragged piece of
    // sequences t + round * kPlanThreads. Items hold no physical page ids:
    // gathering them from the block tables here would make one CU fetch a
    // cache line per item.
    const int rounds = max(cdiv(n, kPlanThreads), cdiv((int)tot, kRoundItems));
    for (int round = 0; round < rounds; ++round) {
      const int r0 = round * kRoundItems;
      if (round > 0) __syncthreads();  // the previous round is done with s_own
      for (int k = t; k < n; k += kPlanThreads) {
        const int lo = max(s_off[k], r0) - r0;
        const int hi = min(s_off[k] + cdiv(s_sl[k], kPage) / chunk, r0 + kRoundItems) - r0;
        for (int i = lo; i < hi; ++i) s_own[i] = k;
      }
      __syncthreads();

      int item[kItemBatch + 1];
      int4 rec[kItemBatch + 1];
      const int k = round * kPlanThreads + t;
      item[kItemBatch] = -1;
      if (k < n) {
        const int sq = base + k, g = s_sg[k], L = s_sl[k];
        v.grp_members[atomicAdd(&s_cnt[g], 1)] = sq;
        const int pages = cdiv(L, kPage), nfull = pages / chunk, rem = pages - nfull * chunk;
        v.seq_parts[sq] = s_gpc[g] + nfull + (rem != 0 ? 1 : 0);
        if (rem != 0) {
          const int p0 = nfull * chunk;
          item[kItemBatch] = atomicAdd(&s_hoff[rem], 1);
          rec[kItemBatch] = make_int4(sq, p0, L - p0 * kPage, s_gpc[g] + nfull);
        }
      }
#pragma unroll
      for (int u = 0; u < kItemBatch; ++u) {
        const int i = r0 + u * kPlanThreads + t;
        item[u] = -1;
        if (i < (int)tot) {
          const int o = s_own[i - r0];
          const int sq = base + o, c = i - s_off[o], p0 = c * chunk;
          item[u] = carry_f + i;
          rec[u] = make_int4(sq, p0, min(chunk * kPage, s_sl[o] - p0 * kPage), s_gpc[s_sg[o]] + c);
        }
      }
#pragma unroll
      for (int u = 0; u <= kItemBatch; ++u) {
        if (item[u] >= 0) v.resp_items[item[u]] = rec[u];
      }
    }
    carry_f += (int)tot;
  }
}

__global__ __launch_bounds__(64) void plan_small_kernel(PlanArgs a) {
  __shared__ int s_cnt[kPlanMaxGroups];
  plan_small(a, s_cnt);
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t stream) {
  if (a.num_seqs <= kSmallPlanMaxSeqs) plan_small_kernel<<<1, 64, 0, stream>>>(a);
  else if (a.num_seqs <= kMediumPlanSeqs) plan_kernel<256, 1024><<<1, 256, 0, stream>>>(a);
  else plan_kernel<1024, 4096><<<1, 1024, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rp
