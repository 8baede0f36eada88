// Work planner (one workgroup): from the group map and the lengths it builds
//  * per-group member lists (CSR over sequences),
//  * prefix work items (group, chunk of kPrefixChunkPages prefix pages) for
//    groups with at least one live member,
//  * the response chunk length for this batch (short or long, from the
//    average response length),
//  * response work items (sequence, chunk, clamped response length, prefix
//    chunks of the sequence's group) with the physical id of each item's first
//    page, ordered longest first: every full chunk, then the ragged last chunks
//    by decreasing page count, so the last free slots get the least work.
// Group counters live in LDS; scans are wavefront scans plus one pass over
// the wave totals.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;

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
__device__ long long block_excl_scan(long long v, long long* s_tot, long long& total) {
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

__device__ inline long long pack2(int hi, int lo) { return ((long long)hi << 32) + (long long)(unsigned)lo; }
__device__ inline int hi32(long long v) { return (int)(v >> 32); }
__device__ inline int lo32(long long v) { return (int)(v & 0xFFFFFFFFll); }

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ int s_cnt[kPlanMaxGroups];
  __shared__ int s_fill[kPlanMaxGroups];
  __shared__ int s_hist[kRespChunkPagesMax];   // ragged chunks per page count
  __shared__ int s_hoff[kRespChunkPagesMax];
  __shared__ long long s_tot[kPlanWaves];
  __shared__ unsigned long long s_pages;
  __shared__ int s_off[kPlanThreads];   // per-thread item offsets of one chunk of sequences
  __shared__ int s_len[kPlanThreads];
  __shared__ int s_npc[kPlanThreads];
  const int t = threadIdx.x;
  const int S = a.num_seqs, G = a.num_groups;
  const PlanView v = a.view;
  const int* bt = a.resp_block_table;

  for (int g = t; g < G; g += kPlanThreads) {
    s_cnt[g] = 0;
    s_fill[g] = 0;
  }
  if (t < kRespChunkPagesMax) s_hist[t] = 0;
  if (t == 0) s_pages = 0;
  __syncthreads();

  // Live members per group and the total number of response pages.
  unsigned long long my_pages = 0;
  for (int s = t; s < S; s += kPlanThreads) {
    atomicAdd(&s_cnt[clamp_group(a.seq_to_group[s], G)], 1);
    my_pages += cdiv(clamp_len(a.resp_lens[s], a.max_resp_pages), kPage);
  }
  atomicAdd(&s_pages, my_pages);
  __syncthreads();
  const int chunk =
      s_pages >= (unsigned long long)S * kLongResponsePages ? kRespChunkPagesMax : kRespChunkPagesMin;
  for (int s = t; s < S; s += kPlanThreads) {
    const int rem = cdiv(clamp_len(a.resp_lens[s], a.max_resp_pages), kPage) % chunk;
    if (rem != 0) atomicAdd(&s_hist[rem], 1);
  }

  // Groups: member offsets and prefix items.
  int carry_m = 0, carry_i = 0;
  for (int base = 0; base < G; base += kPlanThreads) {
    const int g = base + t;
    int cnt = 0, npc = 0;
    if (g < G) {
      cnt = s_cnt[g];
      npc = cnt > 0 ? prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks) : 0;
    }
    long long tot;
    const long long ex = block_excl_scan(pack2(cnt, npc), s_tot, tot);
    if (g < G) {
      const int off = carry_m + hi32(ex);
      v.grp_off[g] = off;
      s_cnt[g] = off;  // from here on: the group's first member slot
      const int i0 = carry_i + lo32(ex);
      for (int c = 0; c < npc; ++c) v.prefix_items[i0 + c] = make_int2(g, c);
    }
    carry_m += hi32(tot);
    carry_i += lo32(tot);
  }
  if (t == 0) {
    v.grp_off[G] = carry_m;
    v.hdr[kHdrPrefixItems] = carry_i;
    v.hdr[kHdrRespChunkPages] = chunk;
  }
  __syncthreads();

  // Sequences: member placement and full response chunks. The items of each
  // chunk of sequences are written by all threads together; item k belongs to
  // the last sequence whose offset is <= k.
  int carry_f = 0;
  for (int base = 0; base < S; base += kPlanThreads) {
    const int s = base + t;
    int nfull = 0, L = 0, npc = 0;
    if (s < S) {
      const int g = clamp_group(a.seq_to_group[s], G);
      v.grp_members[s_cnt[g] + atomicAdd(&s_fill[g], 1)] = s;
      L = clamp_len(a.resp_lens[s], a.max_resp_pages);
      npc = prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks);
      nfull = cdiv(L, kPage) / chunk;
    }
    long long tot;
    const int ex = (int)block_excl_scan(nfull, s_tot, tot);
    s_off[t] = ex;
    s_len[t] = L;
    s_npc[t] = npc;
    __syncthreads();
    for (int k = t; k < (int)tot; k += kPlanThreads) {
      int lo = 0, hi = kPlanThreads - 1;  // largest j with s_off[j] <= k
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= k) lo = mid;
        else hi = mid - 1;
      }
      const int sj = base + lo, c = k - s_off[lo];
      const int item = carry_f + k;
      v.resp_items[item] = make_int4(sj, c, s_len[lo], s_npc[lo]);
      v.resp_first_page[item] = bt[(size_t)sj * a.max_resp_pages + c * chunk];
    }
    __syncthreads();
    carry_f += (int)tot;
  }

  // Ragged last chunks after all full ones, largest first.
  if (t == 0) {
    int off = carry_f;
    for (int r = chunk - 1; r >= 1; --r) {
      s_hoff[r] = off;
      off += s_hist[r];
    }
    v.hdr[kHdrRespItems] = off;
    v.hdr[kHdrFullRespItems] = carry_f;
  }
  __syncthreads();
  for (int s = t; s < S; s += kPlanThreads) {
    const int L = clamp_len(a.resp_lens[s], a.max_resp_pages);
    const int pages = cdiv(L, kPage);
    const int rem = pages % chunk;
    if (rem != 0) {
      const int g = clamp_group(a.seq_to_group[s], G);
      const int npc = prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks);
      const int c = pages / chunk;
      const int item = atomicAdd(&s_hoff[rem], 1);
      v.resp_items[item] = make_int4(s, c, L, npc);
      v.resp_first_page[item] = bt[(size_t)s * a.max_resp_pages + c * chunk];
    }
  }
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t stream) {
  plan_kernel<<<1, kPlanThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rp
