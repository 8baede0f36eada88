// Work planner: turns the layout's lengths and group map into
//  * per-group member lists (a CSR over sequences),
//  * prefix work items (group, chunk of kPrefixChunkPages prefix pages),
//  * response work items (sequence, chunk of kRespChunkPages response pages),
//  * the CSR of partial results per (sequence, query head) row: first the
//    group's prefix chunks, then the sequence's own response chunks.
// One workgroup does it all; S and the group count are a few thousand at most,
// so the cost is a few microseconds.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

namespace {

constexpr int kPlanThreads = 1024;

// Inclusive-to-exclusive block scan of a 64-bit value (two packed 32-bit
// counters add independently as long as neither half overflows).
__device__ long long block_exclusive_scan(long long v, long long* s_buf, long long& total) {
  const int t = threadIdx.x;
  s_buf[t] = v;
  __syncthreads();
  for (int o = 1; o < kPlanThreads; o <<= 1) {
    long long add = t >= o ? s_buf[t - o] : 0;
    __syncthreads();
    s_buf[t] += add;
    __syncthreads();
  }
  total = s_buf[kPlanThreads - 1];
  long long incl = s_buf[t];
  __syncthreads();
  return incl - v;
}

__device__ inline long long pack2(int hi, int lo) {
  return ((long long)hi << 32) + (long long)(unsigned)lo;
}
__device__ inline int hi32(long long v) { return (int)(v >> 32); }
__device__ inline int lo32(long long v) { return (int)(v & 0xFFFFFFFFll); }

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ long long s_buf[kPlanThreads];
  const int t = threadIdx.x;
  const int S = a.num_seqs, G = a.num_groups, Hq = a.num_q_heads;
  PlanView v = a.view;

  for (int g = t; g < G; g += kPlanThreads) {
    v.grp_count[g] = 0;
    v.grp_fill[g] = 0;
  }
  __syncthreads();
  for (int s = t; s < S; s += kPlanThreads) atomicAdd(&v.grp_count[clamp_group(a.seq_to_group[s], G)], 1);
  __syncthreads();

  // Groups: member offsets and prefix items.
  int carry_m = 0, carry_i = 0;
  for (int base = 0; base < G; base += kPlanThreads) {
    const int g = base + t;
    int cnt = 0, npc = 0;
    if (g < G) {
      // Counts were produced by L2 atomics: read them past the per-CU cache.
      cnt = __hip_atomic_load(&v.grp_count[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      npc = cnt > 0 ? prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks) : 0;
    }
    long long tot;
    const long long ex = block_exclusive_scan(pack2(cnt, npc), s_buf, tot);
    if (g < G) {
      v.grp_off[g] = carry_m + hi32(ex);
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
  __syncthreads();

  for (int s = t; s < S; s += kPlanThreads) {
    const int g = clamp_group(a.seq_to_group[s], G);
    const int pos = atomicAdd(&v.grp_fill[g], 1);
    v.grp_members[v.grp_off[g] + pos] = s;
  }

  // Sequences: partial-result rows and response items.
  int carry_p = 0, carry_r = 0;
  for (int base = 0; base < S; base += kPlanThreads) {
    const int s = base + t;
    int np = 0, nrc = 0;
    if (s < S) {
      const int g = clamp_group(a.seq_to_group[s], G);
      nrc = resp_chunks(a.resp_lens[s], a.max_resp_pages, v.max_resp_chunks);
      np = prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, v.max_prefix_chunks) + nrc;
    }
    long long tot;
    const long long ex = block_exclusive_scan(pack2(np * Hq, nrc), s_buf, tot);
    if (s < S) {
      const int b = carry_p + hi32(ex);
      for (int j = 0; j < Hq; ++j) v.row_offs[(size_t)s * Hq + j] = b + j * np;
      const int r0 = carry_r + lo32(ex);
      for (int c = 0; c < nrc; ++c) v.resp_items[r0 + c] = make_int2(s, c);
    }
    carry_p += hi32(tot);
    carry_r += lo32(tot);
  }
  if (t == 0) {
    v.row_offs[(size_t)S * Hq] = carry_p;
    v.hdr[kHdrRespItems] = carry_r;
    v.hdr[kHdrParts] = carry_p;
  }
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t stream) {
  plan_kernel<<<1, kPlanThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rp
