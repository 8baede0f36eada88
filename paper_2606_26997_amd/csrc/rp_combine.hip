// Log-sum-exp merge of partial results: one wave per output row.
//   lse = ln sum_i exp(lse_i),  out = sum_i exp(lse_i - lse) o_i
// Parts with lse_i = -inf are empty and their o_i is never added. A row's
// parts are read in batches: LPP lanes cover one part's head_dim with float4
// loads, so one load instruction fetches 64 / LPP parts and a batch keeps
// kBatch such loads in flight per wave. The first batch's partial outputs are
// requested together with their lse values, before the row maximum is known.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kCombineWaves = 4;
constexpr int kBatch = 8;

template <int D>
__device__ inline void load_batch(const CombineArgs& a, int p0, int n, int base, int slot, int sub, float* lp,
                                  float4* ov) {
  constexpr int PPI = 64 / (D / 4);
#pragma unroll
  for (int b = 0; b < kBatch; ++b) {
    const int k = base + b * PPI + slot;
    lp[b] = -INFINITY;
    ov[b] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (k < n) {
      lp[b] = a.lse_parts[p0 + k];
      ov[b] = *reinterpret_cast<const float4*>(a.o_parts + (size_t)(p0 + k) * D + sub * 4);
    }
  }
}

__device__ inline void add_batch(const float* lp, const float4* ov, float mx, float4& acc, float& wsum) {
#pragma unroll
  for (int b = 0; b < kBatch; ++b) {
    const bool live = lp[b] != -INFINITY;
    const float w = live ? fast_exp2((lp[b] - mx) * kLog2e) : 0.f;
    wsum += w;
    acc.x = live ? fmaf(w, ov[b].x, acc.x) : acc.x;
    acc.y = live ? fmaf(w, ov[b].y, acc.y) : acc.y;
    acc.z = live ? fmaf(w, ov[b].z, acc.z) : acc.z;
    acc.w = live ? fmaf(w, ov[b].w, acc.w) : acc.w;
  }
}

template <int D>
__global__ __launch_bounds__(64 * kCombineWaves) void combine_kernel(const CombineArgs a) {
  constexpr int LPP = D / 4;     // lanes per part
  constexpr int PPI = 64 / LPP;  // parts per load instruction
  const int row = blockIdx.x * kCombineWaves + (threadIdx.x >> 6);
  if (row >= a.num_rows) return;
  const int lane = threadIdx.x & 63;
  const int slot = lane / LPP, sub = lane - slot * LPP;

  int p0, n;
  if (a.row_offs != nullptr) {
    p0 = a.row_offs[row];
    n = a.row_offs[row + 1] - p0;
  } else {
    n = min(max(a.seq_parts[row / a.num_q_heads], 0), a.parts_per_row);
    p0 = row * a.parts_per_row;
  }

  float lp[kBatch];
  float4 ov[kBatch];
  load_batch<D>(a, p0, n, 0, slot, sub, lp, ov);
  float mx = -INFINITY;
#pragma unroll
  for (int b = 0; b < kBatch; ++b) mx = fmaxf(mx, lp[b]);
  for (int i = PPI * kBatch + lane; i < n; i += 64) mx = fmaxf(mx, a.lse_parts[p0 + i]);
  mx = xor_max_from<1>(mx);

  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float wsum = 0.f;
  if (mx != -INFINITY) {
    add_batch(lp, ov, mx, acc, wsum);
    for (int base = PPI * kBatch; base < n; base += PPI * kBatch) {
      load_batch<D>(a, p0, n, base, slot, sub, lp, ov);
      add_batch(lp, ov, mx, acc, wsum);
    }
  }
  acc.x = xor_sum_from<LPP>(acc.x);
  acc.y = xor_sum_from<LPP>(acc.y);
  acc.z = xor_sum_from<LPP>(acc.z);
  acc.w = xor_sum_from<LPP>(acc.w);
  wsum = xor_sum_from<LPP>(wsum);

  if (slot == 0) {
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    uint2 packed;
    packed.x = pack_bf16x2(acc.x * inv, acc.y * inv);
    packed.y = pack_bf16x2(acc.z * inv, acc.w * inv);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + (size_t)row * D + sub * 4) = packed;
  }
  if (a.lse != nullptr && lane == 0) a.lse[row] = wsum > 0.f ? mx + fast_log2(wsum) * kLn2 : -INFINITY;
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, int head_dim, hipStream_t stream) {
  if (a.num_rows <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)cdiv(a.num_rows, kCombineWaves);
  if (head_dim == 128) combine_kernel<128><<<blocks, 64 * kCombineWaves, 0, stream>>>(a);
  else if (head_dim == 64) combine_kernel<64><<<blocks, 64 * kCombineWaves, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace rp
