// Log-sum-exp merge of partial results: one wave per output row.
//   lse = ln sum_i exp(lse_i),  out = sum_i exp(lse_i - lse) o_i
// Parts with lse_i = -inf are empty and their o_i is never read into the sum.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kCombineWaves = 4;

template <int D>
__global__ __launch_bounds__(64 * kCombineWaves) void combine_kernel(const CombineArgs a) {
  constexpr int EPL = D / 64;  // output elements per lane
  const int row = blockIdx.x * kCombineWaves + (threadIdx.x >> 6);
  if (row >= a.num_rows) return;
  const int lane = threadIdx.x & 63;
  const int p0 = a.row_offs[row], p1 = a.row_offs[row + 1];

  float mx = -INFINITY;
  for (int p = p0 + lane; p < p1; p += 64) mx = fmaxf(mx, a.lse_parts[p]);
  mx = xor_max_from<1>(mx);

  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
  float wsum = 0.f;
  if (mx != -INFINITY) {
#pragma unroll 4
    for (int p = p0; p < p1; ++p) {
      const float lp = a.lse_parts[p];
      const float w = fast_exp2((lp - mx) * kLog2e);  // 0 for an empty part
      const float* src = a.o_parts + (size_t)p * D + lane * EPL;
      float ov[EPL];
      if constexpr (EPL == 2) {
        const float2 t = *reinterpret_cast<const float2*>(src);
        ov[0] = t.x;
        ov[1] = t.y;
      } else {
        ov[0] = src[0];
      }
      const bool live = lp != -INFINITY;
      wsum += w;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = live ? fmaf(w, ov[e], acc[e]) : acc[e];
    }
  }

  uint16_t* out = static_cast<uint16_t*>(a.out) + (size_t)row * D + lane * EPL;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  if constexpr (EPL == 2) {
    *reinterpret_cast<uint32_t*>(out) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  } else {
    out[0] = (uint16_t)f32_to_bf16_bits(acc[0] * inv);
  }
  if (a.lse != nullptr && lane == 0)
    a.lse[row] = wsum > 0.f ? mx + fast_log2(wsum) * kLn2 : -INFINITY;
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
