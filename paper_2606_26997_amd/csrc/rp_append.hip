// KV append: one wave per (sequence, kv-head) writes the new token into
// response slot L = resp_lens[s] (page resp_block_table[s][L / 16], row L % 16).
// bf16 pools copy the values. fp8 pools quantise with the per-(page, kv-head)
// scale rule: row 0 sets scale = amax / 448; a later row keeps the scale when
// amax <= 448 * scale, and otherwise raises it to amax / 448 after
// requantising rows 0..r-1 from code * old_scale. All of it is plain IEEE fp32
// (no contraction, correctly rounded division), so the bytes written are a
// deterministic function of the inputs.
#include "rp_device.h"
#include "rp_internal.h"

#pragma clang fp contract(off)

namespace rp {
namespace {

template <int D>
__device__ void append_fp8_head(uint8_t* blk, float* scale_slot, int r, const uint16_t* x_bits, int lane) {
  constexpr int EPL = D / 64;
  float x[EPL];
  float amax = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    x[e] = __uint_as_float((uint32_t)x_bits[lane * EPL + e] << 16);
    amax = fmaxf(amax, fabsf(x[e]));
  }
  amax = xor_max_from<1>(amax);
  const float old = *scale_slot;
  float scale;
  if (r == 0) {
    scale = amax > 0.f ? amax / 448.0f : 1.0f;
  } else if (amax <= 448.0f * old) {
    scale = old;
  } else {
    scale = amax / 448.0f;
    for (int rr = 0; rr < r; ++rr) {
      uint8_t* row = blk + (size_t)rr * D + lane * EPL;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float val = e4m3_to_f32(row[e]) * old;
        row[e] = (uint8_t)f32_to_e4m3(val / scale);
      }
    }
  }
  uint8_t* row = blk + (size_t)r * D + lane * EPL;
#pragma unroll
  for (int e = 0; e < EPL; ++e) row[e] = (uint8_t)f32_to_e4m3(x[e] / scale);
  if (lane == 0) *scale_slot = scale;
}

template <int D, bool FP8>
__global__ __launch_bounds__(64) void append_kernel(const AppendArgs a) {
  constexpr int EPL = D / 64;
  const int Hkv = a.num_kv_heads;
  const int s = blockIdx.x / Hkv;
  const int h = blockIdx.x - s * Hkv;
  const int L = a.resp_lens[s];
  if (L < 0 || L >= a.max_resp_pages * kPage) return;  // no slot for the new token
  const int page = clamp_page(a.resp_block_table[(size_t)s * a.max_resp_pages + L / kPage], a.num_pages);
  const int r = L % kPage;
  const int lane = threadIdx.x;
  const size_t head_off = ((size_t)s * Hkv + h) * D;
  const uint16_t* kn = static_cast<const uint16_t*>(a.k_new) + head_off;
  const uint16_t* vn = static_cast<const uint16_t*>(a.v_new) + head_off;
  const size_t blk = ((size_t)page * Hkv + h) * kPage * D;  // in elements
  if constexpr (!FP8) {
    uint16_t* kd = static_cast<uint16_t*>(a.k_pages) + blk + (size_t)r * D + lane * EPL;
    uint16_t* vd = static_cast<uint16_t*>(a.v_pages) + blk + (size_t)r * D + lane * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      kd[e] = kn[lane * EPL + e];
      vd[e] = vn[lane * EPL + e];
    }
  } else {
    const size_t sidx = (size_t)page * Hkv + h;
    append_fp8_head<D>(static_cast<uint8_t*>(a.k_pages) + blk, a.k_scale + sidx, r, kn, lane);
    append_fp8_head<D>(static_cast<uint8_t*>(a.v_pages) + blk, a.v_scale + sidx, r, vn, lane);
  }
}

// Layout checker (test utility): records the number of bad entries and one example.
__device__ void report(int* res, int kind, int index, int value) {
  if (atomicAdd(&res[0], 1) == 0) {
    res[1] = kind;
    res[2] = index;
    res[3] = value;
  }
}

__global__ __launch_bounds__(256) void validate_kernel(const ValidateArgs a) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int nt = gridDim.x * blockDim.x;
  for (int s = t; s < a.num_seqs; s += nt) {
    const int g = a.seq_to_group[s];
    if (g < 0 || g >= a.num_groups) report(a.result, 1, s, g);
    const int L = a.resp_lens[s];
    if (L < 0 || L > a.max_resp_pages * kPage) {
      report(a.result, 3, s, L);
      continue;
    }
    for (int p = 0; p < cdiv(L, kPage); ++p) {
      const int page = a.resp_block_table[(size_t)s * a.max_resp_pages + p];
      if (page < 0 || page >= a.num_pages) report(a.result, 5, s, page);
    }
  }
  for (int g = t; g < a.num_groups; g += nt) {
    const int P = a.prefix_lens[g];
    if (P < 0 || P > a.max_prefix_pages * kPage) {
      report(a.result, 2, g, P);
      continue;
    }
    for (int p = 0; p < cdiv(P, kPage); ++p) {
      const int page = a.prefix_block_table[(size_t)g * a.max_prefix_pages + p];
      if (page < 0 || page >= a.num_pages) report(a.result, 4, g, page);
    }
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int head_dim, bool fp8, hipStream_t stream) {
  const long long blocks = (long long)a.num_seqs * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(64);
  if (head_dim == 128) {
    if (fp8) append_kernel<128, true><<<grid, block, 0, stream>>>(a);
    else append_kernel<128, false><<<grid, block, 0, stream>>>(a);
  } else if (head_dim == 64) {
    if (fp8) append_kernel<64, true><<<grid, block, 0, stream>>>(a);
    else append_kernel<64, false><<<grid, block, 0, stream>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateArgs& a, hipStream_t stream) {
  validate_kernel<<<64, 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rp
