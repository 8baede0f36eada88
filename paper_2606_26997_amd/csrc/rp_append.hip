// KV append: one wave per (sequence, kv-head) writes the new token into
// response slot L = resp_lens[s] (page resp_block_table[s][L / 16], row L % 16).
// bf16 pools copy the values; fp8 pools apply the per-(page, kv-head) scale
// rule of append_fp8_row. Lane l handles columns l + 64 e.
#include "rp_device.h"
#include "rp_internal.h"

#pragma clang fp contract(off)

namespace rp {
namespace {

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
    uint16_t* kd = static_cast<uint16_t*>(a.k_pages) + blk + (size_t)r * D + lane;
    uint16_t* vd = static_cast<uint16_t*>(a.v_pages) + blk + (size_t)r * D + lane;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      kd[64 * e] = kn[64 * e + lane];
      vd[64 * e] = vn[64 * e + lane];
    }
  } else {
    const size_t sidx = (size_t)page * Hkv + h;
    float kx[EPL], vx[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      kx[e] = __uint_as_float((uint32_t)kn[64 * e + lane] << 16);
      vx[e] = __uint_as_float((uint32_t)vn[64 * e + lane] << 16);
    }
    const auto col = [lane](int e) { return lane + 64 * e; };
    append_fp8_row<D, 64>(static_cast<uint8_t*>(a.k_pages) + blk, a.k_scale + sidx, r, kx, col, lane == 0);
    append_fp8_row<D, 64>(static_cast<uint8_t*>(a.v_pages) + blk, a.v_scale + sidx, r, vx, col, lane == 0);
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
