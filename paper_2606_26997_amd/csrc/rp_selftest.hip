// Self-test and measurement probes.
//
// Lane layouts: the attention and prefill kernels assume fixed lane layouts
// for gfx950's matrix cores and its transposing LDS read (rp_device.h); one
// wave forms the operands of a single MFMA from row-major A [M][K] and
// B [K][N] in those layouts and writes the accumulator back as C [M][N]
// under the output layout they assume, so C = A B exactly when the layouts
// hold (small integer inputs make every product and sum exact in fp32).
//
// Streaming read: the HBM read rate a plain kernel reaches on the device,
// the practical ceiling for the memory-bound decode kernels.
#include "rp.h"
#include "rp_internal.h"

namespace rp {
namespace {

typedef unsigned short u16x8_t __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4_t __attribute__((ext_vector_type(4)));

constexpr int kTrPitch = 32;  // staged A^T rows (bf16), 8-byte aligned rows

// bf16 elements src[idx(0)] .. src[idx(7)] as an MFMA operand.
template <class F>
__device__ inline bf16x8_t gather8(const uint16_t* src, F idx) {
  u16x8_t v;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = src[idx(j)];
  return __builtin_bit_cast(bf16x8_t, v);
}

__global__ __launch_bounds__(64) void selftest_mfma_kernel(int shape, const uint16_t* a, const uint16_t* b,
                                                           float* c) {
  __shared__ __attribute__((aligned(16))) uint16_t at[32 * kTrPitch];  // A^T, 32 keys x 16 columns
  const int l = threadIdx.x;
  const int r = l & 15, q = l >> 4;  // 16x16 tiles: lane (r, q)
  if (shape == RP_SELFTEST_MFMA_16X16X32) {
    constexpr int K = 32, N = 16;
    const bf16x8_t av = gather8(a, [&](int j) { return r * K + 8 * q + j; });
    const bf16x8_t bv = gather8(b, [&](int j) { return (8 * q + j) * N + r; });
    const f32x4_t acc = mfma16x16x32(av, bv, f32x4_t{0.f, 0.f, 0.f, 0.f});
#pragma unroll
    for (int i = 0; i < 4; ++i) c[(4 * q + i) * N + r] = acc[i];
  } else if (shape == RP_SELFTEST_MFMA_16X16X16) {
    constexpr int K = 16, N = 16;
    u16x4_t av, bv;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      av[j] = a[r * K + 4 * q + j];
      bv[j] = b[(4 * q + j) * N + r];
    }
    const f32x4_t acc = mfma16x16x16(__builtin_bit_cast(bf16x4_t, av), __builtin_bit_cast(bf16x4_t, bv),
                                     f32x4_t{0.f, 0.f, 0.f, 0.f});
#pragma unroll
    for (int i = 0; i < 4; ++i) c[(4 * q + i) * N + r] = acc[i];
  } else if (shape == RP_SELFTEST_MFMA_16X16X32_LDS_TR) {
    // The prefill's P V with 16x16 tiles: A^T (keys x columns) staged
    // row-major; lane (r, q) takes column r of keys 4q .. 4q+3 and
    // 16+4q .. 16+4q+3, and its B entries follow the same key order.
    constexpr int M = 16, K = 32, N = 16;
    for (int i = l; i < M * K; i += 64) at[(i % K) * kTrPitch + i / K] = a[i];
    __syncthreads();
    const uint16_t* p = at + (4 * q + r / 4) * kTrPitch + 4 * (r % 4);
    const bf16x4_t a0 = lds_read_tr(p), a1 = lds_read_tr(p + 16 * kTrPitch);
    const bf16x8_t av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    const bf16x8_t bv = gather8(b, [&](int j) { return (j < 4 ? 4 * q + j : 12 + 4 * q + j) * N + r; });
    const f32x4_t acc = mfma16x16x32(av, bv, f32x4_t{0.f, 0.f, 0.f, 0.f});
#pragma unroll
    for (int i = 0; i < 4; ++i) c[(4 * q + i) * N + r] = acc[i];
  }
}

// Workgroup b reads the b-th of RP_STREAM_READ_BLOCKS contiguous chunks of
// the buffer, kUnroll 16-byte loads per thread issued before any is used
// (load u of a round covers the round's piece u * threads + t). Measured on
// a 4 GiB buffer, contiguous chunks read faster than a grid-wide stride (7.0
// against 6.6-6.7 TB/s with non-temporal loads, 6.2 against 6.0 without).
// Each wave folds its words with XOR and lane 0 writes the result, so no
// load can be dropped or moved behind a branch.
constexpr int kStreamThreads = 256, kStreamUnroll = 8;
typedef uint32_t u32x4s_t __attribute__((ext_vector_type(4)));

template <bool NT>
__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4s_t* src, uint64_t n16,
                                                                     uint32_t* sink) {
  const uint64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const uint64_t lo = (uint64_t)blockIdx.x * per;
  const uint64_t hi = lo + per < n16 ? lo + per : n16;
  uint32_t acc = 0;
  for (uint64_t base = lo; base < hi; base += (uint64_t)kStreamThreads * kStreamUnroll) {
    u32x4s_t v[kStreamUnroll];
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) {
      const uint64_t i = base + (uint64_t)u * kStreamThreads + threadIdx.x;
      v[u] = u32x4s_t{0u, 0u, 0u, 0u};
      if (i < hi) v[u] = NT ? __builtin_nontemporal_load(src + i) : src[i];
    }
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * (kStreamThreads / 64) + (threadIdx.x >> 6)] = acc;
}

}  // namespace

hipError_t launch_stream_read(const void* src, uint64_t bytes, uint32_t* sink, bool nontemporal,
                              hipStream_t stream) {
  static_assert(RP_STREAM_READ_BLOCKS * (kStreamThreads / 64) == RP_STREAM_READ_SINK_WORDS, "sink size");
  const auto* p = static_cast<const u32x4s_t*>(src);
  if (nontemporal) stream_read_kernel<true><<<RP_STREAM_READ_BLOCKS, kStreamThreads, 0, stream>>>(p, bytes / 16, sink);
  else stream_read_kernel<false><<<RP_STREAM_READ_BLOCKS, kStreamThreads, 0, stream>>>(p, bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_selftest_mfma(int shape, const void* a, const void* b, float* c, hipStream_t stream) {
  selftest_mfma_kernel<<<1, 64, 0, stream>>>(shape, static_cast<const uint16_t*>(a),
                                             static_cast<const uint16_t*>(b), c);
  return hipGetLastError();
}

}  // namespace rp
