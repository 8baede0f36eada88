// Self-test of the lane layouts that the attention and prefill kernels assume
// for gfx950's matrix cores and its transposing LDS read (rp_device.h): one
// wave forms the operands of a single MFMA from row-major A [M][K] and
// B [K][N] in those layouts and writes the accumulator back as C [M][N]
// under the output layout they assume, so C = A B exactly when the layouts
// hold (small integer inputs make every product and sum exact in fp32).
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

}  // namespace

hipError_t launch_selftest_mfma(int shape, const void* a, const void* b, float* c, hipStream_t stream) {
  selftest_mfma_kernel<<<1, 64, 0, stream>>>(shape, static_cast<const uint16_t*>(a),
                                             static_cast<const uint16_t*>(b), c);
  return hipGetLastError();
}

}  // namespace rp
