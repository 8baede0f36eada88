// Device-side helpers shared by the gfx950 kernels: vector types, bf16 and
// OCP e4m3fn conversions, wavefront reductions, and the work-plan layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rp {

// Tokens per KV page (the only page size the kernels are built for).
constexpr int kPage = 16;
// Pages per response work item (split-KV chunk) and per prefix work item.
constexpr int kRespChunkPages = 16;
constexpr int kPrefixChunkPages = 4;
// Query-row tiles (16 rows each) one prefix wave keeps in registers per pass.
constexpr int kPrefixTiles = 2;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Plan header slots.
enum : int { kHdrPrefixItems = 0, kHdrRespItems = 1, kHdrParts = 2, kHdrSlots = 16 };

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Pointers into a planned workspace (all device memory).
struct PlanView {
  int* hdr;            // [kHdrSlots]
  int* grp_count;      // [G]  live members per group
  int* grp_fill;       // [G]  placement cursor
  int* grp_off;        // [G+1] CSR of members
  int* grp_members;    // [S]
  int2* prefix_items;  // [max_prefix_items]  (group, chunk)
  int2* resp_items;    // [max_resp_items]    (sequence, chunk)
  int* row_offs;       // [S*Hq + 1] CSR of partial results per (sequence, query head)
  float* part_o;       // [max_parts][D]
  float* part_lse;     // [max_parts]
  int max_prefix_chunks;  // per group
  int max_resp_chunks;    // per sequence
  int max_parts;          // capacity of part_o / part_lse
};

// Partial-result slot, kept inside the workspace even for a workspace that was
// never planned (garbage offsets then give garbage numbers, not stray writes).
__device__ inline int clamp_part(int p, int max_parts) {
  return (unsigned)p < (unsigned)max_parts ? p : 0;
}

// ---- bf16 ---------------------------------------------------------------
__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ inline uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// ---- OCP e4m3fn -----------------------------------------------------------
// Exact decode of two codes (bytes 0 and 1 of `w` when hi == false, bytes 2
// and 3 otherwise) to fp32. Each code's 7 magnitude bits are placed as an
// fp16 with exponent field e and mantissa m << 7, which equals the e4m3 value
// times 2^-8 for normal and subnormal codes alike; the caller folds the 2^8
// into its per-page scale. The NaN code (S.1111.111) is never produced by the
// append path and decodes to 480 here.
__device__ inline void e4m3x2_to_f32_scaled(uint32_t w, bool hi, float& a, float& b) {
  uint32_t x = hi ? (w >> 16) : w;  // codes in bits 0..7 and 8..15
  // Spread byte 1 into bits 16..23: x' = b0 | b1 << 16.
  uint32_t sp = (x & 0xFFu) | ((x & 0xFF00u) << 8);
  uint32_t h = ((sp & 0x00800080u) << 8) | ((sp & 0x007F007Fu) << 7);
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  f16x2_t hv = __builtin_bit_cast(f16x2_t, h);
  a = (float)hv[0];
  b = (float)hv[1];
}
constexpr float kE4m3DecodeScale = 256.0f;  // undoes the 2^-8 of e4m3x2_to_f32_scaled

// fp32 -> e4m3fn code, round to nearest even, saturating at +-448.
__device__ inline uint32_t f32_to_e4m3(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  uint32_t code;
  if (a >= 0x43E00000u) {                 // |x| >= 448 (or inf)
    code = 0x7Eu;
  } else if (a < 0x3C800000u) {           // |x| < 2^-6: subnormal grid of step 2^-9
    float q = __builtin_rintf(__uint_as_float(a) * 512.0f);  // exact scaling, RNE
    code = (uint32_t)q;                   // 0..8; 8 encodes 2^-6 exactly
  } else {
    const uint32_t e = (a >> 23) - 127u + 7u;   // 1..8
    const uint32_t m = a & 0x7FFFFFu;
    const uint32_t keep = m >> 20, rem = m & 0xFFFFFu;
    const uint32_t up = (rem > 0x80000u) || (rem == 0x80000u && (keep & 1u));
    code = (e << 3) + keep + up;          // a mantissa carry bumps the exponent
    if (code > 0x7Eu) code = 0x7Eu;
  }
  return code | sign;
}

// ---- wavefront reductions -----------------------------------------------
template <int CTRL>
__device__ inline float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadSwap1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;

// Sum over aligned groups of N lanes (N in {4, 8, 16}); every lane of a group
// gets the same, bitwise identical, total.
template <int N>
__device__ inline float group_sum(float x) {
  static_assert(N == 4 || N == 8 || N == 16, "group size");
  x += dpp<kQuadSwap1>(x);
  x += dpp<kQuadSwap2>(x);
  if constexpr (N >= 8) x += dpp<kRowHalfMirror>(x);
  if constexpr (N >= 16) x += dpp<kRowMirror>(x);
  return x;
}

// Butterfly over the lanes that differ only in bits >= log2(FIRST) of the lane id.
template <int FIRST>
__device__ inline float xor_max_from(float x) {
#pragma unroll
  for (int o = FIRST; o < 64; o <<= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
template <int FIRST>
__device__ inline float xor_sum_from(float x) {
#pragma unroll
  for (int o = FIRST; o < 64; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ inline float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace rp
