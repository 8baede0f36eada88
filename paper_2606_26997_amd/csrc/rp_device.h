// Device-side helpers shared by the gfx950 kernels: vector types, bf16 and
// OCP e4m3fn conversions, wavefront reductions, and the work-plan layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rp {

// Tokens per KV page (the only page size the kernels are built for).
constexpr int kPage = 16;
// Pages per prefix work item, and the split of each response into work items:
// a response of P pages becomes floor(P / B) pieces of B pages and, if P is
// not a multiple of B, one ragged piece with the rest. Items are dispatched
// largest first (all B-sized pieces, then the ragged ones by decreasing
// size). The planner picks B per batch among kRespChunkStep, 2x, 3x and 4x
// that (32 to 128 pages): the multiple of kRespChunkStep nearest to
// W / (kRespChunkStep * kUnitsPerCu * compute units), W being the batch's
// response pages times its kv-heads, so that a batch has about kUnitsPerCu
// B-sized units per compute unit or more. Long pieces amortise each unit's
// start-up latency on big batches; small batches keep enough units in flight
// to fill the memory pipeline. Measured alternatives with extra small pieces
// at the end cost more start-ups than they saved. Batches whose work is below
// three quarters of one 32-page step take 16-page pieces instead, when the
// workspace was sized for them: a layout with at most
// kSmallBatchPageHeads page-heads of response capacity (sequences x table
// width x kv-heads) is sized for 16-page pieces, any other for 32.
constexpr int kPrefixChunkPages = 16;
constexpr int kRespChunkStep = 32;
constexpr int kRespChunkChoices = 4;
constexpr int kRespChunkPagesSmall = 16;
constexpr int kRespChunkPagesMin = kRespChunkStep;
constexpr int kRespChunkPagesMax = kRespChunkStep * kRespChunkChoices;
constexpr int kUnitsPerCu = 6;
constexpr long long kSmallBatchPageHeads = 1ll << 17;

constexpr float kLog2e = 1.4426950408889634f;
// Headroom of a lazily updated softmax running maximum, in log2 units: the
// maximum moves only when new scores exceed it by more than this, so the
// weights exp2(s - m) stay below 2^8 and most updates leave the output
// accumulator unscaled.
constexpr float kLazyMax = 8.0f;
constexpr float kLn2 = 0.6931471805599453f;

// Plan header slots.
enum : int {
  kHdrPrefixItems = 0,
  kHdrRespItems = 1,
  kHdrBigRespItems = 2,   // B-sized response items (they come first)
  kHdrRespChunkPages = 3,
  kHdrSlots = 16
};
// Largest group count the planner keeps in LDS.
constexpr int kPlanMaxGroups = 4096;
// Batches of at most this many sequences are planned by a single wave.
constexpr int kSmallPlanMaxSeqs = 64;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Pointers into a planned workspace (all device memory). Partial results of
// query row r = s * Hq + j live in slots r * parts_per_row + k: first the
// group's prefix chunks (k < prefix chunks of the group), then the sequence's
// response chunks.
struct PlanView {
  int* hdr;            // [kHdrSlots]
  int* grp_off;        // [G+1] CSR of members
  int* grp_members;    // [S]   members of each group in ascending order of arrival
  int2* prefix_items;  // [max_prefix_items]  (group, chunk)
  int4* resp_items;    // [max_resp_items]    (sequence, first page, tokens, slot), longest first
  int* seq_parts;      // [S] partial results per query row of each sequence
  float* part_o;       // [S*Hq*parts_per_row][D]
  float* part_lse;     // [S*Hq*parts_per_row]
  int max_prefix_chunks;  // per group
  int max_resp_chunks;    // response items per sequence (at the smaller big-item length)
  int parts_per_row;      // max_prefix_chunks + max_resp_chunks
  int max_parts;          // capacity of part_o / part_lse
  int max_prefix_items;   // capacity of prefix_items
  int max_resp_items;     // capacity of resp_items
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
// Two fp32 values to packed bf16 (low half first), round to nearest even, by
// gfx950's packed conversion (a NaN stays a NaN).
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
  typedef float f32x2_v __attribute__((ext_vector_type(2)));
  const f32x2_v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_v));
}

// ---- OCP e4m3fn -----------------------------------------------------------
// Decoding uses gfx950's conversion instructions, which implement OCP e4m3fn.
__device__ inline float e4m3_to_f32(uint32_t code) {
  return __builtin_amdgcn_cvt_f32_fp8((int)code, 0);
}

// fp32 -> e4m3fn code, round to nearest even, saturating at +-448. A NaN
// input (inf included among |x| >= 448) also takes the saturated code, with
// its sign bit: the append and page-write rules never store the NaN code.
__device__ inline uint32_t f32_to_e4m3(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  uint32_t code;
  if (a >= 0x43E00000u) {                 // |x| >= 448, inf or NaN
    code = 0x7Eu;
  } else if (a < 0x3C800000u) {           // |x| < 2^-6: subnormal grid of step 2^-9
    float q = __builtin_rintf(__uint_as_float(a) * 512.0f);  // exact scaling, RNE
    code = (uint32_t)q;                   // 0..8; 8 encodes 2^-6 exactly
  } else {
    const uint32_t e = (a >> 23) - 127u + 7u;   // 1..15 (2^-6 <= |x| < 448)
    const uint32_t m = a & 0x7FFFFFu;
    const uint32_t keep = m >> 20, rem = m & 0xFFFFFu;
    const uint32_t up = (rem > 0x80000u) || (rem == 0x80000u && (keep & 1u));
    code = (e << 3) + keep + up;          // a mantissa carry bumps the exponent
    if (code > 0x7Eu) code = 0x7Eu;
  }
  return code | sign;
}

// ---- the fp8 append rule --------------------------------------------------
// Row r of an fp8 (page, kv-head) block [16][D] takes a new token x. An
// aligned group of G lanes holds the row: element e of a lane sits at column
// col(e) (fp32 values of bf16 inputs); `leader` marks the one lane that
// stores the scale. amax = max |x| over the row; row 0 sets
// scale = amax / 448 (1 when amax is 0); a later row keeps the old scale when
// amax <= 448 * old, and otherwise sets scale = amax / 448 after requantising
// rows 0..r-1 from code * old. Plain IEEE fp32 (no contraction, correctly
// rounded division), so the bytes are a deterministic function of the inputs.
// Every lane of a G-lane group must call it, with the same r.
template <int D, int G, int N, class ColFn>
__device__ void append_fp8_row(uint8_t* blk, float* scale_slot, int r, const float (&x)[N], ColFn col,
                               bool leader) {
#pragma clang fp contract(off)
  float amax = 0.f;
#pragma unroll
  for (int e = 0; e < N; ++e) amax = fmaxf(amax, fabsf(x[e]));
#pragma unroll
  for (int o = 1; o < G; o <<= 1) amax = fmaxf(amax, __shfl_xor(amax, o));
  const float old = *scale_slot;
  float scale;
  if (r == 0) {
    scale = amax > 0.f ? amax / 448.0f : 1.0f;
  } else if (amax <= 448.0f * old) {
    scale = old;
  } else {
    scale = amax / 448.0f;
    // Requantise rows 0..r-1, four rows' codes in flight per memory round trip.
    constexpr int kRows = 4;
    for (int r0 = 0; r0 < r; r0 += kRows) {
      uint32_t c[kRows][N];
#pragma unroll
      for (int k = 0; k < kRows; ++k)
#pragma unroll
        for (int e = 0; e < N; ++e) c[k][e] = r0 + k < r ? blk[(size_t)(r0 + k) * D + col(e)] : 0u;
#pragma unroll
      for (int k = 0; k < kRows; ++k) {
        if (r0 + k >= r) break;
        uint8_t* row = blk + (size_t)(r0 + k) * D;
#pragma unroll
        for (int e = 0; e < N; ++e) row[col(e)] = (uint8_t)f32_to_e4m3(e4m3_to_f32(c[k][e]) * old / scale);
      }
    }
  }
  uint8_t* row = blk + (size_t)r * D;
#pragma unroll
  for (int e = 0; e < N; ++e) row[col(e)] = (uint8_t)f32_to_e4m3(x[e] / scale);
  if (leader) *scale_slot = scale;
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

// Max over lanes l, l^16, l^32, l^48 (the four quads of an MFMA tile column)
// with gfx950's row-swap instructions, which stay in the VALU: swapping the
// halves (rows) of two copies of x puts x[l] and x[l^32] (x[l^16]) into the
// two results of every lane.
__device__ inline float max_xor16_32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(x);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// MFMA tiles used by the group-prefix and prefill paths (fp32 accumulate).
// With lane l = 16 q + r (r < 16):
//   16x16x32 bf16: lane (r, q) supplies A[r][8q..8q+7] and B[8q..8q+7][r];
//   16x16x16 bf16: lane (r, q) supplies A[r][4q..4q+3] and B[4q..4q+3][r];
// lane (r, q) receives C[4q..4q+3][r].
// rp_selftest_mfma checks each of these against a matrix product.
__device__ inline f32x4_t mfma16x16x32(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ inline f32x4_t mfma16x16x16(const bf16x4_t& a, const bf16x4_t& b, const f32x4_t& c) {
  typedef short s16x4_t __attribute__((ext_vector_type(4)));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a), __builtin_bit_cast(s16x4_t, b),
                                                   c, 0, 0, 0);
}

// gfx950's transposing LDS read (ds_read_b64_tr_b16): within each 16-lane
// group, lane s supplies the address of 4 consecutive 16-bit elements, and
// lane j receives element j % 4 of the elements addressed by lanes j / 4,
// 4 + j / 4, 8 + j / 4 and 12 + j / 4, in that order. With lane s pointing at
// row r0 + s / 4, columns c0 + 4 (s % 4) ... + 3 of a row-major tile, lane j
// receives rows r0 .. r0 + 3 of column c0 + j.
__device__ inline bf16x4_t lds_read_tr(const uint16_t* p) {
  typedef short s16x4_t __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(
      bf16x4_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(p)));
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ inline float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace rp
