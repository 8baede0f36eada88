// Partial attention over planned work items, in one launch. Work units are
// (item, kv-head) pairs, one per one-wave block: all group-prefix units first,
// then the response units longest first, so the hardware dispatcher hands the
// last free slots the smallest units.
//
// Group-prefix units (MFMA): every response of a GRPO group is sampled from
// the same prompt, so the group's prompt-prefix KV is read once per (group,
// kv-head, chunk) and applied to all of the group's query rows at once: live
// members x (Hq / Hkv) query heads as 16-row tiles, one page per step:
//   S^T  = K Q^T   on mfma 16x16x32 bf16 (M = 16 tokens, N = 16 rows, K = 32 of head_dim)
//   O^T += V^T P^T on mfma 16x16x16 bf16 (M = 16 head_dim columns, N = 16 rows, K = 16 tokens)
// with fp32 accumulation and an online softmax; the page's V goes through LDS
// to feed the transposed operand.
//
// Response units (VALU): one (sequence, chunk of response pages, kv-head). A
// (page, kv-head) block is contiguous in the pool and is read with fully
// coalesced 16-byte loads: lane l holds EPL head_dim elements of token
// (load * TPL + l / LPT). Scores are reduced over the LPT lanes of a token with
// DPP, every group of LPT lanes keeps its own online-softmax state, and the
// states are merged once per unit. Page loads are software-pipelined: the next
// page's K is requested as soon as this page's scores exist and its V as soon as
// this page's V is unpacked (for fp8 pools, whose blocks are half the bytes, the
// page two ahead, so that two pages are in flight). How responses split into
// items is the planner's choice for the batch.
//
// Each unit writes one partial (o normalised, lse natural-log) per query row
// into its fixed slot (row, chunk); the combine kernel merges a row's parts.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

// Waves per work unit: the unit's pages are dealt round-robin to the waves of
// one workgroup and the waves' softmax states are merged through LDS at the
// end, so a unit drains kUnitWaves times faster without adding partial
// results. One wave per unit measured best once V is read non-temporally (two
// waves tie on short responses and lose 1-2% on long ones).
constexpr int kUnitWaves = 1;
constexpr int kUnitThreads = 64 * kUnitWaves;

// V pages are read with the non-temporal hint and K pages without it: both
// streams are read exactly once, and marking one of the two (either one) as
// streaming was measured 6-8% faster on every workload than marking neither
// or both.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ inline uint4 load_v_stream(const char* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Orders this wave's LDS accesses (its staging area is its own).
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// LDS of one workgroup: the staged V page of each wave (prefix units), reused
// for the waves' states while they merge, then the query tile of each wave
// (prefix units). Row pitches are padded so that the column-wise and
// row-wise reads of the MFMA operands do not collide on LDS banks.
template <int D, int NREP>
struct Smem {
  static constexpr int kVStride = D + 4;  // staged V row pitch (bf16)
  static constexpr int kQStride = D + 8;  // query tile row pitch (bf16)
  static constexpr int kStage = kUnitWaves * kPage * kVStride * 2;
  static constexpr int kPrefixMerge = (kUnitWaves - 1) * 64 * (2 + D / 16 * 4) * 4;
  static constexpr int kRespMerge = (kUnitWaves - 1) * NREP * (D + 2) * 4;
  static constexpr int kQOff = kStage > kPrefixMerge ? (kStage > kRespMerge ? kStage : kRespMerge)
                                                     : (kPrefixMerge > kRespMerge ? kPrefixMerge : kRespMerge);
  static constexpr int kBytes = kQOff + kUnitWaves * 16 * kQStride * 2;
};

// ---------------------------------------------------------------------------
// Response path
// ---------------------------------------------------------------------------
template <int D, bool FP8>
struct RespGeom {
  static constexpr int EB = FP8 ? 1 : 2;          // bytes per KV element
  static constexpr int EPL = 16 / EB;             // elements per lane per 16-byte load
  static constexpr int LPT = D / EPL;             // lanes per token
  static constexpr int TPL = 64 / LPT;            // tokens per load instruction
  static constexpr int LOADS = kPage / TPL;       // loads per (page, kv-head) block
  static constexpr int BLOCK_BYTES = kPage * D * EB;
  static constexpr int QW = EPL / 8;              // uint4 words of bf16 q per lane per row
};

__device__ inline float dot2_bf16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), acc,
                                         false);
}
__device__ inline float dot8_bf16(const uint4& a, const uint4& b, float acc) {
  acc = dot2_bf16(a.x, b.x, acc);
  acc = dot2_bf16(a.y, b.y, acc);
  acc = dot2_bf16(a.z, b.z, acc);
  return dot2_bf16(a.w, b.w, acc);
}

__device__ inline void unpack_bf16x8(const uint4& w, float* f) {
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
  f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
  f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

// 4 e4m3 codes -> 4 exact floats (gfx950 converts OCP e4m3fn in hardware).
__device__ inline void e4m3x4_to_f32(uint32_t w, float* f) {
  const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  f[0] = lo[0];
  f[1] = lo[1];
  f[2] = hi[0];
  f[3] = hi[1];
}
__device__ inline void unpack_e4m3x16(const uint4& w, float* f) {
  e4m3x4_to_f32(w.x, f);
  e4m3x4_to_f32(w.y, f + 4);
  e4m3x4_to_f32(w.z, f + 8);
  e4m3x4_to_f32(w.w, f + 12);
}
// 8 e4m3 codes -> 8 bf16 values (exact: every e4m3 value is a bf16 value), by
// gfx950's scaled conversion with scale 1: two codes per instruction.
template <bool HIGH>
__device__ inline uint32_t e4m3x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HIGH));
}
__device__ inline uint4 e4m3x8_to_bf16x8(uint32_t w0, uint32_t w1) {
  return make_uint4(e4m3x2_to_bf16x2<false>(w0), e4m3x2_to_bf16x2<true>(w0), e4m3x2_to_bf16x2<false>(w1),
                    e4m3x2_to_bf16x2<true>(w1));
}

template <int D, bool FP8>
__device__ inline size_t resp_block(const AttnArgs& a, int page, int h, int lane) {
  return ((size_t)page * a.num_kv_heads + h) * RespGeom<D, FP8>::BLOCK_BYTES + (size_t)lane * 16;
}

// ---------------------------------------------------------------------------
// Group-prefix path
// ---------------------------------------------------------------------------

// One page of a prefix unit in flight, as loaded (this lane's share):
//  k: the A operand of S^T = K Q^T, lane (r16, quad) holds
//     K[token r16][kb*32 + quad*8 + 0..7] (8 bf16, or 8 e4m3 codes);
//  v: 16-byte pieces of the page's V block, lane-contiguous, for staging;
//  ks, vs: the fp8 scales of the page.
template <int D, bool FP8>
struct PrefixPage {
  static constexpr int KB = D / 32;
  static constexpr int VL = (FP8 ? kPage * D : kPage * D * 2) / 1024;
  uint4 k[FP8 ? (KB + 1) / 2 : KB];
  uint4 v[VL];
  float ks, vs;
};

// Every load of the page is unconditional: padding rows of a ragged page are
// read (they are inside the page) and masked when used.
template <int D, bool FP8>
__device__ inline void load_prefix_k(const AttnArgs& a, const char* kpool, int pg, int h, int lane,
                                     PrefixPage<D, FP8>& r) {
  constexpr size_t BLOCK_BYTES = (size_t)kPage * D * (FP8 ? 1 : 2);
  const size_t blk = ((size_t)pg * a.num_kv_heads + h) * BLOCK_BYTES;
  const int r16 = lane & 15, quad = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < D / 32; ++kb) {
    const int col = kb * 32 + quad * 8;
    if constexpr (!FP8) {
      r.k[kb] = *reinterpret_cast<const uint4*>(kpool + blk + ((size_t)r16 * D + col) * 2);
    } else {
      const uint2 w = *reinterpret_cast<const uint2*>(kpool + blk + (size_t)r16 * D + col);
      if (kb % 2 == 0) { r.k[kb / 2].x = w.x; r.k[kb / 2].y = w.y; }
      else { r.k[kb / 2].z = w.x; r.k[kb / 2].w = w.y; }
    }
  }
  if constexpr (FP8) r.ks = a.k_scale[(size_t)pg * a.num_kv_heads + h];
}
template <int D, bool FP8>
__device__ inline void load_prefix_v(const AttnArgs& a, const char* vpool, int pg, int h, int lane,
                                     PrefixPage<D, FP8>& r) {
  constexpr size_t BLOCK_BYTES = (size_t)kPage * D * (FP8 ? 1 : 2);
  const size_t blk = ((size_t)pg * a.num_kv_heads + h) * BLOCK_BYTES;
#pragma unroll
  for (int i = 0; i < PrefixPage<D, FP8>::VL; ++i)
    r.v[i] = load_v_stream(vpool + blk + (size_t)i * 1024 + lane * 16);
  if constexpr (FP8) r.vs = a.v_scale[(size_t)pg * a.num_kv_heads + h];
}

template <int D, bool FP8>
__device__ inline bf16x8_t prefix_k_operand(const PrefixPage<D, FP8>& r, int kb) {
  if constexpr (!FP8) {
    return __builtin_bit_cast(bf16x8_t, r.k[kb]);
  } else {
    const uint4& w = r.k[kb / 2];
    return __builtin_bit_cast(bf16x8_t, kb % 2 == 0 ? e4m3x8_to_bf16x8(w.x, w.y) : e4m3x8_to_bf16x8(w.z, w.w));
  }
}

// Write the page's V block (bf16, or fp8 decoded to bf16) into LDS rows
// 0..15; rows at or beyond `nvalid` are written as zeros.
template <int D, bool FP8, int STRIDE>
__device__ inline void stage_v(const PrefixPage<D, FP8>& r, int nvalid, uint16_t* vt, int lane) {
#pragma unroll
  for (int i = 0; i < PrefixPage<D, FP8>::VL; ++i) {
    if constexpr (!FP8) {
      const int e0 = i * 512 + lane * 8;
      const int tok = e0 / D, col = e0 % D;
      const uint4 w = tok < nvalid ? r.v[i] : make_uint4(0, 0, 0, 0);
      uint2* dst = reinterpret_cast<uint2*>(vt + tok * STRIDE + col);
      dst[0] = make_uint2(w.x, w.y);
      dst[1] = make_uint2(w.z, w.w);
    } else {
      const int e0 = i * 1024 + lane * 16;
      const int tok = e0 / D, col = e0 % D;
      uint4 lo = make_uint4(0, 0, 0, 0), hi = make_uint4(0, 0, 0, 0);
      if (tok < nvalid) {
        lo = e4m3x8_to_bf16x8(r.v[i].x, r.v[i].y);
        hi = e4m3x8_to_bf16x8(r.v[i].z, r.v[i].w);
      }
      uint2* dst = reinterpret_cast<uint2*>(vt + tok * STRIDE + col);
      dst[0] = make_uint2(lo.x, lo.y);
      dst[1] = make_uint2(lo.z, lo.w);
      dst[2] = make_uint2(hi.x, hi.y);
      dst[3] = make_uint2(hi.z, hi.w);
    }
  }
}

// One group-prefix unit: kv-head h of (group, chunk of prefix pages), for all
// query rows of the group's live members, 16 rows per pass and one page per
// step. A group with more than 16 query rows reads the chunk again for each
// further pass; the chunk (a few tens of KiB) is then still in this XCD's L2.
template <int D, int NREP, bool FP8>
__device__ void prefix_unit(const AttnArgs& a, int item, int h, char* smem) {
  constexpr int KB = D / 32;       // MFMA k-blocks over head_dim
  constexpr int DT = D / 16;       // 16-column output tiles over head_dim
  constexpr int STRIDE = Smem<D, NREP>::kVStride;
  constexpr int QSTRIDE = Smem<D, NREP>::kQStride;
  const int2 it = a.view.prefix_items[item];
  const int g = clamp_group(it.x, a.num_groups);
  const int c = min(max(it.y, 0), a.view.max_prefix_chunks - 1);
  const int P = clamp_len(a.prefix_lens[g], a.max_prefix_pages);
  const int tok0 = c * (kPrefixChunkPages * kPage);
  const int ntok = min(kPrefixChunkPages * kPage, P - tok0);
  const int npages = cdiv(ntok, kPage);
  const int moff = a.view.grp_off[g];
  const int R = (a.view.grp_off[g + 1] - moff) * NREP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, quad = lane >> 4;
  uint16_t* vt = reinterpret_cast<uint16_t*>(smem) + wave * (kPage * STRIDE);
  uint16_t* qt = reinterpret_cast<uint16_t*>(smem + Smem<D, NREP>::kQOff) + wave * (16 * QSTRIDE);
  uint16_t* qt_lane = qt + r16 * QSTRIDE + quad * 8;  // this lane's 16-byte pieces of its row
  const int* bt = a.prefix_block_table + (size_t)g * a.max_prefix_pages + c * kPrefixChunkPages;
  const char* kpool = static_cast<const char*>(a.k_pages);
  const char* vpool = static_cast<const char*>(a.v_pages);
  const uint16_t* qall = static_cast<const uint16_t*>(a.q);

  for (int r0 = 0; r0 < R; r0 += 16) {
    const int rr = r0 + r16;
    int rowid = -1;
    if (rr < R) {
      const int mem = rr / NREP, rep = rr - mem * NREP;
      const int sq = min(max(a.view.grp_members[moff + mem], 0), a.num_seqs - 1);
      rowid = sq * a.num_q_heads + h * NREP + rep;
    }
    // The pass's query tile lives in this wave's LDS area (registers are the
    // scarce resource); each page reads it back as the B operand of S^T.
    wave_lds_sync();
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      uint4 w = make_uint4(0, 0, 0, 0);
      if (rowid >= 0) w = *reinterpret_cast<const uint4*>(qall + (size_t)rowid * D + kb * 32 + quad * 8);
      *reinterpret_cast<uint4*>(qt_lane + kb * 32) = w;
    }
    wave_lds_sync();

    float mrow = -INFINITY, lrow = 0.f;
    f32x4_t oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Pages are software-pipelined: the next page's V is requested once this
    // page's V is staged, its K once this page's scores exist (after this
    // wave's last page, its last page again: cache hits).
    PrefixPage<D, FP8> pg_regs;
    if (wave < npages) {
      const int pg0 = clamp_page(bt[wave], a.num_pages);
      load_prefix_k<D, FP8>(a, kpool, pg0, h, lane, pg_regs);
      load_prefix_v<D, FP8>(a, vpool, pg0, h, lane, pg_regs);
    }
    for (int p = wave; p < npages; p += kUnitWaves) {
      const int nv = min(kPage, ntok - p * kPage);
      const int pn = clamp_page(bt[p + kUnitWaves < npages ? p + kUnitWaves : p], a.num_pages);
      float sm = a.qk_scale, vm = 1.f;
      if constexpr (FP8) {
        sm *= pg_regs.ks;
        vm = pg_regs.vs;
      }

      wave_lds_sync();  // the previous page's LDS reads are complete
      stage_v<D, FP8, STRIDE>(pg_regs, nv, vt, lane);
      // Keep each refill after the last use of the registers it overwrites.
      __builtin_amdgcn_sched_barrier(0);
      load_prefix_v<D, FP8>(a, vpool, pn, h, lane, pg_regs);

      // Entry i of this lane is token quad*4+i of the page and query row r16 of the tile.
      f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8_t qop = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qt_lane + kb * 32));
        sacc = mfma16x16x32(prefix_k_operand<D, FP8>(pg_regs, kb), qop, sacc);
      }
      __builtin_amdgcn_sched_barrier(0);
      load_prefix_k<D, FP8>(a, kpool, pn, h, lane, pg_regs);
      float x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = quad * 4 + i < nv ? sacc[i] * sm : -INFINITY;
      float mloc = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
      mloc = xor_max_from<16>(mloc);
      const float mx = fmaxf(mrow, mloc);
      const float mu = mx == -INFINITY ? 0.f : mx;
      const float alpha = fast_exp2(mrow - mu);
      float pw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pw[i] = fast_exp2(x[i] - mu);
      lrow = lrow * alpha + ((pw[0] + pw[1]) + (pw[2] + pw[3]));
      mrow = mx;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
      // B operand of O^T = V^T P^T: k-slot quad*4+j is token quad*4+j of the
      // page, i.e. exactly this lane's four probabilities.
      const bf16x4_t pop = __builtin_bit_cast(
          bf16x4_t, make_uint2(pack_bf16x2(pw[0] * vm, pw[1] * vm), pack_bf16x2(pw[2] * vm, pw[3] * vm)));

      wave_lds_sync();  // the staged V is visible to the whole wave
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        // A operand: V^T[column dt*16 + r16][k-slot quad*4 + j] = V[token quad*4 + j][column].
        const uint16_t* col = vt + (quad * 4) * STRIDE + dt * 16 + r16;
        const uint32_t w0 = (uint32_t)col[0] | ((uint32_t)col[STRIDE] << 16);
        const uint32_t w1 = (uint32_t)col[2 * STRIDE] | ((uint32_t)col[3 * STRIDE] << 16);
        oacc[dt] = mfma16x16x16(__builtin_bit_cast(bf16x4_t, make_uint2(w0, w1)), pop, oacc[dt]);
        // One tile's operand in flight at a time: the reads are cheap, registers are not.
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // Merge the waves' states lane by lane (every wave holds the same tile
    // layout): waves 1.. publish theirs, wave 0 folds them in one output tile
    // at a time and writes the partial.
    constexpr int NF = 2 + DT * 4;
    const float* xs = reinterpret_cast<const float*>(smem) + lane * NF;
    if constexpr (kUnitWaves > 1) {
      float* e = reinterpret_cast<float*>(smem) + ((wave - 1) * 64 + lane) * NF;
      __syncthreads();  // every wave is done with its staged V
      if (wave > 0) {
        e[0] = mrow;
        e[1] = lrow;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int i = 0; i < 4; ++i) e[2 + dt * 4 + i] = oacc[dt][i];
      }
      __syncthreads();
    }
    if (wave == 0) {
      float mx = mrow;
#pragma unroll
      for (int w = 1; w < kUnitWaves; ++w) mx = fmaxf(mx, xs[(w - 1) * 64 * NF]);
      const float mu = mx == -INFINITY ? 0.f : mx;
      const float a0 = fast_exp2(mrow - mu);
      float aw[kUnitWaves];
      float lsum = lrow * a0;
#pragma unroll
      for (int w = 1; w < kUnitWaves; ++w) {
        aw[w] = fast_exp2(xs[(w - 1) * 64 * NF] - mu);
        lsum += xs[(w - 1) * 64 * NF + 1] * aw[w];
      }
      const float lt = xor_sum_from<16>(lsum);
      if (rowid >= 0) {
        const int part = clamp_part(rowid * a.view.parts_per_row + c, a.view.max_parts);
        const float inv = 1.f / lt;
        float* dst = a.view.part_o + (size_t)part * D + quad * 4;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          f32x4_t v = oacc[dt] * a0;
#pragma unroll
          for (int w = 1; w < kUnitWaves; ++w)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] += xs[(w - 1) * 64 * NF + 2 + dt * 4 + i] * aw[w];
          v *= inv;
          *reinterpret_cast<float4*>(dst + dt * 16) = make_float4(v[0], v[1], v[2], v[3]);
          __builtin_amdgcn_sched_barrier(0);
        }
        if (quad == 0) a.view.part_lse[part] = (mu + fast_log2(lt)) * kLn2;
      }
    }
    if constexpr (kUnitWaves > 1) __syncthreads();  // the next pass may stage V over the merge area
  }
}

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
// One response unit: kv-head h of response item `item`.
template <int D, int NREP, bool FP8>
__device__ void resp_unit(const AttnArgs& a, int item, int h, char* smem) {
  using G = RespGeom<D, FP8>;
  constexpr int EPL = G::EPL, LPT = G::LPT, TPL = G::TPL, LOADS = G::LOADS, QW = G::QW;
  const int Hkv = a.num_kv_heads;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tg = lane / LPT;
  const int sub = lane - tg * LPT;
  const char* kpool = static_cast<const char*>(a.k_pages);
  const char* vpool = static_cast<const char*>(a.v_pages);

  // The item record: sequence, first page index in its block table, tokens, slot.
  const int4 m = a.view.resp_items[item];
  const int s = min(max(m.x, 0), a.num_seqs - 1);
  const int p0 = min(max(m.y, 0), a.max_resp_pages);
  const int ntok = min(max(m.z, 0), min(kRespChunkPagesMax, a.max_resp_pages - p0) * kPage);
  const int slot = min(max(m.w, 0), a.view.parts_per_row - 1);
  const int npages = cdiv(ntok, kPage);
  const int* bt = a.resp_block_table + (size_t)s * a.max_resp_pages + p0;
  // This wave takes pages wave, wave + kUnitWaves, ...; a wave without pages
  // loads the item's first page once and skips the loop.
  int page = npages > 0 ? clamp_page(bt[wave < npages ? wave : 0], a.num_pages) : 0;
  uint4 kr[LOADS], vr[LOADS];
  {
    const size_t blk = resp_block<D, FP8>(a, page, h, lane);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) kr[i] = *reinterpret_cast<const uint4*>(kpool + blk + i * 1024);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) vr[i] = load_v_stream(vpool + blk + i * 1024);
  }

  // This lane's EPL head_dim elements of the NREP query rows of kv-head h (bf16).
  const uint16_t* qrow =
      reinterpret_cast<const uint16_t*>(a.q) + ((size_t)s * a.num_q_heads + (size_t)h * NREP) * D + sub * EPL;
  uint4 qb[NREP][QW];
#pragma unroll
  for (int r = 0; r < NREP; ++r)
#pragma unroll
    for (int w = 0; w < QW; ++w) qb[r][w] = *reinterpret_cast<const uint4*>(qrow + (size_t)r * D + w * 8);

  float mrun[NREP], l[NREP], o[NREP][EPL];
#pragma unroll
  for (int r = 0; r < NREP; ++r) {
    mrun[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[r][e] = 0.f;
  }

  // One page: scores from the K registers, which are then refilled with the
  // page `ahead` pages on (this page again past the unit's end: a cache hit),
  // V unpacked and refilled the same way, then the online softmax and P V.
  const auto step = [&](int p, int ahead, int& pg, uint4 (&kx)[LOADS], uint4 (&vx)[LOADS])
                        __attribute__((always_inline)) {
    const int next_page = p + ahead < npages ? clamp_page(bt[p + ahead], a.num_pages) : pg;
    const size_t next_blk = resp_block<D, FP8>(a, next_page, h, lane);
    const int nvalid = min(kPage, ntok - p * kPage);
    float smul = a.qk_scale, vmul = 1.f;
    if constexpr (FP8) {
      smul *= a.k_scale[(size_t)pg * Hkv + h];
      vmul = a.v_scale[(size_t)pg * Hkv + h];
    }

    float sc[LOADS][NREP];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if constexpr (!FP8) {
#pragma unroll
        for (int r = 0; r < NREP; ++r) sc[i][r] = group_sum<LPT>(dot8_bf16(qb[r][0], kx[i], 0.f)) * smul;
      } else {
        const uint4 k0 = e4m3x8_to_bf16x8(kx[i].x, kx[i].y);
        const uint4 k1 = e4m3x8_to_bf16x8(kx[i].z, kx[i].w);
#pragma unroll
        for (int r = 0; r < NREP; ++r)
          sc[i][r] = group_sum<LPT>(dot8_bf16(qb[r][1], k1, dot8_bf16(qb[r][0], k0, 0.f))) * smul;
      }
    }
#pragma unroll
    for (int i = 0; i < LOADS; ++i) kx[i] = *reinterpret_cast<const uint4*>(kpool + next_blk + i * 1024);

    float vf[LOADS][EPL];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if constexpr (!FP8) unpack_bf16x8(vx[i], vf[i]);
      else unpack_e4m3x16(vx[i], vf[i]);
    }
#pragma unroll
    for (int i = 0; i < LOADS; ++i) vx[i] = load_v_stream(vpool + next_blk + i * 1024);

    if (nvalid < kPage) {  // ragged last page: padding rows may hold anything
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const bool ok = i * TPL + tg < nvalid;
#pragma unroll
        for (int r = 0; r < NREP; ++r) sc[i][r] = ok ? sc[i][r] : -INFINITY;
#pragma unroll
        for (int e = 0; e < EPL; ++e) vf[i][e] = ok ? vf[i][e] : 0.f;
      }
    }

#pragma unroll
    for (int r = 0; r < NREP; ++r) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) mx = fmaxf(mx, sc[i][r]);
      // Lazy running maximum (kLazyMax): alpha is exactly 1 unless it moved,
      // and the rescale of the accumulator is skipped when no lane needs it.
      const float mnew = mx > mrun[r] + kLazyMax ? mx : mrun[r];
      const float mu = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = fast_exp2(mrun[r] - mu);
      float pw[LOADS], ps = 0.f;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        pw[i] = fast_exp2(sc[i][r] - mu);
        ps += pw[i];
      }
      l[r] = l[r] * alpha + ps;
      mrun[r] = mnew;
      if (__any(alpha != 1.f)) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[r][e] *= alpha;
      }
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const float pv = pw[i] * vmul;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[r][e] = fmaf(pv, vf[i][e], o[r][e]);
      }
    }
    pg = next_page;
  };

  if constexpr (!FP8 || kUnitWaves > 1) {
    // One page in flight per wave (bf16: 8 KiB of K and V at d = 128).
    for (int p = wave; p < npages; p += kUnitWaves) step(p, kUnitWaves, page, kr, vr);
  } else {
    // fp8 blocks are half the bytes: two pages in flight per wave (register
    // sets A and B alternate), for the same bytes in flight as bf16 at three
    // waves per SIMD instead of four.
    uint4 kb[LOADS], vb[LOADS];
    int page_b = npages > 1 ? clamp_page(bt[1], a.num_pages) : page;
    {
      const size_t blk = resp_block<D, FP8>(a, page_b, h, lane);
#pragma unroll
      for (int i = 0; i < LOADS; ++i) kb[i] = *reinterpret_cast<const uint4*>(kpool + blk + i * 1024);
#pragma unroll
      for (int i = 0; i < LOADS; ++i) vb[i] = load_v_stream(vpool + blk + i * 1024);
    }
    for (int p = 0; p < npages; p += 2) {
      step(p, 2, page, kr, vr);
      if (p + 1 < npages) step(p + 1, 2, page_b, kb, vb);
    }
  }

  // Merge the TPL lane groups' states of each wave, then the waves' states
  // (through LDS), and write one partial per query row.
  const int row0 = s * a.num_q_heads + h * NREP;
  float* xs = reinterpret_cast<float*>(smem);  // [kUnitWaves - 1][NREP][D + 2]
#pragma unroll
  for (int r = 0; r < NREP; ++r) {
    float M = xor_max_from<LPT>(mrun[r]);
    const float Mu = M == -INFINITY ? 0.f : M;
    const float w = fast_exp2(mrun[r] - Mu);
    float lt = xor_sum_from<LPT>(l[r] * w);
    float oo[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) oo[e] = xor_sum_from<LPT>(o[r][e] * w);
    if constexpr (kUnitWaves > 1) {
      float* e0 = xs + ((size_t)r * (kUnitWaves - 1) + (wave - 1)) * (D + 2);
      if (wave > 0 && tg == 0) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) e0[2 + sub * EPL + e] = oo[e];
        if (sub == 0) {
          e0[0] = M;
          e0[1] = lt;
        }
      }
      __syncthreads();
      if (wave == 0 && tg == 0) {
#pragma unroll
        for (int w2 = 1; w2 < kUnitWaves; ++w2) {
          const float* e1 = xs + ((size_t)r * (kUnitWaves - 1) + (w2 - 1)) * (D + 2);
          const float m1 = e1[0];
          const float mx = fmaxf(M, m1);
          const float mu = mx == -INFINITY ? 0.f : mx;
          const float a0 = fast_exp2(M - mu), a1 = fast_exp2(m1 - mu);
          lt = lt * a0 + e1[1] * a1;
#pragma unroll
          for (int e = 0; e < EPL; ++e) oo[e] = oo[e] * a0 + e1[2 + sub * EPL + e] * a1;
          M = mx;
        }
      }
    }
    if (wave == 0) {
      const int part = clamp_part((row0 + r) * a.view.parts_per_row + slot, a.view.max_parts);
      const float inv = 1.f / lt;
      if (tg == 0) {
        float4* dst = reinterpret_cast<float4*>(a.view.part_o + (size_t)part * D + sub * EPL);
#pragma unroll
        for (int e = 0; e < EPL; e += 4) dst[e / 4] = make_float4(oo[e] * inv, oo[e + 1] * inv, oo[e + 2] * inv, oo[e + 3] * inv);
      }
      if (lane == 0) a.view.part_lse[part] = (M + fast_log2(lt)) * kLn2;
    }
  }
}

// All partial results in one launch, one unit per workgroup: the first
// blocks take the group-prefix units (dispatched first; their short,
// latency-bound MFMA work overlaps the response units that fill the rest of
// the GPU), the following blocks the response units in plan order (big items
// first, then small ones by decreasing size), and blocks beyond the planned
// counts exit at once. Units are not interleaved by block id: workgroups are
// dealt round-robin to XCDs and then to shader engines, and any periodic
// pattern of unit kinds would correlate with that and unbalance them. The
// counts are clamped to the plan's capacity, so even a workspace that was
// never planned cannot send a wave outside the item lists.
template <int D, int NREP, bool FP8>
__global__ __launch_bounds__(kUnitThreads) void attn_parts_kernel(const AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[Smem<D, NREP>::kBytes];
  const int Hkv = a.num_kv_heads;
  const int n_pre = min(max(a.view.hdr[kHdrPrefixItems], 0), a.view.max_prefix_items) * Hkv;
  const int n_resp = min(max(a.view.hdr[kHdrRespItems], 0), a.view.max_resp_items) * Hkv;
  const int b = blockIdx.x;
  if (b < n_pre) {
    const int item = b / Hkv;
    prefix_unit<D, NREP, FP8>(a, item, b - item * Hkv, smem);
    return;
  }
  const int resp = b - n_pre;
  if (resp < n_resp) {
    const int item = resp / Hkv;
    resp_unit<D, NREP, FP8>(a, item, resp - item * Hkv, smem);
  }
}

// Grid: one block per unit of the largest plan that fits the workspace.
template <int D, int NREP, bool FP8>
hipError_t launch_one(const AttnArgs& a, long long prefix_blocks, long long resp_blocks, hipStream_t st) {
  const long long blocks = prefix_blocks + resp_blocks;
  attn_parts_kernel<D, NREP, FP8><<<dim3((unsigned)blocks), dim3(kUnitThreads), 0, st>>>(a);
  return hipGetLastError();
}

template <int D, bool FP8>
hipError_t by_nrep(const AttnArgs& a, int n_rep, long long pb, long long rb, hipStream_t st) {
  switch (n_rep) {
    case 1: return launch_one<D, 1, FP8>(a, pb, rb, st);
    case 2: return launch_one<D, 2, FP8>(a, pb, rb, st);
    case 4: return launch_one<D, 4, FP8>(a, pb, rb, st);
    case 8: return launch_one<D, 8, FP8>(a, pb, rb, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attn_parts(const AttnArgs& a, int head_dim, int n_rep, bool fp8, long long max_prefix_items,
                             long long max_resp_items, hipStream_t stream) {
  const long long pb = max_prefix_items * a.num_kv_heads, rb = max_resp_items * a.num_kv_heads;
  if (pb + rb <= 0) return hipSuccess;
  if (head_dim == 128) return fp8 ? by_nrep<128, true>(a, n_rep, pb, rb, stream) : by_nrep<128, false>(a, n_rep, pb, rb, stream);
  if (head_dim == 64) return fp8 ? by_nrep<64, true>(a, n_rep, pb, rb, stream) : by_nrep<64, false>(a, n_rep, pb, rb, stream);
  return hipErrorInvalidValue;
}

}  // namespace rp
