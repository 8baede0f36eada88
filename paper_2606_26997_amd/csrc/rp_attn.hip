// Partial attention over planned work items.
//
// Group-prefix items (MFMA): every response of a GRPO group is sampled from the
// same prompt, so the group's prompt-prefix KV is read once per (group, kv-head,
// chunk) and applied to all of the group's query rows at once: live members x
// (Hq / Hkv) query heads, as 16-row tiles on the bf16 MFMA
//   S^T = K Q^T   (M = 16 tokens, N = 16 query rows, K = head_dim)
//   O^T = V^T P^T (M = 16 head_dim columns, N = 16 query rows, K = 32 tokens)
// with fp32 accumulation and an online softmax over the chunk.
//
// Response items (VALU): each (sequence, kv-head, chunk of response pages) is
// one wave. A (page, kv-head) block is contiguous in the pool and is read with
// fully coalesced 16-byte loads: lane l holds EPL head_dim elements of token
// (load * TPL + l / LPT). Scores are reduced over the LPT lanes of a token with
// DPP, and every group of LPT lanes keeps its own online-softmax state over its
// tokens; the states are merged once at the end of the item.
//
// Each item writes one partial (o normalised, lse natural-log) per query row
// into the plan's CSR slot; the combine kernel merges the parts of a row.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

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
};

__device__ inline float dot8_bf16(const uint4& a, const uint4& b, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x), __builtin_bit_cast(bf16x2_t, b.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y), __builtin_bit_cast(bf16x2_t, b.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z), __builtin_bit_cast(bf16x2_t, b.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w), __builtin_bit_cast(bf16x2_t, b.w), acc, false);
  return acc;
}

__device__ inline void unpack_bf16x8(const uint4& w, float* f) {
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
  f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
  f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

// 16 e4m3 codes -> 16 floats scaled by 2^-8 (exact).
__device__ inline void unpack_e4m3x16(const uint4& w, float* f) {
  e4m3x2_to_f32_scaled(w.x, false, f[0], f[1]);
  e4m3x2_to_f32_scaled(w.x, true, f[2], f[3]);
  e4m3x2_to_f32_scaled(w.y, false, f[4], f[5]);
  e4m3x2_to_f32_scaled(w.y, true, f[6], f[7]);
  e4m3x2_to_f32_scaled(w.z, false, f[8], f[9]);
  e4m3x2_to_f32_scaled(w.z, true, f[10], f[11]);
  e4m3x2_to_f32_scaled(w.w, false, f[12], f[13]);
  e4m3x2_to_f32_scaled(w.w, true, f[14], f[15]);
}

template <int D, int NREP, bool FP8>
__global__ __launch_bounds__(64) void resp_parts_kernel(const AttnArgs a) {
  using G = RespGeom<D, FP8>;
  constexpr int EPL = G::EPL, LPT = G::LPT, TPL = G::TPL, LOADS = G::LOADS;
  const int Hkv = a.num_kv_heads;
  const int item = blockIdx.x / Hkv;
  const int h = blockIdx.x - item * Hkv;
  if (item >= a.view.hdr[kHdrRespItems]) return;

  const int2 it = a.view.resp_items[item];
  const int s = min(max(it.x, 0), a.num_seqs - 1);
  const int c = min(max(it.y, 0), a.view.max_resp_chunks - 1);
  const int L = clamp_len(a.resp_lens[s], a.max_resp_pages);
  const int g = clamp_group(a.seq_to_group[s], a.num_groups);
  const int npc = prefix_chunks(a.prefix_lens[g], a.max_prefix_pages, a.view.max_prefix_chunks);
  const int tok0 = c * (kRespChunkPages * kPage);
  const int ntok = min(kRespChunkPages * kPage, L - tok0);
  const int npages = cdiv(ntok, kPage);
  const int lane = threadIdx.x;
  const int tg = lane / LPT;
  const int sub = lane - tg * LPT;

  // This lane's EPL head_dim elements of the NREP query rows of kv-head h.
  const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                         ((size_t)s * a.num_q_heads + (size_t)h * NREP) * D + sub * EPL;
  uint4 qb[NREP];
  float qf[FP8 ? NREP : 1][FP8 ? EPL : 1];
#pragma unroll
  for (int r = 0; r < NREP; ++r) {
    if constexpr (!FP8) {
      qb[r] = *reinterpret_cast<const uint4*>(qrow + (size_t)r * D);
    } else {
      const uint4 lo = *reinterpret_cast<const uint4*>(qrow + (size_t)r * D);
      const uint4 hi = *reinterpret_cast<const uint4*>(qrow + (size_t)r * D + 8);
      unpack_bf16x8(lo, &qf[r][0]);
      unpack_bf16x8(hi, &qf[r][8]);
    }
  }

  float m[NREP], l[NREP], o[NREP][EPL];
#pragma unroll
  for (int r = 0; r < NREP; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[r][e] = 0.f;
  }

  const int* bt = a.resp_block_table + (size_t)s * a.max_resp_pages + c * kRespChunkPages;
  const char* kpool = static_cast<const char*>(a.k_pages);
  const char* vpool = static_cast<const char*>(a.v_pages);

  for (int p = 0; p < npages; ++p) {
    const int page = clamp_page(bt[p], a.num_pages);
    const size_t blk = ((size_t)page * Hkv + h) * G::BLOCK_BYTES + (size_t)lane * 16;
    uint4 kr[LOADS], vr[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) kr[i] = *reinterpret_cast<const uint4*>(kpool + blk + i * 1024);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) vr[i] = *reinterpret_cast<const uint4*>(vpool + blk + i * 1024);

    const int nvalid = min(kPage, ntok - p * kPage);
    float smul = a.qk_scale, vmul = 1.f;
    if constexpr (FP8) {
      smul *= a.k_scale[(size_t)page * Hkv + h] * kE4m3DecodeScale;
      vmul = a.v_scale[(size_t)page * Hkv + h] * kE4m3DecodeScale;
    }

    float sc[LOADS][NREP];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if constexpr (!FP8) {
#pragma unroll
        for (int r = 0; r < NREP; ++r) sc[i][r] = group_sum<LPT>(dot8_bf16(qb[r], kr[i], 0.f)) * smul;
      } else {
        float kf[EPL];
        unpack_e4m3x16(kr[i], kf);
#pragma unroll
        for (int r = 0; r < NREP; ++r) {
          float acc = 0.f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc = fmaf(qf[r][e], kf[e], acc);
          sc[i][r] = group_sum<LPT>(acc) * smul;
        }
      }
    }

    float vf[LOADS][EPL];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if constexpr (!FP8) unpack_bf16x8(vr[i], vf[i]);
      else unpack_e4m3x16(vr[i], vf[i]);
    }

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
      float mx = m[r];
#pragma unroll
      for (int i = 0; i < LOADS; ++i) mx = fmaxf(mx, sc[i][r]);
      const float mu = mx == -INFINITY ? 0.f : mx;
      const float alpha = fast_exp2(m[r] - mu);
      float pw[LOADS], ps = 0.f;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        pw[i] = fast_exp2(sc[i][r] - mu);
        ps += pw[i];
      }
      l[r] = l[r] * alpha + ps;
      m[r] = mx;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[r][e] *= alpha;
#pragma unroll
      for (int i = 0; i < LOADS; ++i) {
        const float pv = pw[i] * vmul;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[r][e] = fmaf(pv, vf[i][e], o[r][e]);
      }
    }
  }

  // Merge the TPL lane groups' states and write one partial per query row.
  const int row0 = s * a.num_q_heads + h * NREP;
#pragma unroll
  for (int r = 0; r < NREP; ++r) {
    const float M = xor_max_from<LPT>(m[r]);
    const float Mu = M == -INFINITY ? 0.f : M;
    const float w = fast_exp2(m[r] - Mu);
    const float lt = xor_sum_from<LPT>(l[r] * w);
    const float inv = 1.f / lt;
    float oo[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) oo[e] = xor_sum_from<LPT>(o[r][e] * w) * inv;
    const int part = clamp_part(a.view.row_offs[row0 + r] + npc + c, a.view.max_parts);
    if (tg == 0) {
      float4* dst = reinterpret_cast<float4*>(a.view.part_o + (size_t)part * D + sub * EPL);
#pragma unroll
      for (int e = 0; e < EPL; e += 4) dst[e / 4] = make_float4(oo[e], oo[e + 1], oo[e + 2], oo[e + 3]);
    }
    if (lane == 0) a.view.part_lse[part] = (M + fast_log2(lt)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// Group-prefix path (MFMA 16x16x32 bf16)
// ---------------------------------------------------------------------------
__device__ inline f32x4_t mfma16x16x32(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Two floats known to be exact in bf16 -> packed bf16 pair (truncation is exact).
__device__ inline uint32_t pack_exact_bf16x2(float lo, float hi) {
  return (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
}

// 8 e4m3 codes -> 8 bf16 values scaled by 2^-8 (exact).
__device__ inline uint4 e4m3x8_to_bf16x8(uint32_t w0, uint32_t w1) {
  float f[8];
  e4m3x2_to_f32_scaled(w0, false, f[0], f[1]);
  e4m3x2_to_f32_scaled(w0, true, f[2], f[3]);
  e4m3x2_to_f32_scaled(w1, false, f[4], f[5]);
  e4m3x2_to_f32_scaled(w1, true, f[6], f[7]);
  return make_uint4(pack_exact_bf16x2(f[0], f[1]), pack_exact_bf16x2(f[2], f[3]),
                    pack_exact_bf16x2(f[4], f[5]), pack_exact_bf16x2(f[6], f[7]));
}

// A operand of S^T = K Q^T for one page: lane (r16, quad) holds K[token r16][kb*32 + quad*8 + 0..7].
template <int D, bool FP8>
__device__ inline void load_k_operand(const char* pool, size_t blk_bytes, int r16, int quad, bf16x8_t* op) {
#pragma unroll
  for (int kb = 0; kb < D / 32; ++kb) {
    const int col = kb * 32 + quad * 8;
    if constexpr (!FP8) {
      const uint4 w = *reinterpret_cast<const uint4*>(pool + blk_bytes + ((size_t)r16 * D + col) * 2);
      op[kb] = __builtin_bit_cast(bf16x8_t, w);
    } else {
      const uint2 w = *reinterpret_cast<const uint2*>(pool + blk_bytes + (size_t)r16 * D + col);
      op[kb] = __builtin_bit_cast(bf16x8_t, e4m3x8_to_bf16x8(w.x, w.y));
    }
  }
}

// Copy one page's V block (bf16, or fp8 decoded to bf16 * 2^-8) into LDS rows
// [row0, row0 + 16); rows at or beyond `nvalid` are written as zeros.
template <int D, bool FP8, int STRIDE>
__device__ inline void stage_v(const char* pool, size_t blk_bytes, int nvalid, uint16_t* vt, int row0,
                               int lane) {
  if constexpr (!FP8) {
#pragma unroll
    for (int i = 0; i < kPage * D * 2 / 1024; ++i) {
      const int e0 = i * 512 + lane * 8;
      const int tok = e0 / D, col = e0 % D;
      uint4 w = make_uint4(0, 0, 0, 0);
      if (tok < nvalid) w = *reinterpret_cast<const uint4*>(pool + blk_bytes + (size_t)e0 * 2);
      uint2* dst = reinterpret_cast<uint2*>(vt + (row0 + tok) * STRIDE + col);
      dst[0] = make_uint2(w.x, w.y);
      dst[1] = make_uint2(w.z, w.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPage * D / 1024; ++i) {
      const int e0 = i * 1024 + lane * 16;
      const int tok = e0 / D, col = e0 % D;
      uint4 lo = make_uint4(0, 0, 0, 0), hi = make_uint4(0, 0, 0, 0);
      if (tok < nvalid) {
        const uint4 w = *reinterpret_cast<const uint4*>(pool + blk_bytes + e0);
        lo = e4m3x8_to_bf16x8(w.x, w.y);
        hi = e4m3x8_to_bf16x8(w.z, w.w);
      }
      uint2* dst = reinterpret_cast<uint2*>(vt + (row0 + tok) * STRIDE + col);
      dst[0] = make_uint2(lo.x, lo.y);
      dst[1] = make_uint2(lo.z, lo.w);
      dst[2] = make_uint2(hi.x, hi.y);
      dst[3] = make_uint2(hi.z, hi.w);
    }
  }
}

template <int D, int NREP, bool FP8>
__global__ __launch_bounds__(64) void prefix_parts_kernel(const AttnArgs a) {
  constexpr int KB = D / 32;       // MFMA k-blocks over head_dim
  constexpr int DT = D / 16;       // 16-column output tiles over head_dim
  constexpr int T = kPrefixTiles;  // 16-row query tiles per pass
  constexpr int STRIDE = D + 4;    // staged V row pitch (bf16 elements)
  constexpr int EB = FP8 ? 1 : 2;
  constexpr size_t BLOCK_BYTES = (size_t)kPage * D * EB;
  __shared__ __attribute__((aligned(16))) uint16_t vt[2 * kPage * STRIDE];

  const int Hkv = a.num_kv_heads;
  const int item = blockIdx.x / Hkv;
  const int h = blockIdx.x - item * Hkv;
  if (item >= a.view.hdr[kHdrPrefixItems]) return;

  const int2 it = a.view.prefix_items[item];
  const int g = clamp_group(it.x, a.num_groups);
  const int c = min(max(it.y, 0), a.view.max_prefix_chunks - 1);
  const int P = clamp_len(a.prefix_lens[g], a.max_prefix_pages);
  const int tok0 = c * (kPrefixChunkPages * kPage);
  const int ntok = min(kPrefixChunkPages * kPage, P - tok0);
  const int npages = cdiv(ntok, kPage);
  const int moff = a.view.grp_off[g];
  const int R = (a.view.grp_off[g + 1] - moff) * NREP;
  const int lane = threadIdx.x;
  const int r16 = lane & 15, quad = lane >> 4;
  const int* bt = a.prefix_block_table + (size_t)g * a.max_prefix_pages + c * kPrefixChunkPages;
  const char* kpool = static_cast<const char*>(a.k_pages);
  const char* vpool = static_cast<const char*>(a.v_pages);
  const uint16_t* qall = static_cast<const uint16_t*>(a.q);

  for (int r0 = 0; r0 < R; r0 += 16 * T) {
    const int ntiles = min(T, cdiv(R - r0, 16));
    bf16x8_t qop[T][KB];
    int rowid[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int rr = r0 + t * 16 + r16;
      rowid[t] = -1;
      if (t < ntiles && rr < R) {
        const int mem = rr / NREP, rep = rr - mem * NREP;
        const int sq = min(max(a.view.grp_members[moff + mem], 0), a.num_seqs - 1);
        rowid[t] = sq * a.num_q_heads + h * NREP + rep;
      }
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        uint4 w = make_uint4(0, 0, 0, 0);
        if (rowid[t] >= 0)
          w = *reinterpret_cast<const uint4*>(qall + (size_t)rowid[t] * D + kb * 32 + quad * 8);
        qop[t][kb] = __builtin_bit_cast(bf16x8_t, w);
      }
    }

    float mrow[T], lrow[T];
    f32x4_t oacc[T][DT];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      mrow[t] = -INFINITY;
      lrow[t] = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[t][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    for (int pb = 0; pb < npages; pb += 2) {
      const bool has_b = pb + 1 < npages;
      const int nva = min(kPage, ntok - pb * kPage);
      const int nvb = has_b ? min(kPage, ntok - (pb + 1) * kPage) : 0;
      const int pa = clamp_page(bt[pb], a.num_pages);
      const int pbp = has_b ? clamp_page(bt[pb + 1], a.num_pages) : pa;
      const size_t blk_a = ((size_t)pa * Hkv + h) * BLOCK_BYTES;
      const size_t blk_b = ((size_t)pbp * Hkv + h) * BLOCK_BYTES;

      bf16x8_t ka[KB], kbop[KB];
      load_k_operand<D, FP8>(kpool, blk_a, r16, quad, ka);
      load_k_operand<D, FP8>(kpool, blk_b, r16, quad, kbop);

      __syncthreads();  // the previous block's LDS reads are complete
      stage_v<D, FP8, STRIDE>(vpool, blk_a, nva, vt, 0, lane);
      stage_v<D, FP8, STRIDE>(vpool, blk_b, nvb, vt, kPage, lane);
      __syncthreads();

      float sa = a.qk_scale, sb = a.qk_scale, va = 1.f, vb = 1.f;
      if constexpr (FP8) {
        sa *= a.k_scale[(size_t)pa * Hkv + h] * kE4m3DecodeScale;
        sb *= a.k_scale[(size_t)pbp * Hkv + h] * kE4m3DecodeScale;
        va = a.v_scale[(size_t)pa * Hkv + h] * kE4m3DecodeScale;
        vb = a.v_scale[(size_t)pbp * Hkv + h] * kE4m3DecodeScale;
      }

      bf16x8_t pop[T];
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (t >= ntiles) continue;
        f32x4_t s_a = {0.f, 0.f, 0.f, 0.f}, s_b = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          s_a = mfma16x16x32(ka[kb], qop[t][kb], s_a);
          s_b = mfma16x16x32(kbop[kb], qop[t][kb], s_b);
        }
        // Entry i of this lane is token quad*4+i of the page, query row r16 of the tile.
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          x[i] = quad * 4 + i < nva ? s_a[i] * sa : -INFINITY;
          x[4 + i] = quad * 4 + i < nvb ? s_b[i] * sb : -INFINITY;
        }
        float mloc = x[0];
#pragma unroll
        for (int k = 1; k < 8; ++k) mloc = fmaxf(mloc, x[k]);
        mloc = xor_max_from<16>(mloc);
        const float mx = fmaxf(mrow[t], mloc);
        const float mu = mx == -INFINITY ? 0.f : mx;
        const float alpha = fast_exp2(mrow[t] - mu);
        float pw[8], ps = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          pw[k] = fast_exp2(x[k] - mu);
          ps += pw[k];
        }
        lrow[t] = lrow[t] * alpha + ps;
        mrow[t] = mx;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[t][dt] *= alpha;
        // B operand of O^T = V^T P^T: k-slot quad*8+j is token quad*4+j of page a
        // (j < 4) or of page b (j >= 4): exactly this lane's eight probabilities.
        const uint4 pk = make_uint4(pack_bf16x2(pw[0] * va, pw[1] * va), pack_bf16x2(pw[2] * va, pw[3] * va),
                                    pack_bf16x2(pw[4] * vb, pw[5] * vb), pack_bf16x2(pw[6] * vb, pw[7] * vb));
        pop[t] = __builtin_bit_cast(bf16x8_t, pk);
      }

#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        // A operand: V^T[column dt*16 + r16][k-slot quad*8 + j], same token order as the B operand.
        const uint16_t* col = vt + dt * 16 + r16;
        const int ta = quad * 4, tb = kPage + quad * 4;
        uint32_t w[4];
        w[0] = (uint32_t)col[(ta + 0) * STRIDE] | ((uint32_t)col[(ta + 1) * STRIDE] << 16);
        w[1] = (uint32_t)col[(ta + 2) * STRIDE] | ((uint32_t)col[(ta + 3) * STRIDE] << 16);
        w[2] = (uint32_t)col[(tb + 0) * STRIDE] | ((uint32_t)col[(tb + 1) * STRIDE] << 16);
        w[3] = (uint32_t)col[(tb + 2) * STRIDE] | ((uint32_t)col[(tb + 3) * STRIDE] << 16);
        const bf16x8_t vop = __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
#pragma unroll
        for (int t = 0; t < T; ++t)
          if (t < ntiles) oacc[t][dt] = mfma16x16x32(vop, pop[t], oacc[t][dt]);
      }
    }

#pragma unroll
    for (int t = 0; t < T; ++t) {
      if (t >= ntiles) continue;
      const float lt = xor_sum_from<16>(lrow[t]);
      if (rowid[t] < 0) continue;
      const int part = clamp_part(a.view.row_offs[rowid[t]] + c, a.view.max_parts);
      const float inv = 1.f / lt;
      float* dst = a.view.part_o + (size_t)part * D + quad * 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const f32x4_t v = oacc[t][dt] * inv;
        *reinterpret_cast<float4*>(dst + dt * 16) = make_float4(v[0], v[1], v[2], v[3]);
      }
      if (quad == 0) a.view.part_lse[part] = (mrow[t] + fast_log2(lt)) * kLn2;
    }
  }
}

template <int D, int NREP, bool FP8>
hipError_t launch_one_resp(const AttnArgs& a, long long blocks, hipStream_t st) {
  resp_parts_kernel<D, NREP, FP8><<<dim3((unsigned)blocks), dim3(64), 0, st>>>(a);
  return hipGetLastError();
}
template <int D, int NREP, bool FP8>
hipError_t launch_one_prefix(const AttnArgs& a, long long blocks, hipStream_t st) {
  prefix_parts_kernel<D, NREP, FP8><<<dim3((unsigned)blocks), dim3(64), 0, st>>>(a);
  return hipGetLastError();
}

template <bool PREFIX, int D, bool FP8>
hipError_t by_nrep(const AttnArgs& a, int n_rep, long long blocks, hipStream_t st) {
  switch (n_rep) {
    case 1: return PREFIX ? launch_one_prefix<D, 1, FP8>(a, blocks, st) : launch_one_resp<D, 1, FP8>(a, blocks, st);
    case 2: return PREFIX ? launch_one_prefix<D, 2, FP8>(a, blocks, st) : launch_one_resp<D, 2, FP8>(a, blocks, st);
    case 4: return PREFIX ? launch_one_prefix<D, 4, FP8>(a, blocks, st) : launch_one_resp<D, 4, FP8>(a, blocks, st);
    case 8: return PREFIX ? launch_one_prefix<D, 8, FP8>(a, blocks, st) : launch_one_resp<D, 8, FP8>(a, blocks, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool PREFIX>
hipError_t dispatch(const AttnArgs& a, int head_dim, int n_rep, bool fp8, long long blocks, hipStream_t st) {
  if (blocks <= 0) return hipSuccess;
  if (head_dim == 128) return fp8 ? by_nrep<PREFIX, 128, true>(a, n_rep, blocks, st) : by_nrep<PREFIX, 128, false>(a, n_rep, blocks, st);
  if (head_dim == 64) return fp8 ? by_nrep<PREFIX, 64, true>(a, n_rep, blocks, st) : by_nrep<PREFIX, 64, false>(a, n_rep, blocks, st);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_prefix_parts(const AttnArgs& a, int head_dim, int n_rep, bool fp8, long long max_items,
                               hipStream_t stream) {
  return dispatch<true>(a, head_dim, n_rep, fp8, max_items * a.num_kv_heads, stream);
}

hipError_t launch_resp_parts(const AttnArgs& a, int head_dim, int n_rep, bool fp8, long long max_items,
                             hipStream_t stream) {
  return dispatch<false>(a, head_dim, n_rep, fp8, max_items * a.num_kv_heads, stream);
}

}  // namespace rp
