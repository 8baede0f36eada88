// Shared-prefix prefill. Every response of a GRPO group is sampled from the
// same prompt, so the prompt is processed once per group: its K/V are written
// into the group's prefix pages (the pages every response then reads while
// decoding) and its tokens attend causally within the prompt.
//
// K/V write: one wave per (group, prefix page, kv-head). bf16 pools copy the
// rows; fp8 pools get, in plain IEEE fp32, scale = amax / 448 over the page's
// written rows (1 when amax = 0) and codes e4m3(x / scale), round to nearest
// even, saturating.
//
// Causal attention: a workgroup of 4 waves per (group, kv-head, block of
// query rows); a 16-row tile holds 16 / n_rep consecutive prompt tokens times
// the n_rep query heads that share the kv-head, so every key block serves all
// of them (details at the kernel). K/V are read from the projections (not
// from the pool), as the prompt's own attention needs no quantised copy.
//
// Grid: workgroup b takes (group, kv-head) pair b % NP and row block
// max_blocks - 1 - b / NP (the last rows, which see the most keys, first).
// Workgroups are dealt to the 8 XCDs round-robin, so with NP a multiple of 8
// every row block of a pair runs on one XCD and re-reads the pair's K/V from
// that XCD's L2.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

// Length and first packed row of group g's prompt, clamped to the table width
// and to the packed arrays.
__device__ inline int prompt_len(const PrefillArgs& a, int g, int* first) {
  const int o0 = min(max(a.prompt_offs[g], 0), a.num_tokens);
  const int o1 = min(max(a.prompt_offs[g + 1], o0), a.num_tokens);
  *first = o0;
  return min(o1 - o0, a.max_prefix_pages * kPage);
}

// ---------------------------------------------------------------------------
// K/V page write
// ---------------------------------------------------------------------------
template <int D>
__device__ void write_fp8_head(uint8_t* blk, float* scale_slot, const uint16_t* src, size_t src_row_pitch,
                               int rows, int lane) {
#pragma clang fp contract(off)
  constexpr int CPR = D / 8;  // 8-element chunks per row
  float amax = 0.f;
  for (int c = lane; c < rows * CPR; c += 64) {
    const int r = c / CPR, col = (c - r * CPR) * 8;
    const uint4 w = *reinterpret_cast<const uint4*>(src + (size_t)r * src_row_pitch + col);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) amax = fmaxf(amax, fmaxf(fabsf(bf16_lo(ws[e])), fabsf(bf16_hi(ws[e]))));
  }
  amax = xor_max_from<1>(amax);
  const float scale = amax > 0.f ? amax / 448.0f : 1.0f;
  for (int c = lane; c < rows * CPR; c += 64) {
    const int r = c / CPR, col = (c - r * CPR) * 8;
    const uint4 w = *reinterpret_cast<const uint4*>(src + (size_t)r * src_row_pitch + col);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
    uint32_t codes[2] = {0, 0};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = f32_to_e4m3(bf16_lo(ws[e]) / scale), hi = f32_to_e4m3(bf16_hi(ws[e]) / scale);
      codes[e / 2] |= (lo | (hi << 8)) << (16 * (e % 2));
    }
    *reinterpret_cast<uint2*>(blk + (size_t)r * D + col) = make_uint2(codes[0], codes[1]);
  }
  if (lane == 0) *scale_slot = scale;
}

template <int D, bool FP8>
__global__ __launch_bounds__(64) void prefill_kv_write_kernel(const PrefillArgs a) {
  const int Hkv = a.num_kv_heads;
  const int b = blockIdx.x;
  const int h = b % Hkv;
  const int p = (b / Hkv) % a.max_prefix_pages;
  const int g = b / (Hkv * a.max_prefix_pages);
  int first;
  const int P = prompt_len(a, g, &first);
  const int rows = min(kPage, P - p * kPage);
  if (rows <= 0) return;
  const int page = clamp_page(a.prefix_block_table[(size_t)g * a.max_prefix_pages + p], a.num_pages);
  const int lane = threadIdx.x;
  const size_t pitch = (size_t)Hkv * D;  // elements between consecutive tokens of the projections
  const size_t src0 = (size_t)(first + p * kPage) * pitch + (size_t)h * D;
  const uint16_t* ks = static_cast<const uint16_t*>(a.k) + src0;
  const uint16_t* vs = static_cast<const uint16_t*>(a.v) + src0;
  const size_t blk = ((size_t)page * Hkv + h) * kPage * D;  // in elements
  if constexpr (!FP8) {
    constexpr int CPR = D / 8;
    uint16_t* kd = static_cast<uint16_t*>(a.k_pages) + blk;
    uint16_t* vd = static_cast<uint16_t*>(a.v_pages) + blk;
    for (int c = lane; c < rows * CPR; c += 64) {
      const int r = c / CPR, col = (c - r * CPR) * 8;
      *reinterpret_cast<uint4*>(kd + (size_t)r * D + col) = *reinterpret_cast<const uint4*>(ks + r * pitch + col);
      *reinterpret_cast<uint4*>(vd + (size_t)r * D + col) = *reinterpret_cast<const uint4*>(vs + r * pitch + col);
    }
  } else {
    const size_t sidx = (size_t)page * Hkv + h;
    write_fp8_head<D>(static_cast<uint8_t*>(a.k_pages) + blk, a.k_scale + sidx, ks, pitch, rows, lane);
    write_fp8_head<D>(static_cast<uint8_t*>(a.v_pages) + blk, a.v_scale + sidx, vs, pitch, rows, lane);
  }
}

// ---------------------------------------------------------------------------
// Causal attention
// ---------------------------------------------------------------------------
// Workgroup of 4 waves on (group, kv-head) pair and a block of query rows:
// wave w holds RT 16-row tiles (each 16 / n_rep consecutive prompt tokens
// times the n_rep query heads of the kv-head), so a workgroup covers
// 64 RT / n_rep tokens. Keys go through LDS in blocks of 32, double-buffered:
// while the waves compute on one block, the next block's K and V (both
// row-major, as in the projections) are loaded from the projections and
// written into the other buffer; one barrier per
// block. Per block and row tile: S^T = K Q^T on mfma 16x16x32 (Q stays in
// registers), a causal mask, one online-softmax update per row, and
// O^T += V^T P^T, also on mfma 16x16x32 (all 32 keys per instruction).
constexpr int kPfWaves = 4;
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kKeyBlk = 32;

// Both K and V are staged row-major, as they come from the projections. The
// V^T operand of P V is read with gfx950's transposing LDS read (lds_read_tr:
// four rows of one column per lane).
template <int D>
struct PfSmem {
  static constexpr int kKPitch = D + 16;  // K rows, bf16: the 16-byte reads of 16 rows hit no bank twice
  static constexpr int kVPitch = D + 16;  // V rows, bf16: 4 consecutive rows start 8 banks apart
  static constexpr int kKElems = kKeyBlk * kKPitch;
  static constexpr int kStage = kKElems + kKeyBlk * kVPitch;
  static constexpr int kBytes = 2 * kStage * 2;
  static constexpr int kChunks = kKeyBlk * D / 8;  // 16-byte pieces of a K (or V) block
  static constexpr int kPerThread = kChunks / kPfThreads;
  static_assert(kChunks % kPfThreads == 0, "block split");
  static_assert(kPerThread == 1 || kPerThread == 2, "pieces per thread");
};

// This thread's share of one key block, in registers between the global
// loads and the LDS writes. Clang vector types, not HIP's uint4: copies of
// the latter go through memcpy and kept these values in scratch memory. Rows
// at or past the prompt's end are read from its last token (inside the packed
// arrays); their scores are masked.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
struct PfBlock {
  u32x4_t k0, k1, v0, v1;
};

// Byte offsets within one prompt's rows fit 32 bits (the host checks it), so
// the loads take the group's wave-uniform base plus a 32-bit offset: no
// 64-bit address arithmetic per block.
template <int D>
__device__ inline void pf_load(const uint16_t* kbase, const uint16_t* vbase, uint32_t pitch, int u0, int last, int t,
                               PfBlock& r) {
  using L = PfSmem<D>;
  const char* kb = reinterpret_cast<const char*>(kbase);
  const char* vb = reinterpret_cast<const char*>(vbase);
  {
    const int key = t / (D / 8), col = (t - key * (D / 8)) * 8;
    const uint32_t off = ((uint32_t)min(u0 + key, last) * pitch + (uint32_t)col) * 2u;
    r.k0 = *reinterpret_cast<const u32x4_t*>(kb + off);
    r.v0 = *reinterpret_cast<const u32x4_t*>(vb + off);
  }
  if constexpr (L::kPerThread == 2) {
    const int c = t + kPfThreads;
    const int key = c / (D / 8), col = (c - key * (D / 8)) * 8;
    const uint32_t off = ((uint32_t)min(u0 + key, last) * pitch + (uint32_t)col) * 2u;
    r.k1 = *reinterpret_cast<const u32x4_t*>(kb + off);
    r.v1 = *reinterpret_cast<const u32x4_t*>(vb + off);
  }
}

template <int D>
__device__ inline void pf_store(uint16_t* stage, int t, const PfBlock& r) {
  using L = PfSmem<D>;
  uint16_t* vst = stage + L::kKElems;
  {
    const int key = t / (D / 8), col = (t - key * (D / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(stage + key * L::kKPitch + col) = r.k0;
    *reinterpret_cast<u32x4_t*>(vst + key * L::kVPitch + col) = r.v0;
  }
  if constexpr (L::kPerThread == 2) {
    const int c = t + kPfThreads;
    const int key = c / (D / 8), col = (c - key * (D / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(stage + key * L::kKPitch + col) = r.k1;
    *reinterpret_cast<u32x4_t*>(vst + key * L::kVPitch + col) = r.v1;
  }
}

// The one-launch prefill of a bf16 pool writes every prompt token's K/V rows
// into the group's prefix pages from the workgroup whose query rows hold the
// token (exactly one), in one of two ways; rows past the prompt's end are not
// written, as in the page-write kernel.
//
// With one row tile per wave, the workgroup writes a key block's staged
// registers (after they went to LDS) when the block starts with one of its
// tokens. With two row tiles, the page addresses held across the key loop
// would cost the kernel its third wave per SIMD (178 VGPRs), so the workgroup
// copies its own rows in the prologue instead: the copy's loads are issued
// together with the q rows and the first key block, and its stores follow
// them (1024-token prompts 296 -> 280 us; with one row tile the prologue
// copy was 5% slower on config-2 prompts, U[64, 512] tokens).
template <int D, int TPB>
struct PfOwnRows {
  static constexpr int kCh = TPB * (D / 8);  // 16-byte pieces of the workgroup's rows (K or V)
  static constexpr int kPer = (kCh + kPfThreads - 1) / kPfThreads;
  u32x4_t k[kPer], v[kPer];

  __device__ inline void load(int T0, int last, int t, const uint16_t* kbase, const uint16_t* vbase, uint32_t pitch) {
    const char* kb = reinterpret_cast<const char*>(kbase);
    const char* vb = reinterpret_cast<const char*>(vbase);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = t + i * kPfThreads, tok = c / (D / 8), col = (c - tok * (D / 8)) * 8, u = T0 + tok;
      if (c < kCh && u <= last) {
        const uint32_t off = ((uint32_t)u * pitch + (uint32_t)col) * 2u;
        k[i] = *reinterpret_cast<const u32x4_t*>(kb + off);
        v[i] = *reinterpret_cast<const u32x4_t*>(vb + off);
      }
    }
  }

  __device__ inline void store(const PrefillArgs& a, int g, int h, int T0, int last, int t) const {
    const int* pbt = a.prefix_block_table + (size_t)g * a.max_prefix_pages;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = t + i * kPfThreads, tok = c / (D / 8), col = (c - tok * (D / 8)) * 8, u = T0 + tok;
      if (c < kCh && u <= last) {
        const int page = clamp_page(pbt[u / kPage], a.num_pages);
        const size_t off = (((size_t)page * a.num_kv_heads + h) * kPage + (u % kPage)) * D + col;
        *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(a.k_pages) + off) = k[i];
        *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(a.v_pages) + off) = v[i];
      }
    }
  }
};

template <int D>
__device__ inline void pf_write_pages(const PrefillArgs& a, int g, int h, int u0, int last, int t,
                                      const PfBlock& r) {
  using L = PfSmem<D>;
  const int* pbt = a.prefix_block_table + (size_t)g * a.max_prefix_pages;
  uint16_t* kp = static_cast<uint16_t*>(a.k_pages);
  uint16_t* vp = static_cast<uint16_t*>(a.v_pages);
  const auto put = [&](int c, const u32x4_t& kk, const u32x4_t& vv) __attribute__((always_inline)) {
    const int key = c / (D / 8), col = (c - key * (D / 8)) * 8, u = u0 + key;
    if (u > last) return;
    const int page = clamp_page(pbt[u / kPage], a.num_pages);
    const size_t off = (((size_t)page * a.num_kv_heads + h) * kPage + (u % kPage)) * D + col;
    *reinterpret_cast<u32x4_t*>(kp + off) = kk;
    *reinterpret_cast<u32x4_t*>(vp + off) = vv;
  };
  put(t, r.k0, r.v0);
  if constexpr (L::kPerThread == 2) put(t + kPfThreads, r.k1, r.v1);
}


// One 32-key block from LDS stage `kst` (keys u0 .. u0 + 31) for this wave's
// RT row tiles: the scores of both 16-key sub-tiles, the causal mask, one
// online-softmax update per row for the whole block, then O^T += V^T P^T.
// A row's running maximum moves only when a block exceeds it by more than
// kLazyMax; the accumulator is rescaled only when some row's maximum moved
// (alpha is exactly 1 otherwise), a test uniform over the wave. MASK = false for
// blocks that lie wholly at or below the diagonal of every row of the wave.
template <int D, int NREP, int RT, bool MASK>
__device__ __forceinline__ void pf_compute(const uint16_t* kst, int u0, int last, float qk_scale, int r16, int quad,
                                           const int (&tr)[RT], const bf16x8_t (&qop)[RT][D / 32],
                                           f32x4_t (&oacc)[RT][D / 16], float (&mrow)[RT], float (&lrow)[RT]) {
  using L = PfSmem<D>;
  constexpr int KB = D / 32, DT = D / 16, ST = kKeyBlk / 16;
  const uint16_t* vst = kst + L::kKElems;
  // Entry i of sub-tile st: key u0 + st*16 + quad*4 + i against row r16.
  f32x4_t sacc[RT][ST];
  // The waves of a SIMD come from different workgroups and drift in and out
  // of phase; raising the priority of a wave while it issues its MFMAs lets
  // another wave's softmax fill the matrix core's shadow instead of
  // competing for issue slots (config-2 prompts 58.3 -> 54.2 us; prompts
  // of 512-2048 tokens, with two row tiles per wave, unchanged).
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int st = 0; st < ST; ++st) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) sacc[rt][st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const bf16x8_t kop = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const uint4*>(kst + (st * 16 + r16) * L::kKPitch + kb * 32 + quad * 8));
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) sacc[rt][st] = mfma16x16x32(kop, qop[rt][kb], sacc[rt][st]);
    }
  }
  __builtin_amdgcn_s_setprio(0);
  // V^T operands are read inside P V, one 16-column tile at a time: fewer
  // live registers than reading the whole block's ahead of the softmax,
  // which keeps four waves per SIMD with one row tile and three with two.
  const uint16_t* vtr = vst + (quad * 4 + r16 / 4) * L::kVPitch + 4 * (r16 % 4);
  const auto read_vop = [&](int dt) __attribute__((always_inline)) {
    const bf16x4_t v0 = lds_read_tr(vtr + dt * 16);
    const bf16x4_t v1 = lds_read_tr(vtr + 16 * L::kVPitch + dt * 16);
    return __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  bf16x4_t pop[RT][ST];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    // Raw scores (masked to -inf); the scale is applied inside the exponent,
    // max(s * c) = max(s) * c for c > 0.
    float x[ST][4];
    float mloc = -INFINITY;
#pragma unroll
    for (int st = 0; st < ST; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (MASK) {
          const int u = u0 + st * 16 + quad * 4 + i;
          x[st][i] = (tr[rt] <= last && u <= tr[rt]) ? sacc[rt][st][i] : -INFINITY;
        } else {
          x[st][i] = sacc[rt][st][i];
        }
        mloc = fmaxf(mloc, x[st][i]);
      }
    mloc = max_xor16_32(mloc) * qk_scale;
    // The running maximum moves only when this block exceeds it by more than
    // kLazyMax (log2 units): the probabilities then stay below 2^kLazyMax,
    // and most blocks leave the accumulator unscaled (alpha = exp2(0) = 1).
    const float mnew = mloc > mrow[rt] + kLazyMax ? mloc : mrow[rt];
    const float mu = mnew == -INFINITY ? 0.f : mnew;
    const float alpha = fast_exp2(mrow[rt] - mu);
    mrow[rt] = mnew;
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < ST; ++st) {
      float pw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pw[i] = fast_exp2(fmaf(x[st][i], qk_scale, -mu));
      psum += (pw[0] + pw[1]) + (pw[2] + pw[3]);
      pop[rt][st] =
          __builtin_bit_cast(bf16x4_t, make_uint2(pack_bf16x2(pw[0], pw[1]), pack_bf16x2(pw[2], pw[3])));
    }
    lrow[rt] = lrow[rt] * alpha + psum;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[rt][dt] *= alpha;
    }
  }
  // O^T += V^T P^T over all 32 keys in one mfma 16x16x32 per 16 output
  // columns: lane (r16, quad) supplies contraction slots 8 quad .. 8 quad + 7,
  // taken as keys quad*4 .. quad*4 + 3 and 16 + quad*4 .. 16 + quad*4 + 3 in
  // both operands (any key order serves, as long as V^T and P^T share it).
  // The V^T operand of lane (r16, quad) is column dt*16 + r16 of those keys:
  // two transposing reads, in which lane s of the quad's 16 points at row
  // quad*4 + s/4 (then 16 rows further on), columns dt*16 + 4 (s % 4) ...+3.
  static_assert(ST == 2, "two 16-key sub-tiles per block");
  bf16x8_t pop8[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
    pop8[rt] = __builtin_shufflevector(pop[rt][0], pop[rt][1], 0, 1, 2, 3, 4, 5, 6, 7);
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const bf16x8_t vo = read_vop(dt);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) oacc[rt][dt] = mfma16x16x32(vo, pop8[rt], oacc[rt][dt]);
  }
  __builtin_amdgcn_s_setprio(0);
}

// Register budget: one row tile per wave fits four waves per SIMD (128
// VGPRs), two row tiles three (168 VGPRs).
template <int D, int NREP, int RT, bool WP>
__global__ __launch_bounds__(kPfThreads) __attribute__((amdgpu_waves_per_eu(RT == 1 ? 4 : 3, 8)))
void prefill_attn_kernel(const PrefillArgs a, int max_blocks) {
  using L = PfSmem<D>;
  constexpr int KB = D / 32;              // MFMA k-blocks over head_dim
  constexpr int DT = D / 16;              // 16-column output tiles
  constexpr int TPT = 16 / NREP;          // prompt tokens per 16-row tile
  constexpr int TPW = RT * TPT;           // prompt tokens per wave
  constexpr int TPB = kPfWaves * TPW;     // prompt tokens per workgroup
  __shared__ __attribute__((aligned(16))) uint16_t smem[L::kBytes / 2];

  const int Hkv = a.num_kv_heads, Hq = a.num_q_heads;
  const int NP = a.num_groups * Hkv;
  const int pair = (int)(blockIdx.x % (unsigned)NP);
  const int rb = max_blocks - 1 - (int)(blockIdx.x / (unsigned)NP);
  const int g = pair / Hkv, h = pair - g * Hkv;
  int first;
  const int P = prompt_len(a, g, &first);
  const int T0 = rb * TPB;
  if (T0 >= P) return;  // uniform over the workgroup
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, r16 = lane & 15, quad = lane >> 4;
  const int last = P - 1;
  const size_t qpitch = (size_t)Hq * D, kpitch = (size_t)Hkv * D;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (size_t)first * kpitch + (size_t)h * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (size_t)first * kpitch + (size_t)h * D;

  constexpr bool kOwnCopy = WP && RT == 2, kBlockWrite = WP && RT == 1;
  PfOwnRows<D, TPB> own;
  if constexpr (kOwnCopy) own.load(T0, last, t, kbase, vbase, (uint32_t)kpitch);

  // Row r16 of row tile rt: token T0 + wave * TPW + rt * TPT + r16 / NREP,
  // query head h * NREP + r16 % NREP. Q is the B operand of S^T = K Q^T.
  const int jr = h * NREP + r16 % NREP;
  int tr[RT];
  bf16x8_t qop[RT][KB];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    tr[rt] = T0 + wave * TPW + rt * TPT + r16 / NREP;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + (size_t)(first + min(tr[rt], last)) * qpitch +
                           (size_t)jr * D + quad * 8;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      qop[rt][kb] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + kb * 32));
  }

  const int tlast = min(T0 + TPB, P) - 1;  // the workgroup's last token bounds its keys
  const int w_first = T0 + wave * TPW, w_last = w_first + TPW - 1;  // this wave's tokens
  const int nblk = tlast / kKeyBlk + 1;
  float mrow[RT], lrow[RT];
  f32x4_t oacc[RT][DT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    mrow[rt] = -INFINITY;
    lrow[rt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[rt][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // The next block's loads are issued before this block's compute and
  // written to the other LDS buffer after it (past the last block they read
  // clamped rows and are never used).
  PfBlock nx;
  pf_load<D>(kbase, vbase, (uint32_t)kpitch, 0, last, t, nx);
  if constexpr (kOwnCopy) own.store(a, g, h, T0, last, t);
  pf_store<D>(smem, t, nx);
  if (kBlockWrite && T0 == 0) pf_write_pages<D>(a, g, h, 0, last, t, nx);
  __syncthreads();
  for (int blk = 0; blk < nblk; ++blk) {
    pf_load<D>(kbase, vbase, (uint32_t)kpitch, (blk + 1) * kKeyBlk, last, t, nx);
    // Blocks wholly below the diagonal for every (valid) row of the wave skip the mask.
    if ((blk + 1) * kKeyBlk - 1 <= w_first && w_last <= last)
      pf_compute<D, NREP, RT, false>(smem + (blk & 1) * L::kStage, blk * kKeyBlk, last, a.qk_scale, r16, quad, tr,
                                     qop, oacc, mrow, lrow);
    else
      pf_compute<D, NREP, RT, true>(smem + (blk & 1) * L::kStage, blk * kKeyBlk, last, a.qk_scale, r16, quad, tr,
                                    qop, oacc, mrow, lrow);
    pf_store<D>(smem + ((blk + 1) & 1) * L::kStage, t, nx);
    const int un = (blk + 1) * kKeyBlk;
    if (kBlockWrite && un >= T0 && un < T0 + TPB) pf_write_pages<D>(a, g, h, un, last, t, nx);
    __syncthreads();  // the next block is staged; this block's buffer may be overwritten next
  }

#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const float lt = xor_sum_from<16>(lrow[rt]);
    if (tr[rt] > last) continue;
    const float inv = 1.f / lt;
    uint16_t* orow = static_cast<uint16_t*>(a.out) + (size_t)(first + tr[rt]) * qpitch + (size_t)jr * D + quad * 4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const f32x4_t v = oacc[rt][dt] * inv;
      *reinterpret_cast<uint2*>(orow + dt * 16) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
    }
    if (a.lse != nullptr && quad == 0) a.lse[(size_t)(first + tr[rt]) * Hq + jr] = (mrow[rt] + fast_log2(lt)) * kLn2;
  }
}

// Row tiles per wave: two when prompts average 384 tokens or more (each K/V
// operand read from LDS serves two MFMAs), one otherwise (twice the
// workgroups, which balances ragged short prompts better; measured).
template <int D, int NREP>
hipError_t attn_launch(const PrefillArgs& a, hipStream_t st) {
  const long long NP = (long long)a.num_groups * a.num_kv_heads;
  const int max_tokens = a.max_prefix_pages * kPage;
  const int rt = (long long)a.num_tokens >= 384ll * a.num_groups ? 2 : 1;
  const int tpb = kPfWaves * rt * (16 / NREP);
  const int max_blocks = cdiv(max_tokens, tpb);
  const long long blocks = NP * max_blocks;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(kPfThreads);
  if (a.write_pages) {
    if (rt == 2) prefill_attn_kernel<D, NREP, 2, true><<<grid, block, 0, st>>>(a, max_blocks);
    else prefill_attn_kernel<D, NREP, 1, true><<<grid, block, 0, st>>>(a, max_blocks);
  } else {
    if (rt == 2) prefill_attn_kernel<D, NREP, 2, false><<<grid, block, 0, st>>>(a, max_blocks);
    else prefill_attn_kernel<D, NREP, 1, false><<<grid, block, 0, st>>>(a, max_blocks);
  }
  return hipGetLastError();
}

template <int D>
hipError_t attn_by_nrep(const PrefillArgs& a, int n_rep, hipStream_t st) {
  switch (n_rep) {
    case 1: return attn_launch<D, 1>(a, st);
    case 2: return attn_launch<D, 2>(a, st);
    case 4: return attn_launch<D, 4>(a, st);
    case 8: return attn_launch<D, 8>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill_kv_write(const PrefillArgs& a, int head_dim, bool fp8, hipStream_t stream) {
  const long long blocks = (long long)a.num_groups * a.max_prefix_pages * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(64);
  if (head_dim == 128) {
    if (fp8) prefill_kv_write_kernel<128, true><<<grid, block, 0, stream>>>(a);
    else prefill_kv_write_kernel<128, false><<<grid, block, 0, stream>>>(a);
  } else if (head_dim == 64) {
    if (fp8) prefill_kv_write_kernel<64, true><<<grid, block, 0, stream>>>(a);
    else prefill_kv_write_kernel<64, false><<<grid, block, 0, stream>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_prefill_attn(const PrefillArgs& a, int head_dim, int n_rep, hipStream_t stream) {
  if (head_dim == 128) return attn_by_nrep<128>(a, n_rep, stream);
  if (head_dim == 64) return attn_by_nrep<64>(a, n_rep, stream);
  return hipErrorInvalidValue;
}

}  // namespace rp
