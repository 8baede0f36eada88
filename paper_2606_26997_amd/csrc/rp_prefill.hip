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
// Causal attention: one wave per (group, kv-head, 16-row query tile). A tile
// holds 16 / n_rep consecutive prompt tokens times the n_rep query heads that
// share the kv-head, so the key blocks it reads serve all of them. Per 16-key
// block: S^T = K Q^T on mfma 16x16x32 bf16, a causal mask on the diagonal,
// an online softmax per row, O^T += V^T P^T on mfma 16x16x16 bf16 with V
// staged through LDS; the next block's V is requested once this block's V is
// staged and its K once the scores exist. K/V are read from the projections
// (not from the pool), as the prompt's own attention needs no quantised copy.
//
// Grid: workgroup b takes (group, kv-head) pair b % NP and tile
// max_tiles - 1 - b / NP (longest tiles, which see the most keys, first).
// Workgroups are dealt to the 8 XCDs round-robin, so with NP a multiple of 8
// every tile of a pair runs on one XCD and re-reads the pair's K/V from that
// XCD's L2.
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
// One 16-key block of kv-head h in flight (this lane's share): the A operand of
// S^T = K Q^T (lane (r16, quad) holds key r16, columns kb*32 + quad*8 + 0..7)
// and 16-byte pieces of the block's V rows for staging.
template <int D>
struct KeyBlock {
  uint4 k[D / 32];
  uint4 v[kPage * D * 2 / 1024];
};

// Rows at or past the prompt's end are read from its last token (inside the
// packed arrays) and masked where used.
template <int D>
__device__ inline void load_block_k(const uint16_t* kbase, size_t pitch, int u0, int last, int lane, KeyBlock<D>& r) {
  const int r16 = lane & 15, quad = lane >> 4;
  const uint16_t* row = kbase + (size_t)min(u0 + r16, last) * pitch + quad * 8;
#pragma unroll
  for (int kb = 0; kb < D / 32; ++kb) r.k[kb] = *reinterpret_cast<const uint4*>(row + kb * 32);
}
template <int D>
__device__ inline void load_block_v(const uint16_t* vbase, size_t pitch, int u0, int last, int lane, KeyBlock<D>& r) {
#pragma unroll
  for (int i = 0; i < kPage * D * 2 / 1024; ++i) {
    const int e0 = i * 512 + lane * 8;
    const int tok = e0 / D, col = e0 % D;
    r.v[i] = *reinterpret_cast<const uint4*>(vbase + (size_t)min(u0 + tok, last) * pitch + col);
  }
}

template <int D, int NREP>
__global__ __launch_bounds__(64) void prefill_attn_kernel(const PrefillArgs a, int max_tiles) {
  constexpr int KB = D / 32;        // MFMA k-blocks over head_dim
  constexpr int DT = D / 16;        // 16-column output tiles
  constexpr int STRIDE = D + 4;     // staged V row pitch (bf16)
  constexpr int QSTRIDE = D + 8;    // query tile row pitch (bf16)
  constexpr int TPT = 16 / NREP;    // prompt tokens per 16-row tile
  __shared__ __attribute__((aligned(16))) uint16_t vt[kPage * STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t qt[16 * QSTRIDE];

  const int Hkv = a.num_kv_heads, Hq = a.num_q_heads;
  const int NP = a.num_groups * Hkv;
  const int pair = (int)(blockIdx.x % (unsigned)NP);
  const int tile = max_tiles - 1 - (int)(blockIdx.x / (unsigned)NP);
  const int g = pair / Hkv, h = pair - g * Hkv;
  int first;
  const int P = prompt_len(a, g, &first);
  const int t0 = tile * TPT;
  if (t0 >= P) return;
  const int lane = threadIdx.x, r16 = lane & 15, quad = lane >> 4;
  const int last = P - 1;

  // Row r16 of the tile: token t0 + r16 / NREP, query head h * NREP + r16 % NREP.
  const int tr = t0 + r16 / NREP;
  const bool row_ok = tr < P;
  const int jr = h * NREP + r16 % NREP;
  const size_t qpitch = (size_t)Hq * D, kpitch = (size_t)Hkv * D;
  const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + (size_t)(first + min(tr, last)) * qpitch + (size_t)jr * D;
  const uint16_t* kbase = static_cast<const uint16_t*>(a.k) + (size_t)first * kpitch + (size_t)h * D;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v) + (size_t)first * kpitch + (size_t)h * D;
  uint16_t* qt_lane = qt + r16 * QSTRIDE + quad * 8;
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    uint4 w = make_uint4(0, 0, 0, 0);
    if (row_ok) w = *reinterpret_cast<const uint4*>(qrow + kb * 32 + quad * 8);
    *reinterpret_cast<uint4*>(qt_lane + kb * 32) = w;
  }

  const int tlast = min(t0 + TPT, P) - 1;  // the tile's last token bounds its keys
  const int nblk = tlast / kPage + 1;
  float mrow = -INFINITY, lrow = 0.f;
  f32x4_t oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  KeyBlock<D> kv;
  load_block_k<D>(kbase, kpitch, 0, last, lane, kv);
  load_block_v<D>(vbase, kpitch, 0, last, lane, kv);
  for (int blk = 0; blk < nblk; ++blk) {
    const int u0 = blk * kPage;
    const int un = blk + 1 < nblk ? u0 + kPage : u0;  // the next block (this one again after the last)

    // Stage this block's V (rows past the prompt as zeros), then request the next.
    __syncthreads();  // the previous block's LDS reads (and the query tile writes) are complete
#pragma unroll
    for (int i = 0; i < kPage * D * 2 / 1024; ++i) {
      const int e0 = i * 512 + lane * 8;
      const int tok = e0 / D, col = e0 % D;
      const uint4 w = u0 + tok <= last ? kv.v[i] : make_uint4(0, 0, 0, 0);
      uint2* dst = reinterpret_cast<uint2*>(vt + tok * STRIDE + col);
      dst[0] = make_uint2(w.x, w.y);
      dst[1] = make_uint2(w.z, w.w);
    }
    __builtin_amdgcn_sched_barrier(0);
    load_block_v<D>(vbase, kpitch, un, last, lane, kv);

    // Entry i of this lane: key u0 + quad*4 + i against tile row r16.
    f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const bf16x8_t qop = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qt_lane + kb * 32));
      sacc = mfma16x16x32(__builtin_bit_cast(bf16x8_t, kv.k[kb]), qop, sacc);
    }
    __builtin_amdgcn_sched_barrier(0);
    load_block_k<D>(kbase, kpitch, un, last, lane, kv);

    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = u0 + quad * 4 + i;
      x[i] = (row_ok && u <= tr) ? sacc[i] * a.qk_scale : -INFINITY;
    }
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
    const bf16x4_t pop =
        __builtin_bit_cast(bf16x4_t, make_uint2(pack_bf16x2(pw[0], pw[1]), pack_bf16x2(pw[2], pw[3])));

    __syncthreads();  // the staged V is visible
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const uint16_t* col = vt + (quad * 4) * STRIDE + dt * 16 + r16;
      const uint32_t w0 = (uint32_t)col[0] | ((uint32_t)col[STRIDE] << 16);
      const uint32_t w1 = (uint32_t)col[2 * STRIDE] | ((uint32_t)col[3 * STRIDE] << 16);
      oacc[dt] = mfma16x16x16(__builtin_bit_cast(bf16x4_t, make_uint2(w0, w1)), pop, oacc[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  const float lt = xor_sum_from<16>(lrow);
  if (!row_ok) return;
  const float inv = 1.f / lt;
  uint16_t* orow = static_cast<uint16_t*>(a.out) + (size_t)(first + tr) * qpitch + (size_t)jr * D + quad * 4;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const f32x4_t v = oacc[dt] * inv;
    *reinterpret_cast<uint2*>(orow + dt * 16) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
  if (a.lse != nullptr && quad == 0) a.lse[(size_t)(first + tr) * Hq + jr] = (mrow + fast_log2(lt)) * kLn2;
}

template <int D>
hipError_t attn_by_nrep(const PrefillArgs& a, int n_rep, hipStream_t st) {
  const long long NP = (long long)a.num_groups * a.num_kv_heads;
  const int max_tiles = cdiv(a.max_prefix_pages * kPage, 16 / n_rep);
  const long long blocks = NP * max_tiles;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(64);
  switch (n_rep) {
    case 1: prefill_attn_kernel<D, 1><<<grid, block, 0, st>>>(a, max_tiles); break;
    case 2: prefill_attn_kernel<D, 2><<<grid, block, 0, st>>>(a, max_tiles); break;
    case 4: prefill_attn_kernel<D, 4><<<grid, block, 0, st>>>(a, max_tiles); break;
    case 8: prefill_attn_kernel<D, 8><<<grid, block, 0, st>>>(a, max_tiles); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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
