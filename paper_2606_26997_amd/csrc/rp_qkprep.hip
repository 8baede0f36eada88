// Pre-attention side of one decode step of a Qwen3-style attention layer.
// For sequence s (group g = seq_to_group[s]) the new token sits at position
// prefix_lens[g] + resp_lens[s]. Every q head and k head is RMS-normalised
// with the layer's per-channel weights and rotated by the rotary embedding
// (pairs (i, i + D/2), angle position * inv_freq[i]); q goes to q_out, k and
// the unchanged v are appended at response slot resp_lens[s] (bf16 copy or
// the fp8 append rule).
//
// The arithmetic is fp64 on the bf16 inputs with one rounding to bf16 at the
// end, so each output is the correctly rounded value unless the exact value
// lies within a few fp64 ulps of a bf16 rounding boundary.
//
// Work split: a sequence has Hq + 2 Hkv head slots (q heads, k heads, v
// heads); a group of 16 lanes owns one slot (or two, j and j + 16, on large
// batches), a block of 256 threads 16 (32) slots of one sequence, all of
// their loads in flight at once. Lane l of a group holds the D/32 pairs
// l*D/32 + p, that is columns l*D/32 + p and D/2 + l*D/32 + p, so each pair
// is rotated in-lane and every row is read and written as whole 16-lane
// runs. Each block computes the cos/sin of the D/2 angles of its sequence
// once, folded with the norm weights into LDS tables.
#include "rp_device.h"
#include "rp_internal.h"
#include "rp_plan_small.h"

namespace rp {
namespace {

constexpr int kSlotLanes = 16;
constexpr int kPrepThreads = 256;
constexpr int kGroups = kPrepThreads / kSlotLanes;

// fp64 -> bf16 bits, one rounding to nearest even, in two steps: the fp32
// rounding f of y, then f's own rounding to bf16 (pack_bf16x2, nearest
// even). That is the single rounding of y except when f lands exactly on a
// bf16 tie while y does not; then y's side of the tie decides
// (bf16_tie_fix). bf16_tie reports that case.
__device__ inline bool bf16_tie(float f) { return (__float_as_uint(f) & 0xFFFFu) == 0x8000u; }
__device__ inline uint32_t bf16_tie_fix(double y, float f) {
  const uint32_t u = __float_as_uint(f);
  const double d = y - (double)f;  // exact
  if (d == 0.0) return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return (u >> 16) + ((d > 0.0) == ((u >> 31) == 0u) ? 1u : 0u);
}
__device__ inline void set_half(uint32_t& w, int hi, uint32_t v) {
  w = hi ? (w & 0xFFFFu) | (v << 16) : (w & 0xFFFF0000u) | v;
}

// W 32-bit words (2W bf16) starting at element `col` of a row.
template <int W>
__device__ inline void load_words(const uint16_t* row, int col, uint32_t (&w)[W]) {
  if constexpr (W == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(row + col);
    w[0] = v.x;
    w[1] = v.y;
  } else {
    w[0] = *reinterpret_cast<const uint32_t*>(row + col);
  }
}
template <int W>
__device__ inline void store_words(uint16_t* row, int col, const uint32_t (&w)[W]) {
  if constexpr (W == 2) {
    *reinterpret_cast<uint2*>(row + col) = make_uint2(w[0], w[1]);
  } else {
    *reinterpret_cast<uint32_t*>(row + col) = w[0];
  }
}

__device__ inline double bf16_word_f64(const uint32_t* w, int p) {
  return (double)(p & 1 ? bf16_hi(w[p >> 1]) : bf16_lo(w[p >> 1]));
}

template <int D, bool FP8>
__device__ inline void prep_slot(const QkPrepArgs& a, int s, int kind, int head, int l16, int L,
                                 const uint32_t (&x1)[D / 64], const uint32_t (&x2)[D / 64],
                                 const double (*s_tab)[4][D / 2]) {
  constexpr int NP = D / 32;   // pairs per lane
  constexpr int W = NP / 2;    // 32-bit words per lane and half row
  constexpr int HALF = D / 2;
  const int Hq = a.num_q_heads, Hkv = a.num_kv_heads;
  const int c1 = l16 * NP, c2 = HALF + l16 * NP;  // first columns of the lane's two runs
  uint32_t o1[W], o2[W];
  if (kind == 2) {
#pragma unroll
    for (int k = 0; k < W; ++k) {
      o1[k] = x1[k];
      o2[k] = x2[k];
    }
  } else {
    double y1[NP], y2[NP];
    double ss = 0.0;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      y1[p] = bf16_word_f64(x1, p);
      y2[p] = bf16_word_f64(x2, p);
      ss += y1[p] * y1[p] + y2[p] * y2[p];
    }
#pragma unroll
    for (int o = kSlotLanes / 2; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
    // 1 / sqrt(mean + eps): hardware estimate refined by two Newton steps
    // (a few fp64 ulps).
    const double m = ss / D + a.rms_eps;
    const double hm = 0.5 * m;
    double inv = __builtin_amdgcn_rsq(m);
    inv = inv * fma(-hm * inv, inv, 1.5);
    inv = inv * fma(-hm * inv, inv, 1.5);
    const double(*tab)[HALF] = s_tab[kind];
    double z1[NP], z2[NP];
    float f1[NP], f2[NP];
    bool tie = false;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int i = c1 + p;
      z1[p] = inv * fma(y1[p], tab[0][i], -(y2[p] * tab[1][i]));
      z2[p] = inv * fma(y2[p], tab[2][i], y1[p] * tab[3][i]);
      f1[p] = (float)z1[p];
      f2[p] = (float)z2[p];
      tie = tie || bf16_tie(f1[p]) || bf16_tie(f2[p]);
    }
#pragma unroll
    for (int k = 0; k < W; ++k) {
      o1[k] = pack_bf16x2(f1[2 * k], f1[2 * k + 1]);
      o2[k] = pack_bf16x2(f2[2 * k], f2[2 * k + 1]);
    }
    if (tie) {  // rare: some fp32 value sits exactly on a bf16 tie
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        if (bf16_tie(f1[p])) set_half(o1[p >> 1], p & 1, bf16_tie_fix(z1[p], f1[p]));
        if (bf16_tie(f2[p])) set_half(o2[p >> 1], p & 1, bf16_tie_fix(z2[p], f2[p]));
      }
    }
    if (kind == 0) {
      uint16_t* dst = a.q_out + ((size_t)s * Hq + head) * D;
      store_words<W>(dst, c1, o1);
      store_words<W>(dst, c2, o2);
      return;
    }
    if (a.k_out != nullptr) {
      uint16_t* dst = a.k_out + ((size_t)s * Hkv + head) * D;
      store_words<W>(dst, c1, o1);
      store_words<W>(dst, c2, o2);
    }
  }

  // Append of k (kind 1) or v (kind 2) at response slot L.
  if (L < 0 || L >= a.max_resp_pages * kPage) return;  // no slot for the new token
  const int page = clamp_page(a.resp_block_table[(size_t)s * a.max_resp_pages + L / kPage], a.num_pages);
  const int r = L % kPage;
  const size_t blk = ((size_t)page * Hkv + head) * kPage * D;  // in elements
  if constexpr (!FP8) {
    uint16_t* dst = static_cast<uint16_t*>(kind == 1 ? a.k_pages : a.v_pages) + blk + (size_t)r * D;
    store_words<W>(dst, c1, o1);
    store_words<W>(dst, c2, o2);
  } else {
    float xf[2 * NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      xf[p] = p & 1 ? bf16_hi(o1[p >> 1]) : bf16_lo(o1[p >> 1]);
      xf[NP + p] = p & 1 ? bf16_hi(o2[p >> 1]) : bf16_lo(o2[p >> 1]);
    }
    const auto col = [c1, c2](int e) { return e < NP ? c1 + e : c2 + (e - NP); };
    uint8_t* pages = static_cast<uint8_t*>(kind == 1 ? a.k_pages : a.v_pages);
    float* scales = kind == 1 ? a.k_scale : a.v_scale;
    append_fp8_row<D, kSlotLanes>(pages + blk, scales + (size_t)page * Hkv + head, r, xf, col, l16 == 0);
  }
}

// Per pair i and weight set (0: q, 1: k): A = w[i] cos, B = w[i + D/2] sin,
// C = w[i + D/2] cos, E = w[i] sin, so that with the norm factor inv
//   out[i] = inv (x[i] A - x[i + D/2] B),  out[i + D/2] = inv (x[i + D/2] C + x[i] E).
template <int D>
using PrepTables = double[2][4][D / 2];

// Block `bid` of the prep grid (blocks_per_seq blocks per sequence).
template <int D, bool FP8, int SPL>
__device__ __forceinline__ void prep_block(const QkPrepArgs& a, int bid, PrepTables<D>& s_tab) {
  constexpr int W = D / 64;
  constexpr int HALF = D / 2;
  const int Hq = a.num_q_heads, Hkv = a.num_kv_heads;
  const int t = threadIdx.x, l16 = t & (kSlotLanes - 1);
  const int s = bid / a.blocks_per_seq;
  const int slot0 = (bid - s * a.blocks_per_seq) * (kGroups * SPL) + t / kSlotLanes;
  const int c1 = l16 * (D / 32), c2 = HALF + l16 * (D / 32);
  const int g = clamp_group(a.seq_to_group[s], a.num_groups);
  const int L = a.resp_lens[s];

  // The lane's slots slot0 + 16 k (k < SPL); kind 0 = q head, 1 = k head,
  // 2 = v head. Every load is issued before the tables are built.
  int kind[SPL], head[SPL];
  uint32_t x1[SPL][W], x2[SPL][W];
#pragma unroll
  for (int k = 0; k < SPL; ++k) {
    const int slot = slot0 + k * kGroups;
    kind[k] = slot < Hq ? 0 : (slot < Hq + Hkv ? 1 : (slot < Hq + 2 * Hkv ? 2 : 3));
    head[k] = kind[k] == 0 ? slot : (kind[k] == 1 ? slot - Hq : slot - Hq - Hkv);
    if (kind[k] < 3) {
      const uint16_t* src = kind[k] == 0 ? a.q_in + ((size_t)s * Hq + head[k]) * D
                                         : (kind[k] == 1 ? a.k_in : a.v_in) + ((size_t)s * Hkv + head[k]) * D;
      load_words<W>(src, c1, x1[k]);
      load_words<W>(src, c2, x2[k]);
    }
  }
  if (t < HALF) {
    const double pos = (double)a.prefix_lens[g] + (double)L;
    double sn, cs;
    sincos(pos * a.inv_freq[t], &sn, &cs);
#pragma unroll
    for (int set = 0; set < 2; ++set) {
      const uint16_t* w = set == 0 ? a.q_norm_w : a.k_norm_w;
      const double w1 = (double)__uint_as_float((uint32_t)w[t] << 16);
      const double w2 = (double)__uint_as_float((uint32_t)w[t + HALF] << 16);
      s_tab[set][0][t] = w1 * cs;
      s_tab[set][1][t] = w2 * sn;
      s_tab[set][2][t] = w2 * cs;
      s_tab[set][3][t] = w1 * sn;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < SPL; ++k) {
    if (kind[k] < 3) prep_slot<D, FP8>(a, s, kind[k], head[k], l16, L, x1[k], x2[k], s_tab);
  }
}

template <int D, bool FP8, int SPL>
__global__ __launch_bounds__(kPrepThreads) void qk_prep_kernel(const QkPrepArgs a) {
  __shared__ PrepTables<D> s_tab;
  prep_block<D, FP8, SPL>(a, blockIdx.x, s_tab);
}

// The prep of a small batch and the plan of the attention that follows, in
// one launch: the first workgroup's first wave builds the plan (the planner
// of rp_plan_small.h; the workgroup's other waves have nothing to do), every
// other workgroup is a prep block. The two share no data.
template <int D, bool FP8>
__global__ __launch_bounds__(kPrepThreads) void qk_prep_plan_kernel(const QkPrepArgs a, const PlanArgs p) {
  __shared__ union {
    PrepTables<D> tab;
    int cnt[kPlanMaxGroups];
  } sm;
  if (blockIdx.x == 0) {
    if (threadIdx.x < 64) plan_small(p, sm.cnt);
    return;
  }
  prep_block<D, FP8, 1>(a, blockIdx.x - 1, sm.tab);
}

template <int D, int SPL>
hipError_t launch_d(QkPrepArgs a, bool fp8, hipStream_t stream) {
  a.blocks_per_seq = cdiv(a.num_q_heads + 2 * a.num_kv_heads, kGroups * SPL);
  const dim3 grid((unsigned)((long long)a.num_seqs * a.blocks_per_seq)), block(kPrepThreads);
  if (fp8) qk_prep_kernel<D, true, SPL><<<grid, block, 0, stream>>>(a);
  else qk_prep_kernel<D, false, SPL><<<grid, block, 0, stream>>>(a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_prep_plan_d(QkPrepArgs a, const PlanArgs& p, bool fp8, hipStream_t stream) {
  a.blocks_per_seq = cdiv(a.num_q_heads + 2 * a.num_kv_heads, kGroups);
  const dim3 grid((unsigned)((long long)a.num_seqs * a.blocks_per_seq + 1)), block(kPrepThreads);
  if (fp8) qk_prep_plan_kernel<D, true><<<grid, block, 0, stream>>>(a, p);
  else qk_prep_plan_kernel<D, false><<<grid, block, 0, stream>>>(a, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_qk_prep_plan(QkPrepArgs a, const PlanArgs& p, int head_dim, bool fp8, hipStream_t stream) {
  if (a.num_seqs <= 0) return hipSuccess;
  if (a.num_seqs > kSmallPlanMaxSeqs || p.num_seqs != a.num_seqs) return hipErrorInvalidValue;
  if (head_dim == 128) return launch_prep_plan_d<128>(a, p, fp8, stream);
  if (head_dim == 64) return launch_prep_plan_d<64>(a, p, fp8, stream);
  return hipErrorInvalidValue;
}

// Small batches give each 16-lane group one slot (more blocks in flight);
// from 1024 sequences on, two slots, so that a block covers 32 slots and
// computes its sequence's tables once for twice the work.
hipError_t launch_qk_prep(QkPrepArgs a, int head_dim, bool fp8, hipStream_t stream) {
  if (a.num_seqs <= 0) return hipSuccess;
  const bool two = a.num_seqs >= 1024;
  if (head_dim == 128) return two ? launch_d<128, 2>(a, fp8, stream) : launch_d<128, 1>(a, fp8, stream);
  if (head_dim == 64) return two ? launch_d<64, 2>(a, fp8, stream) : launch_d<64, 1>(a, fp8, stream);
  return hipErrorInvalidValue;
}

}  // namespace rp
