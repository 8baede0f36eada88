// Pre-attention side of one decode step of a Qwen3-style attention layer.
// For sequence s (group g = seq_to_group[s]) the new token sits at position
// prefix_lens[g] + resp_lens[s]. Every q head and k head is RMS-normalised
// with the layer's per-channel weights and rotated by the rotary embedding
// (pairs (i, i + D/2), angle position * theta^(-2i/D)); q goes to q_out, k
// and the unchanged v are appended at response slot resp_lens[s] (bf16 copy
// or the fp8 append rule).
//
// The arithmetic is fp64 on the bf16 inputs with one rounding to bf16 at the
// end, so each output is the correctly rounded value unless the exact value
// lies within a few fp64 ulps of a bf16 rounding boundary. The angles are
// computed once per block into LDS.
//
// Grid: blocks of 4 waves; one block covers heads_per_block of the Hq + Hkv
// heads of one sequence, wave w taking heads h0 + w, h0 + w + 4, ...; q head
// j < Hq, kv-head j - Hq otherwise. Lane l handles columns l + 64 e.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kPrepWaves = 4;
constexpr int kPrepThreads = 64 * kPrepWaves;

// fp64 -> bf16 bits with a single rounding to nearest even. Below 2^-126 the
// bf16 grid is the subnormal step 2^-133; above, the 52-bit mantissa is
// rounded to 7 bits on the integer pattern (a carry bumps the exponent) and
// the result converts to fp32 exactly. Finite inputs (NaN maps to 0x7FC0).
__device__ inline uint32_t f64_to_bf16_rne(double x) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const uint32_t sign = (uint32_t)(u >> 48) & 0x8000u;
  const unsigned long long a = u & 0x7FFFFFFFFFFFFFFFull;
  if (a > 0x7FF0000000000000ull) return 0x7FC0u;
  if (a < 0x3810000000000000ull) {                     // |x| < 2^-126
    const double q = rint(__longlong_as_double((long long)a) * 0x1p133);  // exact scaling
    return sign | (uint32_t)q;                          // 0..128; 128 is 2^-126
  }
  const unsigned long long r = (a + 0x00000FFFFFFFFFFFull + ((a >> 45) & 1ull)) & ~0x00001FFFFFFFFFFFull;
  const float f = (float)__longlong_as_double((long long)r);  // exact (inf past the bf16 range)
  return sign | (__float_as_uint(f) >> 16);
}

__device__ inline double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// RMS norm and rotary embedding of one head (all lanes of the wave), rounded
// to bf16 bits.
template <int D>
__device__ inline void norm_rope(const uint16_t* src, const uint16_t* w, double eps, const double* s_cos,
                                 const double* s_sin, int lane, uint32_t (&out)[D / 64]) {
  constexpr int EPL = D / 64;
  double x[EPL];
  double ss = 0.0;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    x[e] = (double)__uint_as_float((uint32_t)src[64 * e + lane] << 16);
    ss += x[e] * x[e];
  }
  const double den = sqrt(wave_sum_f64(ss) / D + eps);
#pragma unroll
  for (int e = 0; e < EPL; ++e) x[e] = x[e] / den * (double)__uint_as_float((uint32_t)w[64 * e + lane] << 16);
  if constexpr (EPL == 2) {
    // Columns lane and lane + 64 form pair `lane`.
    const double c = s_cos[lane], sn = s_sin[lane];
    out[0] = f64_to_bf16_rne(x[0] * c - x[1] * sn);
    out[1] = f64_to_bf16_rne(x[1] * c + x[0] * sn);
  } else {
    // Column lane pairs with lane ^ 32.
    const double p = __shfl_xor(x[0], 32);
    const double c = s_cos[lane & 31], sn = s_sin[lane & 31];
    out[0] = f64_to_bf16_rne(lane < 32 ? x[0] * c - p * sn : x[0] * c + p * sn);
  }
}

template <int D, bool FP8>
__global__ __launch_bounds__(kPrepThreads) void qk_prep_kernel(const QkPrepArgs a) {
  constexpr int EPL = D / 64;
  constexpr int HALF = D / 2;
  __shared__ double s_cos[HALF], s_sin[HALF];
  const int Hq = a.num_q_heads, Hkv = a.num_kv_heads;
  const int s = blockIdx.x / a.blocks_per_seq;
  const int h0 = (blockIdx.x - s * a.blocks_per_seq) * a.heads_per_block;
  const int h1 = min(h0 + a.heads_per_block, Hq + Hkv);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int g = clamp_group(a.seq_to_group[s], a.num_groups);
  const int L = a.resp_lens[s];
  if (t < HALF) {
    const double pos = (double)a.prefix_lens[g] + (double)L;
    double sn, cs;
    sincos(pos * pow(a.rope_theta, (-2.0 * t) / D), &sn, &cs);
    s_cos[t] = cs;
    s_sin[t] = sn;
  }
  __syncthreads();

  const bool slot_ok = L >= 0 && L < a.max_resp_pages * kPage;
  int page = 0;
  if (slot_ok) page = clamp_page(a.resp_block_table[(size_t)s * a.max_resp_pages + L / kPage], a.num_pages);
  const int r = L % kPage;

  for (int j = h0 + wave; j < h1; j += kPrepWaves) {
    uint32_t o[EPL];
    if (j < Hq) {
      const size_t off = ((size_t)s * Hq + j) * D;
      norm_rope<D>(a.q_in + off, a.q_norm_w, a.rms_eps, s_cos, s_sin, lane, o);
#pragma unroll
      for (int e = 0; e < EPL; ++e) a.q_out[off + 64 * e + lane] = (uint16_t)o[e];
      continue;
    }
    const int h = j - Hq;
    const size_t off = ((size_t)s * Hkv + h) * D;
    norm_rope<D>(a.k_in + off, a.k_norm_w, a.rms_eps, s_cos, s_sin, lane, o);
    uint32_t vb[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) vb[e] = a.v_in[off + 64 * e + lane];
    if (a.k_out != nullptr) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) a.k_out[off + 64 * e + lane] = (uint16_t)o[e];
    }
    if (!slot_ok) continue;
    const size_t blk = ((size_t)page * Hkv + h) * kPage * D;  // in elements
    if constexpr (!FP8) {
      uint16_t* kd = static_cast<uint16_t*>(a.k_pages) + blk + (size_t)r * D + lane;
      uint16_t* vd = static_cast<uint16_t*>(a.v_pages) + blk + (size_t)r * D + lane;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        kd[64 * e] = (uint16_t)o[e];
        vd[64 * e] = (uint16_t)vb[e];
      }
    } else {
      const size_t sidx = (size_t)page * Hkv + h;
      float kx[EPL], vx[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        kx[e] = __uint_as_float(o[e] << 16);
        vx[e] = __uint_as_float(vb[e] << 16);
      }
      append_fp8_row<D>(static_cast<uint8_t*>(a.k_pages) + blk, a.k_scale + sidx, r, kx, lane);
      append_fp8_row<D>(static_cast<uint8_t*>(a.v_pages) + blk, a.v_scale + sidx, r, vx, lane);
    }
  }
}

template <int D>
hipError_t launch_d(const QkPrepArgs& a, bool fp8, hipStream_t stream) {
  const dim3 grid((unsigned)((long long)a.num_seqs * a.blocks_per_seq)), block(kPrepThreads);
  if (fp8) qk_prep_kernel<D, true><<<grid, block, 0, stream>>>(a);
  else qk_prep_kernel<D, false><<<grid, block, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

// Small batches split a sequence's heads over blocks of one head per wave
// (more blocks in flight); from 1024 sequences on, one block per sequence
// computes the angles once for all of its heads.
hipError_t launch_qk_prep(QkPrepArgs a, int head_dim, bool fp8, hipStream_t stream) {
  if (a.num_seqs <= 0) return hipSuccess;
  const int heads = a.num_q_heads + a.num_kv_heads;
  a.blocks_per_seq = a.num_seqs >= 1024 ? 1 : cdiv(heads, kPrepWaves);
  a.heads_per_block = cdiv(heads, a.blocks_per_seq);
  if (head_dim == 128) return launch_d<128>(a, fp8, stream);
  if (head_dim == 64) return launch_d<64>(a, fp8, stream);
  return hipErrorInvalidValue;
}

}  // namespace rp
