// GRPO group statistics and advantages (Eq. 1): for each group of K rewards,
// mu = sum r / K, sigma = sqrt(sum (r - mu)^2 / (K - ddof)) (0 when
// K - ddof < 1) and A_i = (r_i - mu) / (sigma + eps), all in fp64 from the
// fp32 rewards, each output rounded once to fp32. One thread per group; for
// K = 4, 8 and 16 the group is loaded with 16-byte vector loads and kept in
// registers, otherwise it is read from memory (and cache) once per pass.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kGrpoThreads = 256;

template <int KC>
__global__ __launch_bounds__(kGrpoThreads) void grpo_fixed_kernel(const GrpoArgs a) {
  const int g = blockIdx.x * kGrpoThreads + threadIdx.x;
  if (g >= a.num_groups) return;
  const float4* src = reinterpret_cast<const float4*>(a.rewards + (size_t)g * KC);
  float x[KC];
#pragma unroll
  for (int v = 0; v < KC / 4; ++v) {
    const float4 f = src[v];
    x[4 * v] = f.x;
    x[4 * v + 1] = f.y;
    x[4 * v + 2] = f.z;
    x[4 * v + 3] = f.w;
  }
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < KC; ++i) s += (double)x[i];
  const double mu = s / KC;
  double ss = 0.0;
#pragma unroll
  for (int i = 0; i < KC; ++i) {
    const double d = (double)x[i] - mu;
    ss += d * d;
  }
  const int den = KC - a.ddof;
  const double sd = den > 0 ? sqrt(ss / den) : 0.0;
  const double div = sd + a.eps_std;
  float4* dst = reinterpret_cast<float4*>(a.advantages + (size_t)g * KC);
#pragma unroll
  for (int v = 0; v < KC / 4; ++v) {
    float4 o;
    o.x = (float)(((double)x[4 * v] - mu) / div);
    o.y = (float)(((double)x[4 * v + 1] - mu) / div);
    o.z = (float)(((double)x[4 * v + 2] - mu) / div);
    o.w = (float)(((double)x[4 * v + 3] - mu) / div);
    dst[v] = o;
  }
  if (a.mean != nullptr) a.mean[g] = (float)mu;
  if (a.stdev != nullptr) a.stdev[g] = (float)sd;
}

__global__ __launch_bounds__(kGrpoThreads) void grpo_any_kernel(const GrpoArgs a) {
  const int g = blockIdx.x * kGrpoThreads + threadIdx.x;
  if (g >= a.num_groups) return;
  const int K = a.group_size;
  const float* x = a.rewards + (size_t)g * K;
  double s = 0.0;
  for (int i = 0; i < K; ++i) s += (double)x[i];
  const double mu = s / K;
  double ss = 0.0;
  for (int i = 0; i < K; ++i) {
    const double d = (double)x[i] - mu;
    ss += d * d;
  }
  const int den = K - a.ddof;
  const double sd = den > 0 ? sqrt(ss / den) : 0.0;
  const double div = sd + a.eps_std;
  float* y = a.advantages + (size_t)g * K;
  for (int i = 0; i < K; ++i) y[i] = (float)(((double)x[i] - mu) / div);
  if (a.mean != nullptr) a.mean[g] = (float)mu;
  if (a.stdev != nullptr) a.stdev[g] = (float)sd;
}

}  // namespace

hipError_t launch_grpo(const GrpoArgs& a, hipStream_t stream) {
  if (a.num_groups <= 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(a.num_groups, kGrpoThreads)), block(kGrpoThreads);
  if (a.vector_ok && a.group_size == 8) grpo_fixed_kernel<8><<<grid, block, 0, stream>>>(a);
  else if (a.vector_ok && a.group_size == 4) grpo_fixed_kernel<4><<<grid, block, 0, stream>>>(a);
  else if (a.vector_ok && a.group_size == 16) grpo_fixed_kernel<16><<<grid, block, 0, stream>>>(a);
  else grpo_any_kernel<<<grid, block, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rp
