// ForkGRPO objective and JustGRPO-Fast position selection (Fork-dLLM paper,
// Section 3.2).
//
// Objective: for each prompt (group g of G rollouts) the advantages
// A_i = (r_i - mean_g) / std_g (std with divisor G; a group with std 0 is
// skipped), the ratios rho_e = exp(log q_new - log q_old) of the rollout's
// fallback-step entries e, the clipped terms min(rho A, clip(rho, 1-eps,
// 1+eps) A), their mean over each rollout's entries, the mean over the
// group's rollouts, and finally the mean over the groups not skipped.  One
// workgroup per group; every sum is a fixed-order reduction, so results are
// bit-reproducible.  The likelihoods themselves come from the teacher-forced
// LM head (gemm_stats target kernels + merge).
//
// Selection: per rollout, the k positions of highest entropy (equal values
// in increasing position): each position counts the positions ordered
// before it, from a copy of the rollout's entropies in LDS.
#include "fork_kernels.h"

#include <math.h>

namespace fork {
namespace {

constexpr int kGrpoThreads = 256;
constexpr int kGrpoWaves = kGrpoThreads / 64;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Sum over the workgroup in a fixed order: wave sums, then wave 0 adds them.
__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kGrpoWaves; ++k) s += red[k];
  __syncthreads();
  return s;
}

__global__ __launch_bounds__(kGrpoThreads) void grpo_group_kernel(
    int G, int n, const float* __restrict__ rewards, const int32_t* __restrict__ offsets,
    const float* __restrict__ lp_new, const float* __restrict__ lp_old, float eps,
    float* __restrict__ adv, float* __restrict__ ratio, float* __restrict__ term,
    float* __restrict__ rollout_obj, float* __restrict__ group_obj,
    uint8_t* __restrict__ skipped) {
  __shared__ float red[kGrpoWaves];
  __shared__ float ro[kMaxGroupSize];
  const int g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* r = rewards + (size_t)g * G;

  float s = 0.f;
  for (int j = tid; j < G; j += kGrpoThreads) s += r[j];
  const float mean = block_sum(s, red) / (float)G;
  float q = 0.f;
  for (int j = tid; j < G; j += kGrpoThreads) q += (r[j] - mean) * (r[j] - mean);
  const float sd = sqrtf(block_sum(q, red) / (float)G);
  const bool skip = !(sd > 0.f);

  // one wave per rollout, lanes over its entries
  for (int j = w; j < G; j += kGrpoWaves) {
    const size_t i = (size_t)g * G + j;
    const float A = skip ? 0.f : (r[j] - mean) / sd;
    const int e0 = min(max(offsets[i], 0), n), e1 = min(max(offsets[i + 1], e0), n);
    float acc = 0.f;
    for (int e = e0 + lane; e < e1; e += 64) {
      const float rho = expf(lp_new[e] - lp_old[e]);
      const float clipped = fminf(fmaxf(rho, 1.f - eps), 1.f + eps);
      const float tm = fminf(rho * A, clipped * A);
      if (ratio) ratio[e] = rho;
      if (term) term[e] = tm;
      acc += tm;
    }
    acc = wave_sum(acc);
    const float obj = e1 > e0 ? acc / (float)(e1 - e0) : 0.f;
    if (lane == 0) {
      ro[j] = obj;
      if (adv) adv[i] = A;
      if (rollout_obj) rollout_obj[i] = obj;
    }
  }
  __syncthreads();
  float t = 0.f;
  for (int j = tid; j < G; j += kGrpoThreads) t += ro[j];
  const float gsum = block_sum(t, red);
  if (tid == 0) {
    group_obj[g] = skip ? 0.f : gsum / (float)G;
    skipped[g] = skip ? 1 : 0;
  }
}

__global__ __launch_bounds__(kGrpoThreads) void grpo_batch_kernel(
    int n_groups, const float* __restrict__ group_obj, const uint8_t* __restrict__ skipped,
    float* __restrict__ J) {
  __shared__ float red[kGrpoWaves];
  float s = 0.f, c = 0.f;
  for (int g = threadIdx.x; g < n_groups; g += kGrpoThreads)
    if (!skipped[g]) {
      s += group_obj[g];
      c += 1.f;
    }
  const float total = block_sum(s, red);
  const float kept = block_sum(c, red);
  if (threadIdx.x == 0) J[0] = kept > 0.f ? total / kept : 0.f;
}

__global__ __launch_bounds__(kGrpoThreads) void top_entropy_kernel(
    int Lg, int k, const float* __restrict__ entropy, uint8_t* __restrict__ sel) {
  __shared__ float h[kMaxTopEntropyLen];
  const size_t base = (size_t)blockIdx.x * Lg;
  for (int p = threadIdx.x; p < Lg; p += kGrpoThreads) h[p] = entropy[base + p];
  __syncthreads();
  for (int p = threadIdx.x; p < Lg; p += kGrpoThreads) {
    const float hp = h[p];
    int ahead = 0;
    for (int q = 0; q < Lg; ++q) {
      const float hq = h[q];
      ahead += (hq > hp || (hq == hp && q < p)) ? 1 : 0;
    }
    sel[base + p] = ahead < k ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_grpo_objective(int n_groups, int G, int n, const float* rewards,
                                 const int32_t* offsets, const float* lp_new,
                                 const float* lp_old, float eps, float* adv, float* ratio,
                                 float* term, float* rollout_obj, float* group_obj,
                                 uint8_t* skipped, float* J, hipStream_t stream) {
  if (n_groups > 0)
    hipLaunchKernelGGL(grpo_group_kernel, dim3((unsigned)n_groups), dim3(kGrpoThreads), 0,
                       stream, G, n, rewards, offsets, lp_new, lp_old, eps, adv, ratio, term,
                       rollout_obj, group_obj, skipped);
  hipLaunchKernelGGL(grpo_batch_kernel, dim3(1), dim3(kGrpoThreads), 0, stream, n_groups,
                     group_obj, skipped, J);
  return hipGetLastError();
}

hipError_t launch_top_entropy(int R, int Lg, int k, const float* entropy, uint8_t* sel,
                              hipStream_t stream) {
  if (R > 0)
    hipLaunchKernelGGL(top_entropy_kernel, dim3((unsigned)R), dim3(kGrpoThreads), 0, stream,
                       Lg, k, entropy, sel);
  return hipGetLastError();
}

}  // namespace fork
