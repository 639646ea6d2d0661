// Group-relative advantages (the comparison of each completion's reward with
// its own group, section 3 of the paper; GRPO's normalisation by the group's
// standard deviation).  One wavefront per group, float64 arithmetic, a fixed
// shuffle-tree reduction order.  Groups whose rewards are all equal (tested as
// max == min, never through a computed standard deviation) and groups of one
// get advantage 0 and are counted as zero-variance groups.
#include "internal.h"

namespace rollout {
namespace {

__device__ __forceinline__ double wsum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ void k_zero_i32(int32_t* p) {
  if (threadIdx.x == 0) *p = 0;
}

__global__ __launch_bounds__(64) void k_grpo(const float* __restrict__ r, int G, double eps, int ddof,
                                             float* __restrict__ adv, int32_t* __restrict__ zero_var) {
  const int g = blockIdx.x, lane = threadIdx.x;
  const float* x = r + (size_t)g * G;
  float* a = adv + (size_t)g * G;
  double mx = -INFINITY, mn = INFINITY, sum = 0.0;
  for (int i = lane; i < G; i += 64) {
    const double v = (double)x[i];
    mx = fmax(mx, v);
    mn = fmin(mn, v);
    sum += v;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmax(mx, __shfl_xor(mx, o, 64));
    mn = fmin(mn, __shfl_xor(mn, o, 64));
  }
  sum = wsum(sum);
  if (G == 1 || mx == mn) {
    for (int i = lane; i < G; i += 64) a[i] = 0.f;
    if (lane == 0 && zero_var) atomicAdd(zero_var, 1);
    return;
  }
  const double mu = sum / (double)G;
  double ss = 0.0;
  for (int i = lane; i < G; i += 64) {
    const double dv = (double)x[i] - mu;
    ss += dv * dv;
  }
  ss = wsum(ss);
  const double sigma = sqrt(ss / (double)(G - ddof));
  for (int i = lane; i < G; i += 64) a[i] = (float)(((double)x[i] - mu) / (sigma + eps));
}

}  // namespace

hipError_t launch_grpo(hipStream_t s, const float* r, int n_groups, int G, float eps, int ddof, float* adv,
                       int32_t* zero_var) {
  if (zero_var) hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, s, zero_var);
  hipLaunchKernelGGL(k_grpo, dim3(n_groups), dim3(64), 0, s, r, G, (double)eps, ddof, adv, zero_var);
  return hipGetLastError();
}

}  // namespace rollout
