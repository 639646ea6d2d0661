// Weight synthesis on the device, and export of a logical weight matrix.
//
// Weights are the "random-init" N(0, std) tensors of the synthetic workload:
// element i = row * cols + col of tensor `id` is hashed with SplitMix64
// (Steele, Lea & Flood, OOPSLA 2014: golden-gamma increment and the
// variant-13 finaliser), h = mix(mix(seed ^ id * gamma) + (i + 1) * gamma);
// the four 16-bit limbs of h are summed (an Irwin-Hall(4) variate s) and the
// value is fp32(((s - 131070) / 65536) * sqrt(3) * std) in IEEE double, left
// to right.  The bf16 path rounds that fp32 value to nearest-even bf16.
// The values are written straight into the physical layout the GEMMs read.
#include "internal.h"

namespace rollout {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

__device__ __forceinline__ float weight_value(uint64_t key, uint64_t i, double std_) {
  const uint64_t h = mix64(key + (i + 1ull) * kGamma);
  const int64_t s = (int64_t)(h & 0xFFFFull) + (int64_t)((h >> 16) & 0xFFFFull) +
                    (int64_t)((h >> 32) & 0xFFFFull) + (int64_t)(h >> 48);
  const double x = (double)(s - 131070);
  // separate statements: no contraction is possible across them
  double w = x / 65536.0;
  w = w * 1.7320508075688772;
  w = w * std_;
  return (float)w;
}

// Physical (row, col) of the 8-element group starting at physical index p.
__device__ __forceinline__ void phys_rc(const WeightDesc& w, size_t p, int* row, int* col) {
  if (w.layout == W_TILED) {
    const int lane = (int)((p >> 3) & 63);
    const size_t tile = p >> 9;
    const int kbs = w.cols / 32;
    const int kb = (int)(tile % (size_t)kbs);
    const int nb = (int)(tile / (size_t)kbs);
    *row = nb * 16 + (lane & 15);
    *col = kb * 32 + (lane >> 4) * 8;
  } else {
    *row = (int)(p / (size_t)w.cols);
    *col = (int)(p % (size_t)w.cols);
  }
}

// Tensor id slot (0, 1, 2) and logical row of a physical row.
__device__ __forceinline__ void row_source(const WeightDesc& w, int prow, int* which, int* lrow) {
  if (w.fuse == FUSE_QKV) {
    if (prow < w.a) { *which = 0; *lrow = prow; }
    else if (prow < w.a + w.b) { *which = 1; *lrow = prow - w.a; }
    else { *which = 2; *lrow = prow - w.a - w.b; }
  } else if (w.fuse == FUSE_GU) {
    *which = prow & 1;
    *lrow = prow >> 1;
  } else {
    *which = 0;
    *lrow = prow;
  }
}

template <typename T>
__global__ void k_synth(T* __restrict__ dst, WeightDesc w, uint64_t k0, uint64_t k1, uint64_t k2, double std_) {
  const size_t n_groups = (size_t)w.rows * (size_t)w.cols / 8;
  for (size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x; g < n_groups; g += (size_t)gridDim.x * blockDim.x) {
    const size_t p = g * 8;
    int prow, pcol, which, lrow;
    phys_rc(w, p, &prow, &pcol);
    row_source(w, prow, &which, &lrow);
    const uint64_t key = which == 0 ? k0 : (which == 1 ? k1 : k2);
    const uint64_t base = (uint64_t)lrow * (uint64_t)w.cols + (uint64_t)pcol;
#pragma unroll
    for (int e = 0; e < 8; ++e) stf(dst, p + e, weight_value(key, base + e, std_));
  }
}

__global__ void k_fill(float* __restrict__ dst, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = v;
}

template <typename T>
__global__ void k_export(const T* __restrict__ src, WeightDesc w, int which, int rows, float* __restrict__ out) {
  const size_t n = (size_t)rows * (size_t)w.cols;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / (size_t)w.cols), c = (int)(i % (size_t)w.cols);
    int prow = r;
    if (w.fuse == FUSE_QKV) prow = which == 0 ? r : (which == 1 ? w.a + r : w.a + w.b + r);
    else if (w.fuse == FUSE_GU) prow = 2 * r + which;
    size_t p;
    if (w.layout == W_TILED) {
      const int nb = prow >> 4, kb = c >> 5;
      const int lane = (prow & 15) + 16 * ((c & 31) >> 3);
      p = (((size_t)nb * (size_t)(w.cols / 32) + (size_t)kb) * 64 + (size_t)lane) * 8 + (size_t)(c & 7);
    } else {
      p = (size_t)prow * (size_t)w.cols + (size_t)c;
    }
    out[i] = ldf(src, p);
  }
}

uint64_t mix64_host(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

inline uint64_t stream_key(uint64_t seed, int id) { return mix64_host(seed ^ ((uint64_t)id * kGamma)); }

inline int grid_for(size_t n, int block) {
  size_t g = (n + block - 1) / block;
  return (int)(g > 65536 ? 65536 : (g < 1 ? 1 : g));
}

}  // namespace

hipError_t launch_synth(hipStream_t s, void* dst, int dtype, const WeightDesc& w, uint64_t seed, double std_) {
  const size_t groups = (size_t)w.rows * (size_t)w.cols / 8;
  const uint64_t k0 = stream_key(seed, w.id0), k1 = stream_key(seed, w.id1), k2 = stream_key(seed, w.id2);
  const int grid = grid_for(groups, 256);
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_synth<uint16_t>, dim3(grid), dim3(256), 0, s, (uint16_t*)dst, w, k0, k1, k2, std_);
  else
    hipLaunchKernelGGL(k_synth<float>, dim3(grid), dim3(256), 0, s, (float*)dst, w, k0, k1, k2, std_);
  return hipGetLastError();
}

hipError_t launch_fill(hipStream_t s, float* dst, size_t n, float value) {
  hipLaunchKernelGGL(k_fill, dim3(grid_for(n, 256)), dim3(256), 0, s, dst, n, value);
  return hipGetLastError();
}

hipError_t launch_export(hipStream_t s, const void* src, int dtype, const WeightDesc& w, int which, int rows,
                         float* out) {
  const size_t n = (size_t)rows * (size_t)w.cols;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_export<uint16_t>, dim3(grid_for(n, 256)), dim3(256), 0, s, (const uint16_t*)src, w, which,
                       rows, out);
  else
    hipLaunchKernelGGL(k_export<float>, dim3(grid_for(n, 256)), dim3(256), 0, s, (const float*)src, w, which, rows,
                       out);
  return hipGetLastError();
}

}  // namespace rollout
