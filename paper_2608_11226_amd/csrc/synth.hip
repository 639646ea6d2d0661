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
    int nb, kb;
    wfrag_inv(p >> 9, w.rows / 16, w.cols / 32, &nb, &kb);
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

// int4 weight-only format (layer projections).  Groups of 128 input features
// of one physical row, each with an fp32 scale s and an integer zero point z:
//   codes  [N/16][K/128][64 lanes][4 words]: lane l = r + 16 g holds, in word
//          j, the codes of row 16 nb + r at k = 128 gi + 32 j + 8 g + e, e = 0..7,
//          so one 16-byte load per lane covers a group.  Within a word the
//          nibbles follow AWQ's interleaved order: element e sits at nibble
//          (e >> 1) + 4 (e & 1), so a shift and one mask lift elements 2t and
//          2t + 1 into the two halves of a dword;
//   s      [N/16][K/128][16] fp32, one per row of the block;
//   z      [N/16][K/128][16] uint8.
// Quantisation (fp32, round-half-even): lo, hi = group min, max;
// s = (hi - lo) / 15 (a constant group: |hi|, or 1 when 0); z = clamp(rint(-lo/s), 0, 15);
// q = clamp(rint(w/s) + z, 0, 15).  The dequantised weight is (q - z) * s; the GEMMs
// never round it to bf16 (the decode GEMM scales each group's integer dot product,
// prefill multiplies a bf16 pair hi + lo that holds it to 16 bits).
__device__ __forceinline__ int q4_nibble(int e) { return (e >> 1) + 4 * (e & 1); }

struct Q4Ptrs {
  uint4* codes;
  float* s;
  uint8_t* z;
};

__host__ __device__ inline Q4Ptrs q4_ptrs(void* base, int rows, int cols) {
  char* b = (char*)base;
  const size_t nc = (size_t)rows * (size_t)cols / 2, ns = (size_t)rows * (size_t)(cols / 128);
  return Q4Ptrs{(uint4*)b, (float*)(b + nc), (uint8_t*)(b + nc + 4 * ns)};
}

// One wave per (16-row block, group): lane l generates its 32 values, the row's
// min and max come from the four lanes r, r + 16, r + 32, r + 48.
__global__ __launch_bounds__(256) void k_synth_q4(Q4Ptrs qp, WeightDesc w, uint64_t k0, uint64_t k1, uint64_t k2,
                                                  double std_) {
  const int lane = threadIdx.x & 63;
  const size_t item = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (nb, group)
  const int gbt = w.cols / 128;
  if (item >= (size_t)(w.rows / 16) * gbt) return;
  const int nb = (int)(item / gbt), gi = (int)(item % gbt);
  const int r = lane & 15, g = lane >> 4;
  int which, lrow;
  row_source(w, nb * 16 + r, &which, &lrow);
  const uint64_t key = which == 0 ? k0 : (which == 1 ? k1 : k2);
  float v[4][8];
  float lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 128 * gi + 32 * j + 8 * g + e;
      v[j][e] = weight_value(key, (uint64_t)lrow * (uint64_t)w.cols + (uint64_t)k, std_);
      lo = fminf(lo, v[j][e]);
      hi = fmaxf(hi, v[j][e]);
    }
  lo = fminf(lo, __shfl_xor(lo, 16, 64));
  lo = fminf(lo, __shfl_xor(lo, 32, 64));
  hi = fmaxf(hi, __shfl_xor(hi, 16, 64));
  hi = fmaxf(hi, __shfl_xor(hi, 32, 64));
  float sc = (hi - lo) / 15.0f;
  if (sc == 0.0f) sc = hi == 0.0f ? 1.0f : fabsf(hi);
  const float z = fminf(fmaxf(rintf(-lo / sc), 0.0f), 15.0f);
  uint32_t word[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t acc = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float q = fminf(fmaxf(rintf(v[j][e] / sc) + z, 0.0f), 15.0f);
      acc |= (uint32_t)q << (4 * q4_nibble(e));
    }
    word[j] = acc;
  }
  qp.codes[item * 64 + lane] = make_uint4(word[0], word[1], word[2], word[3]);
  if (g == 0) {
    qp.s[item * 16 + r] = sc;
    qp.z[item * 16 + r] = (uint8_t)z;
  }
}

// Code, scale and zero of physical element (prow, c).
__device__ __forceinline__ float q4_value(const Q4Ptrs& qp, int gbt, int prow, int c) {
  const size_t item = (size_t)(prow >> 4) * gbt + (size_t)(c >> 7);
  const int kk = c & 127, j = kk >> 5, g = (kk & 31) >> 3, e = kk & 7;
  const uint4 wd = qp.codes[item * 64 + (prow & 15) + 16 * g];
  const uint32_t word = j == 0 ? wd.x : (j == 1 ? wd.y : (j == 2 ? wd.z : wd.w));
  const uint32_t q = (word >> (4 * q4_nibble(e))) & 15u;
  const size_t sr = item * 16 + (prow & 15);
  return ((float)q - (float)qp.z[sr]) * qp.s[sr];
}

// Logical rows of one tensor of an int4 matrix, dequantised ((q - z) * s in fp32).
__global__ void k_export_q4(Q4Ptrs qp, WeightDesc w, int which, int rows, float* __restrict__ out) {
  const size_t n = (size_t)rows * (size_t)w.cols;
  const int gbt = w.cols / 128;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / (size_t)w.cols), c = (int)(i % (size_t)w.cols);
    int prow = r;
    if (w.fuse == FUSE_QKV) prow = which == 0 ? r : (which == 1 ? w.a + r : w.a + w.b + r);
    else if (w.fuse == FUSE_GU) prow = 2 * r + which;
    out[i] = q4_value(qp, gbt, prow, c);
  }
}

// int4 matrix -> two bf16 MFMA A-operand matrices in the weight fragment layout (wfrag), hi = bf16(w) and
// lo = bf16(w - hi) (w - hi is exact in fp32), for the batches the tile GEMM takes.
__global__ void k_dequant_q4(Q4Ptrs qp, int rows, int cols, uint4* __restrict__ hi, uint4* __restrict__ lo) {
  const int kbt = cols / 32, gbt = cols / 128;
  const size_t n = (size_t)(rows / 16) * kbt * 64;  // one fragment lane (8 values) per thread
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const size_t frag = i >> 6;
    const int kb = (int)(frag % kbt);
    const size_t nb = frag / kbt;
    const size_t item = nb * gbt + (size_t)(kb >> 2);
    const uint4 wd = qp.codes[item * 64 + lane];
    const int j = kb & 3;
    const uint32_t word = j == 0 ? wd.x : (j == 1 ? wd.y : (j == 2 ? wd.z : wd.w));
    const size_t sr = item * 16 + (lane & 15);
    const float sc = qp.s[sr], z = (float)qp.z[sr];
    uint32_t oh[4], ol[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t h2 = 0, l2 = 0;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float wv = ((float)((word >> (4 * q4_nibble(2 * t + u))) & 15u) - z) * sc;
        const uint16_t bh = f32_to_bf16(wv);
        const uint16_t bl = f32_to_bf16(wv - bf16_to_f32(bh));
        h2 |= (uint32_t)bh << (16 * u);
        l2 |= (uint32_t)bl << (16 * u);
      }
      oh[t] = h2;
      ol[t] = l2;
    }
    const size_t o = wfrag((int)nb, kb, rows / 16, kbt) * 64 + (size_t)lane;
    hi[o] = make_uint4(oh[0], oh[1], oh[2], oh[3]);
    lo[o] = make_uint4(ol[0], ol[1], ol[2], ol[3]);
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
      p = (wfrag(nb, kb, w.rows / 16, w.cols / 32) * 64 + (size_t)lane) * 8 + (size_t)(c & 7);
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

size_t q4_code_bytes(int rows, int cols) { return (size_t)rows * (size_t)cols / 2; }
size_t q4_sz_bytes(int rows, int cols) { return (size_t)rows * (size_t)(cols / 128) * 5; }

hipError_t launch_synth_q4(hipStream_t s, void* dst, const WeightDesc& w, uint64_t seed, double std_) {
  if (w.rows % 16 || w.cols % 128) return hipErrorInvalidValue;
  const size_t items = (size_t)(w.rows / 16) * (w.cols / 128);
  const uint64_t k0 = stream_key(seed, w.id0), k1 = stream_key(seed, w.id1), k2 = stream_key(seed, w.id2);
  hipLaunchKernelGGL(k_synth_q4, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s, q4_ptrs(dst, w.rows, w.cols), w,
                     k0, k1, k2, std_);
  return hipGetLastError();
}

hipError_t launch_export_q4(hipStream_t s, const void* src, const WeightDesc& w, int which, int rows, float* out) {
  const size_t n = (size_t)rows * (size_t)w.cols;
  hipLaunchKernelGGL(k_export_q4, dim3(grid_for(n, 256)), dim3(256), 0, s, q4_ptrs((void*)src, w.rows, w.cols), w,
                     which, rows, out);
  return hipGetLastError();
}

hipError_t launch_dequant_q4(hipStream_t s, const void* src, int rows, int cols, void* dst_hi, void* dst_lo) {
  if (rows % 16 || cols % 128) return hipErrorInvalidValue;
  const size_t n = (size_t)(rows / 16) * (cols / 32) * 64;
  hipLaunchKernelGGL(k_dequant_q4, dim3(grid_for(n, 256)), dim3(256), 0, s, q4_ptrs((void*)src, rows, cols), rows,
                     cols, (uint4*)dst_hi, (uint4*)dst_lo);
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
