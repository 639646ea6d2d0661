// Projection GEMMs: out[split][m][n] = sum_{k in split} X[m][k] * W[n][k], fp32 result.
//
// bf16 path (CDNA4 MFMA, v_mfma_f32_16x16x32_bf16).  The weight matrix is the
// MFMA A operand: it is stored pre-tiled in operand order (16 rows x 32 k per
// 1 KiB tile, lane-major), so one wave reads one tile with a single fully
// coalesced 16-byte-per-lane load and weights stream from HBM exactly once.
// The activations X (bf16, row-major) are the B operand; each workgroup stages
// a [M_tile x KC] slab of X in LDS, in operand order, and its four waves (one
// 16-row weight block each) reuse it.  Weights for the next K chunk are loaded
// into registers while the MFMAs of the current chunk run.  Small-N
// projections are split over K so a launch has enough workgroups to keep every
// CU streaming; the split partials are summed in a fixed order by the
// epilogue kernels, so results are deterministic.
//
// fp32 path: a plain LDS-tiled VALU GEMM (the fp32 path exists for exact
// parity on small models, not for speed).
#include "internal.h"

#include <algorithm>

namespace rollout {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

template <int MB, int KC>
__global__ __launch_bounds__(256) void k_gemm_bf16(const uint16_t* __restrict__ X, int ldx,
                                                   const uint16_t* __restrict__ W, float* __restrict__ out, int M,
                                                   int N, int K, int kslice) {
  constexpr int KS = KC / 32;
  __shared__ bf16x8_t xs[KS][MB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nb = blockIdx.x * 4 + wave;
  const bool nvalid = nb * 16 < N;
  const int kbt = K / 32;
  const int k0 = blockIdx.y * kslice;
  const int k1 = min(K, k0 + kslice);
  const int m0 = blockIdx.z * (MB * 16);
  const bf16x8_t* wp = reinterpret_cast<const bf16x8_t*>(W) + (size_t)(nvalid ? nb : 0) * (size_t)kbt * 64 + lane;

  bf16x8_t zero;
#pragma unroll
  for (int e = 0; e < 8; ++e) zero[e] = (__bf16)0.0f;

  floatx4_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  bf16x8_t wcur[KS], wnxt[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    wcur[ks] = (nvalid && k0 + ks * 32 < k1) ? wp[(size_t)(k0 / 32 + ks) * 64] : zero;
    wnxt[ks] = zero;
  }

  for (int kc = k0; kc < k1; kc += KC) {
    const int nks = min(KS, (k1 - kc) / 32);
    // stage X[m0 .. m0 + 16 MB) x [kc, kc + 32 nks) into LDS in B-operand order
    const int items = MB * 16 * nks * 4;
    for (int it = threadIdx.x; it < items; it += 256) {
      const int kq = it & 3;
      const int rest = it >> 2;
      const int ks = rest % nks;
      const int ml = rest / nks;
      const int m = m0 + ml;
      bf16x8_t v = zero;
      if (m < M) v = *reinterpret_cast<const bf16x8_t*>(X + (size_t)m * ldx + kc + ks * 32 + kq * 8);
      xs[ks][ml >> 4][(ml & 15) + 16 * kq] = v;
    }
    __syncthreads();
    const int kn = kc + KC;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      if (nvalid && kn + ks * 32 < k1) wnxt[ks] = wp[(size_t)(kn / 32 + ks) * 64];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks < nks) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wcur[ks], xs[ks][mb][lane], acc[mb], 0, 0, 0);
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) wcur[ks] = wnxt[ks];
  }
  if (!nvalid) return;
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
  float* o = out + (size_t)blockIdx.y * (size_t)M * (size_t)N;
  const int n = nb * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 16 + (lane & 15);
    if (m < M)
      *reinterpret_cast<float4*>(o + (size_t)m * N + n) = make_float4(acc[mb][0], acc[mb][1], acc[mb][2], acc[mb][3]);
  }
}

__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ X, int ldx, const float* __restrict__ W,
                                                  float* __restrict__ out, int M, int N, int K) {
  __shared__ float xs[16][33];
  __shared__ float ws[16][33];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int n0 = blockIdx.x * 16, m0 = blockIdx.y * 16;
  float acc = 0.f;
  for (int k0 = 0; k0 < K; k0 += 32) {
    for (int i = threadIdx.x; i < 512; i += 256) {
      const int r = i >> 5, c = i & 31;
      const int k = k0 + c;
      xs[r][c] = (m0 + r < M && k < K) ? X[(size_t)(m0 + r) * ldx + k] : 0.f;
      ws[r][c] = (n0 + r < N && k < K) ? W[(size_t)(n0 + r) * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 32; ++c) acc += xs[ty][c] * ws[tx][c];
    __syncthreads();
  }
  const int m = m0 + ty, n = n0 + tx;
  if (m < M && n < N) out[(size_t)m * N + n] = acc;
}

int mb_for(int M) {
  if (M <= 16) return 1;
  if (M <= 32) return 2;
  if (M <= 64) return 4;
  if (M <= 128) return 8;
  return 16;
}

int kslice_for(int K, int splits) {
  const int per = (K + splits - 1) / splits;
  return (per + 31) / 32 * 32;
}

}  // namespace

int gemm_splits(int dtype, int M, int N, int K, int max_splits) {
  if (dtype != ROLLOUT_DTYPE_BF16 || max_splits <= 1) return 1;
  const int mb = mb_for(M);
  const int mchunks = (M + mb * 16 - 1) / (mb * 16);
  const int nwg = (N + 63) / 64 * mchunks;
  const int target = 1024;  // about four workgroups per CU
  int s = (target + nwg - 1) / nwg;
  s = std::min(s, std::max(1, K / 256));
  s = std::min(s, max_splits);
  s = std::max(s, 1);
  const int ks = kslice_for(K, s);
  return (K + ks - 1) / ks;
}

hipError_t launch_gemm(hipStream_t s, int dtype, const void* X, int ldx, const void* W, float* out, int M, int N,
                       int K, int splits) {
  if (M <= 0) return hipSuccess;
  if (dtype != ROLLOUT_DTYPE_BF16) {
    dim3 grid((N + 15) / 16, (M + 15) / 16);
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, s, (const float*)X, ldx, (const float*)W, out, M, N, K);
    return hipGetLastError();
  }
  const int mb = mb_for(M);
  const int kslice = kslice_for(K, splits);
  dim3 grid((N + 63) / 64, splits, (M + mb * 16 - 1) / (mb * 16));
  const uint16_t* x = (const uint16_t*)X;
  const uint16_t* w = (const uint16_t*)W;
  switch (mb) {
    case 1: hipLaunchKernelGGL((k_gemm_bf16<1, 256>), grid, dim3(256), 0, s, x, ldx, w, out, M, N, K, kslice); break;
    case 2: hipLaunchKernelGGL((k_gemm_bf16<2, 256>), grid, dim3(256), 0, s, x, ldx, w, out, M, N, K, kslice); break;
    case 4: hipLaunchKernelGGL((k_gemm_bf16<4, 256>), grid, dim3(256), 0, s, x, ldx, w, out, M, N, K, kslice); break;
    case 8: hipLaunchKernelGGL((k_gemm_bf16<8, 256>), grid, dim3(256), 0, s, x, ldx, w, out, M, N, K, kslice); break;
    default: hipLaunchKernelGGL((k_gemm_bf16<16, 128>), grid, dim3(256), 0, s, x, ldx, w, out, M, N, K, kslice); break;
  }
  return hipGetLastError();
}

}  // namespace rollout
