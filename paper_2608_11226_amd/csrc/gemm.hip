// Projection GEMMs: y[m][n] = sum_k X[m][k] * W[n][k], fp32 accumulation.
//
// bf16 path (CDNA4 MFMA, v_mfma_f32_16x16x32_bf16).  Both operands live in
// HBM in MFMA operand order, so every global load is a fully coalesced
// 16-byte-per-lane read:
//   W (A operand): tiles of 16 weight rows x 32 k, [N/16][K/32][64 lanes][8],
//                  lane = row%16 + 16*((k%32)/8) -- written once at synthesis;
//   X (B operand): tiles of 32 k x 16 activation rows, [K/32][M/16][64][8],
//                  lane = m%16 + 16*((k%32)/8) -- written by the producing
//                  kernel (norm, SwiGLU, attention).
// Weights are read exactly once per step, with non-temporal loads (keeping
// them out of the caches leaves room for the activations).
//
// k_gemm_ring (decode, M <= 64 rows): one wave per workgroup owns NBW
// 16-row weight blocks and one K split.  Weight and activation fragments
// stream through a D-deep register ring with no LDS and no barriers; every
// load is unconditional (addresses clamped into range, surplus steps masked at
// the MFMA), so the compiler keeps D - 1 ring stages in flight instead of
// draining the load queue at every step.  X is read from L2 by every wave,
// which costs M/(16 NBW) of the weight bytes in L2 traffic and nothing in HBM.
// With several K splits each writes a partial [split][M][N] that the consumer
// sums in split order.  The SwiGLU variant (gate/up, one split) finishes in
// registers: gate row i and up row i are adjacent weight rows, so the lane
// that holds one also holds the other, and h goes straight to the down
// projection's operand layout.
//
// k_gemm_bf16 (prefill and other batches above 64 rows): a workgroup of
// eight waves owns 128 weight rows (16 per wave) and a K range; it stages X
// through a double-buffered LDS slab shared by the eight waves (X is re-read
// from L2 once per 128 weight rows), while the weights and the next slab are
// in flight in registers; split partials as above.
//
// fp32 path: a plain LDS-tiled VALU GEMM over row-major X and W (the fp32
// path exists for exact parity on small models, not for speed).
#include <algorithm>
#include <cstdlib>

#include "internal.h"

namespace rollout {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// MB: 16-row blocks of X per workgroup pass; KS: k-steps (of 32) per staged X slab;
// WV: waves per workgroup (16 weight rows each).
template <int MB, int KS, int WV>
__global__ __launch_bounds__(WV * 64) void k_gemm_bf16(const bf16x8_t* __restrict__ XF, const bf16x8_t* __restrict__ W,
                                                       float* __restrict__ out, int M, int N, int K, int kslice) {
  constexpr int NTH = WV * 64;
  constexpr int XV = KS * MB * 64;  // 16-byte X vectors per slab
  constexpr int XPT = (XV + NTH - 1) / NTH;
  __shared__ bf16x8_t xs[2][XV];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nb = blockIdx.x * WV + wave;  // this wave's 16-row weight block
  const bool nvalid = nb * 16 < N;
  const int kbt = K >> 5;
  const int Mb = (M + 15) >> 4;
  const int kb0 = (int)(blockIdx.y * kslice) >> 5;
  const int kb1 = min(kbt, kb0 + (kslice >> 5));
  const int mb0 = blockIdx.z * MB;
  const bf16x8_t* wp = W + (size_t)(nvalid ? nb : 0) * (size_t)kbt * 64 + lane;

  bf16x8_t zero;
#pragma unroll
  for (int e = 0; e < 8; ++e) zero[e] = (__bf16)0.0f;
  floatx4_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  bf16x8_t wcur[KS], wnxt[KS], xr[XPT];
#define LOAD_W(dst, kb)                                               \
  _Pragma("unroll") for (int ks = 0; ks < KS; ++ks) dst[ks] =         \
      (nvalid && (kb) + ks < kb1) ? __builtin_nontemporal_load(wp + (size_t)((kb) + ks) * 64) : zero;
#define LOAD_X(kb)                                                                      \
  _Pragma("unroll") for (int j = 0; j < XPT; ++j) {                                     \
    const int v = tid + NTH * j;                                                        \
    bf16x8_t t = zero;                                                                  \
    if (v < XV) {                                                                       \
      const int ks = v / (MB * 64), mb = (v >> 6) % MB, ln = v & 63;                    \
      const int m = (mb0 + mb) * 16 + (ln & 15), kk = (kb) + ks;                        \
      if (kk < kb1 && m < M) t = XF[((size_t)kk * Mb + mb0 + mb) * 64 + ln];            \
    }                                                                                   \
    xr[j] = t;                                                                          \
  }
#define STORE_X(buf)                                                                    \
  _Pragma("unroll") for (int j = 0; j < XPT; ++j) {                                     \
    const int v = tid + NTH * j;                                                        \
    if (v < XV) xs[buf][v] = xr[j];                                                     \
  }

  LOAD_W(wcur, kb0);
  LOAD_X(kb0);
  STORE_X(0);
  __syncthreads();
  int buf = 0;
  for (int kb = kb0; kb < kb1; kb += KS) {
    const int kn = kb + KS;
    const bool more = kn < kb1;
    if (more) {
      LOAD_W(wnxt, kn);
      LOAD_X(kn);
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (kb + ks < kb1) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wcur[ks], xs[buf][(ks * MB + mb) * 64 + lane], acc[mb],
                                                            0, 0, 0);
      }
    }
    if (more) STORE_X(buf ^ 1);
    __syncthreads();
    buf ^= 1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) wcur[ks] = wnxt[ks];
  }
#undef LOAD_W
#undef LOAD_X
#undef STORE_X
  if (!nvalid) return;
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
  const int n = nb * 16 + 4 * (lane >> 4);
  float* o = out + (size_t)blockIdx.y * (size_t)M * (size_t)N;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = (mb0 + mb) * 16 + (lane & 15);
    if (m < M)
      *reinterpret_cast<float4*>(o + (size_t)m * N + n) = make_float4(acc[mb][0], acc[mb][1], acc[mb][2], acc[mb][3]);
  }
}

// MB = ceil(M/16) row blocks of X; NBW weight blocks per wave; D ring stages.
template <int MB, int NBW, int D, bool SWI>
__global__ __launch_bounds__(64) void k_gemm_ring(const bf16x8_t* __restrict__ XF, const bf16x8_t* __restrict__ W,
                                                  float* __restrict__ out, int M, int N, int K, int kslice,
                                                  uint16_t* __restrict__ h) {
  const int lane = threadIdx.x;
  const int nb0 = blockIdx.x * NBW;
  const int nbt = N >> 4, kbt = K >> 5;
  const int kb0 = (int)blockIdx.y * (kslice >> 5);
  const int nk = min(kbt, kb0 + (kslice >> 5)) - kb0;
  if (nk <= 0) {  // an empty K split contributes zeros
    if constexpr (!SWI) {
      for (int j = 0; j < NBW && nb0 + j < nbt; ++j)
        for (int m = lane & 15; m < M; m += 16)
          *reinterpret_cast<float4*>(out + ((size_t)blockIdx.y * M + m) * N + (nb0 + j) * 16 + 4 * (lane >> 4)) =
              make_float4(0.f, 0.f, 0.f, 0.f);
    }
    return;
  }
  floatx4_t acc[NBW][MB];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  {
    const bf16x8_t* wp[NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) wp[j] = W + ((size_t)min(nb0 + j, nbt - 1) * kbt + kb0) * 64 + lane;
    const bf16x8_t* xp = XF + (size_t)kb0 * MB * 64 + lane;
    bf16x8_t wr[D][NBW], xr[D][MB];
    // ring stage d holds k-step min(i, nk - 1); steps past nk reload the last one and are not used
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const size_t kk = (size_t)min(d, nk - 1);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) xr[d][mb] = xp[(kk * MB + mb) * 64];
#pragma unroll
      for (int j = 0; j < NBW; ++j) wr[d][j] = __builtin_nontemporal_load(wp[j] + kk * 64);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int i = 0; i < nk; i += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        if (i + d < nk) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < NBW; ++j)
              acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[d][j], xr[d][mb], acc[j][mb], 0, 0, 0);
        }
        const size_t kk = (size_t)min(i + d + D, nk - 1);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) xr[d][mb] = xp[(kk * MB + mb) * 64];
#pragma unroll
        for (int j = 0; j < NBW; ++j) wr[d][j] = __builtin_nontemporal_load(wp[j] + kk * 64);
        // keeps the ring order through scheduling, so each stage waits only for its own loads
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (nb0 + j >= nbt) continue;
    const int n = (nb0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = mb * 16 + (lane & 15);
      if (m >= M) continue;
      if constexpr (SWI) {
        // rows n, n+1 are (gate, up) of output f = n/2; rows n+2, n+3 of output f + 1
        const float g0 = acc[j][mb][0], u0 = acc[j][mb][1], g1 = acc[j][mb][2], u1 = acc[j][mb][3];
        const float h0 = g0 / (1.0f + expf(-g0)) * u0, h1 = g1 / (1.0f + expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(h + xoff(h, m, n >> 1, N >> 1, MB)) = pack_bf16x2(h0, h1);
      } else {
        float* o = out + (size_t)blockIdx.y * M * N;
        *reinterpret_cast<float4*>(o + (size_t)m * N + n) =
            make_float4(acc[j][mb][0], acc[j][mb][1], acc[j][mb][2], acc[j][mb][3]);
      }
    }
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

// m-blocks of 16 rows handled by one workgroup pass
int mb_for(int M) {
  const int mb = (M + 15) / 16;
  if (mb <= 4) return mb;
  if (mb <= 8) return 8;
  return 16;
}

int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  return v ? std::atoi(v) : dflt;
}

int kslice_for(int K, int splits) {
  const int per = (K + splits - 1) / splits;
  return (per + 31) / 32 * 32;
}

hipError_t launch_lds(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                      int splits) {
  constexpr int WV = kGemmTileRows / 16;
  const int mb = mb_for(M);
  const int kslice = kslice_for(K, splits);
  const int mchunks = ((M + 15) / 16 + mb - 1) / mb;
  const dim3 grid((N + kGemmTileRows - 1) / kGemmTileRows, splits, mchunks);
  const dim3 block(WV * 64);
  switch (mb) {
    case 1: hipLaunchKernelGGL((k_gemm_bf16<1, 8, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
    case 2: hipLaunchKernelGGL((k_gemm_bf16<2, 8, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
    case 3: hipLaunchKernelGGL((k_gemm_bf16<3, 4, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
    case 4: hipLaunchKernelGGL((k_gemm_bf16<4, 4, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
    case 8: hipLaunchKernelGGL((k_gemm_bf16<8, 4, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
    default: hipLaunchKernelGGL((k_gemm_bf16<16, 2, WV>), grid, block, 0, s, x, w, out, M, N, K, kslice); break;
  }
  return hipGetLastError();
}

// Ring kernel shape: weight blocks per wave and K splits, aiming at ~512 waves
// with K slices of at least 256 (gate/up with SwiGLU: 4 blocks, one split).
constexpr int kRingMaxRows = 64;
constexpr int kRingTargetWaves = 512;
int ring_splits(int N, int K, int max_splits) {
  const int groups = (N / 16 + 7) / 8;
  int s = (kRingTargetWaves + groups - 1) / groups;
  s = std::min(s, std::max(1, K / 256));
  s = std::max(1, std::min(s, max_splits));
  const int ks = kslice_for(K, s);
  return (K + ks - 1) / ks;
}

template <int NBW, bool SWI>
hipError_t launch_ring(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                       int splits, uint16_t* h) {
  const int kslice = kslice_for(K, splits);
  const dim3 grid((N / 16 + NBW - 1) / NBW, splits);
  switch ((M + 15) / 16) {
    case 1: hipLaunchKernelGGL((k_gemm_ring<1, NBW, 2, SWI>), grid, dim3(64), 0, s, x, w, out, M, N, K, kslice, h); break;
    case 2: hipLaunchKernelGGL((k_gemm_ring<2, NBW, 2, SWI>), grid, dim3(64), 0, s, x, w, out, M, N, K, kslice, h); break;
    case 3: hipLaunchKernelGGL((k_gemm_ring<3, NBW, 2, SWI>), grid, dim3(64), 0, s, x, w, out, M, N, K, kslice, h); break;
    default: hipLaunchKernelGGL((k_gemm_ring<4, NBW, 2, SWI>), grid, dim3(64), 0, s, x, w, out, M, N, K, kslice, h); break;
  }
  return hipGetLastError();
}

}  // namespace

int gemm_splits(int dtype, int M, int N, int K, int max_splits) {
  if (dtype != ROLLOUT_DTYPE_BF16 || max_splits <= 1) return 1;
  if (M <= kRingMaxRows) return ring_splits(N, K, max_splits);
  static const int target = env_int("ROLLOUT_GEMM_TARGET_WG", 768);
  static const int min_k = env_int("ROLLOUT_GEMM_MIN_KSLICE", 256);
  const int mb = mb_for(M);
  const int mchunks = ((M + 15) / 16 + mb - 1) / mb;
  const int nwg = (N + kGemmTileRows - 1) / kGemmTileRows * mchunks;
  int s = (target + nwg - 1) / nwg;
  s = std::min(s, std::max(1, K / min_k));
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
  if (N % 16 || K % 32) return hipErrorInvalidValue;
  const bf16x8_t* x = (const bf16x8_t*)X;
  const bf16x8_t* w = (const bf16x8_t*)W;
  if (M <= kRingMaxRows) return launch_ring<8, false>(s, x, w, out, M, N, K, splits, nullptr);
  return launch_lds(s, x, w, out, M, N, K, splits);
}

hipError_t launch_gemm_swiglu(hipStream_t s, const void* X, const void* W, int M, int N, int K, void* h) {
  if (M <= 0) return hipSuccess;
  if (M > kSwigluMaxRows || M > kRingMaxRows || N % 16 || K % 32) return hipErrorInvalidValue;
  return launch_ring<4, true>(s, (const bf16x8_t*)X, (const bf16x8_t*)W, nullptr, M, N, K, 1, (uint16_t*)h);
}

}  // namespace rollout
