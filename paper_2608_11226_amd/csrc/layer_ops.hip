// Row-wise kernels of the decoder layer: embedding gather, residual add +
// RMSNorm, the QKV epilogue (split-K sum, rotary embedding, paged-KV append),
// SwiGLU, and the per-step bookkeeping of a decode wave.
//
// Every kernel that consumes GEMM partials sums the K splits in split order,
// so the result does not depend on scheduling.  The residual stream is fp32;
// the outputs that feed a GEMM, and the cached K/V, are written in the cache
// dtype (bf16, rounded to nearest-even, on the bf16 path).
#include "internal.h"

namespace rollout {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void k_embed(const T* __restrict__ E, const int32_t* __restrict__ tokens,
                                               int tok_stride, const int32_t* __restrict__ col, int d, int V,
                                               float* __restrict__ x, int32_t* __restrict__ err) {
  const int m = blockIdx.x;
  const int c = col ? col[0] : 0;
  int tok = tokens[(size_t)m * tok_stride + c];
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0) atomicOr(err, 1);
    tok = 0;
  }
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)m * d + i] = ldf(E, (size_t)tok * d + i);
}

// x[m] += sum_s part[s][m]; out[m] = x[m] / sqrt(mean(x[m]^2) + eps) * gain
template <typename T>
__global__ __launch_bounds__(256) void k_residual_norm(const float* __restrict__ part, int splits, int M, int d,
                                                       float* __restrict__ x, const float* __restrict__ gain,
                                                       float eps, T* __restrict__ out) {
  __shared__ float red[32];
  const int m = blockIdx.x;
  float* xr = x + (size_t)m * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    float v = xr[i];
    if (part) {
      float acc = 0.f;
      for (int s = 0; s < splits; ++s) acc += part[((size_t)s * M + m) * d + i];
      v += acc;
      xr[i] = v;
    }
    ss += v * v;
  }
  const float tot = block_sum(ss, red);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += blockDim.x) stf(out, (size_t)m * d + i, xr[i] * r * gain[i]);
}

__device__ __forceinline__ void row_place(const RowMap& rm, int m, int* seq, int* pos, int* copies) {
  if (rm.P > 0) {
    const int p = m / rm.P;
    *pos = m - p * rm.P;
    *seq = rm.seq0 + p * rm.G;
    *copies = 1;
  } else {
    *seq = rm.seq0 + m;
    *pos = rm.ctx_len[m];
    *copies = 1;
  }
}

// One block per row: sum the K splits of [q | k | v], rotate q and k
// (rotate-half pairs (i, i + hd/2), angle table cos/sin[pos][i]), write q in
// the cache dtype and append k and v to the paged cache at the row's position.
template <typename T>
__global__ __launch_bounds__(256) void k_qkv_epilogue(Dims D, const float* __restrict__ part, int splits, int M,
                                                      RowMap rm, const float* __restrict__ rcos,
                                                      const float* __restrict__ rsin, T* __restrict__ q_out,
                                                      T* __restrict__ kv, int n_blocks,
                                                      const int32_t* __restrict__ tables, int max_blocks, int layer,
                                                      int32_t* __restrict__ err) {
  const int m = blockIdx.x;
  int seq, pos, copies;
  row_place(rm, m, &seq, &pos, &copies);
  const int hd = D.hd, half = hd / 2;
  // prefill rows in the last, partly filled prompt block go to every sequence of the group
  if (rm.P > 0 && (pos / D.blk) * D.blk + D.blk > rm.P) copies = rm.G;
  const int n = D.nqkv;
  const float* pr = part + (size_t)m * n;
  const size_t split_stride = (size_t)M * n;
  auto val = [&](int c) {
    float a = 0.f;
    for (int s = 0; s < splits; ++s) a += pr[s * split_stride + c];
    return a;
  };
  const float* cs = rcos + (size_t)pos * half;
  const float* sn = rsin + (size_t)pos * half;
  const int nrot = (D.nh + D.nkv) * half;  // rotated pairs of q and k heads
  const size_t blk_elems = (size_t)D.blk * hd;
  for (int j = threadIdx.x; j < nrot + D.kvd; j += blockDim.x) {
    if (j < nrot) {
      const int h = j / half, i = j - h * half;  // q heads first, then k heads
      const int c0 = h * hd + i;
      const float x1 = val(c0), x2 = val(c0 + half);
      const float o1 = x1 * cs[i] - x2 * sn[i];
      const float o2 = x2 * cs[i] + x1 * sn[i];
      if (h < D.nh) {
        stf(q_out, (size_t)m * D.qd + c0, o1);
        stf(q_out, (size_t)m * D.qd + c0 + half, o2);
      } else {
        const int kvh = h - D.nh;
        for (int c = 0; c < copies; ++c) {
          const int b = tables[(size_t)(seq + c) * max_blocks + pos / D.blk];
          if (b < 0 || b >= n_blocks) { atomicOr(err, 2); continue; }
          T* dst = kv + ((((size_t)b * D.L + layer) * D.nkv + kvh) * 2) * blk_elems + (size_t)(pos % D.blk) * hd;
          stf(dst, i, o1);
          stf(dst, i + half, o2);
        }
      }
    } else {
      const int jv = j - nrot;  // v element
      const int kvh = jv / hd, i = jv - kvh * hd;
      const float v = val(D.qd + D.kvd + jv);
      for (int c = 0; c < copies; ++c) {
        const int b = tables[(size_t)(seq + c) * max_blocks + pos / D.blk];
        if (b < 0 || b >= n_blocks) { atomicOr(err, 2); continue; }
        T* dst = kv + ((((size_t)b * D.L + layer) * D.nkv + kvh) * 2 + 1) * blk_elems + (size_t)(pos % D.blk) * hd;
        stf(dst, i, v);
      }
    }
  }
}

// h[m][f] = silu(g) * u, with gate/up columns interleaved in 16-column blocks
template <typename T>
__global__ __launch_bounds__(256) void k_swiglu(const float* __restrict__ part, int splits, int M, int ff,
                                                T* __restrict__ h) {
  const int m = blockIdx.x;
  const int n = 2 * ff;
  const size_t split_stride = (size_t)M * n;
  const float* pr = part + (size_t)m * n;
  for (int f = threadIdx.x; f < ff; f += blockDim.x) {
    const int cg = (f >> 4) * 32 + (f & 15);
    float g = 0.f, u = 0.f;
    for (int s = 0; s < splits; ++s) {
      g += pr[s * split_stride + cg];
      u += pr[s * split_stride + cg + 16];
    }
    const float sg = g / (1.0f + expf(-g));
    stf(h, (size_t)m * ff + f, sg * u);
  }
}

// dst[p*G + g] = src[p*P + P - 1] (last prompt position, replicated over the group)
template <typename T>
__global__ __launch_bounds__(256) void k_gather_rows(const T* __restrict__ src, int ld, int P, int G,
                                                     T* __restrict__ dst) {
  const int r = blockIdx.x;
  const int p = r / G;
  const T* s = src + ((size_t)p * P + P - 1) * ld;
  for (int i = threadIdx.x; i < ld; i += blockDim.x) dst[(size_t)r * ld + i] = s[i];
}

__global__ void k_advance(int32_t* __restrict__ ctx_len, int S, int32_t* __restrict__ cols) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (ctx_len && i < S) ctx_len[i] += 1;
  if (i == 0 && cols) {
    cols[0] += 1;
    cols[1] += 1;
  }
}

__global__ void k_set_cols(int32_t* cols, int c0, int c1) {
  if (threadIdx.x == 0) {
    cols[0] = c0;
    cols[1] = c1;
  }
}

}  // namespace

hipError_t launch_embed(hipStream_t s, int dtype, const void* E, const int32_t* tokens, int tok_stride,
                        const int32_t* col, int M, int d, int V, float* x, int32_t* err) {
  if (M <= 0) return hipSuccess;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_embed<uint16_t>, dim3(M), dim3(256), 0, s, (const uint16_t*)E, tokens, tok_stride, col, d,
                       V, x, err);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(M), dim3(256), 0, s, (const float*)E, tokens, tok_stride, col, d, V, x,
                       err);
  return hipGetLastError();
}

hipError_t launch_residual_norm(hipStream_t s, int dtype, const float* part, int splits, int M, int d, float* x,
                                const float* gain, float eps, void* out) {
  if (M <= 0) return hipSuccess;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_residual_norm<uint16_t>, dim3(M), dim3(256), 0, s, part, splits, M, d, x, gain, eps,
                       (uint16_t*)out);
  else
    hipLaunchKernelGGL(k_residual_norm<float>, dim3(M), dim3(256), 0, s, part, splits, M, d, x, gain, eps,
                       (float*)out);
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue(hipStream_t s, const Dims& D, const float* part, int splits, int M, RowMap rm,
                               const float* rope_cos, const float* rope_sin, void* q_out, void* kv_pool, int n_blocks,
                               const int32_t* tables, int max_blocks, int layer, int32_t* err) {
  if (M <= 0) return hipSuccess;
  if (D.dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_qkv_epilogue<uint16_t>, dim3(M), dim3(256), 0, s, D, part, splits, M, rm, rope_cos,
                       rope_sin, (uint16_t*)q_out, (uint16_t*)kv_pool, n_blocks, tables, max_blocks, layer, err);
  else
    hipLaunchKernelGGL(k_qkv_epilogue<float>, dim3(M), dim3(256), 0, s, D, part, splits, M, rm, rope_cos, rope_sin,
                       (float*)q_out, (float*)kv_pool, n_blocks, tables, max_blocks, layer, err);
  return hipGetLastError();
}

hipError_t launch_swiglu(hipStream_t s, int dtype, const float* part, int splits, int M, int ff, void* h) {
  if (M <= 0) return hipSuccess;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_swiglu<uint16_t>, dim3(M), dim3(256), 0, s, part, splits, M, ff, (uint16_t*)h);
  else
    hipLaunchKernelGGL(k_swiglu<float>, dim3(M), dim3(256), 0, s, part, splits, M, ff, (float*)h);
  return hipGetLastError();
}

hipError_t launch_gather_rows(hipStream_t s, int dtype, const void* src, int ld, int P, int G, int n_prompts,
                              void* dst) {
  if (n_prompts <= 0) return hipSuccess;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_gather_rows<uint16_t>, dim3(n_prompts * G), dim3(256), 0, s, (const uint16_t*)src, ld, P, G,
                       (uint16_t*)dst);
  else
    hipLaunchKernelGGL(k_gather_rows<float>, dim3(n_prompts * G), dim3(256), 0, s, (const float*)src, ld, P, G,
                       (float*)dst);
  return hipGetLastError();
}

hipError_t launch_advance(hipStream_t s, int32_t* ctx_len, int S, int32_t* cols) {
  hipLaunchKernelGGL(k_advance, dim3(S > 0 ? (S + 255) / 256 : 1), dim3(256), 0, s, ctx_len, S, cols);
  return hipGetLastError();
}

hipError_t launch_set_cols(hipStream_t s, int32_t* cols, int c0, int c1) {
  hipLaunchKernelGGL(k_set_cols, dim3(1), dim3(64), 0, s, cols, c0, c1);
  return hipGetLastError();
}

}  // namespace rollout
