// Row-wise kernels of the decoder layer: embedding gather, residual add +
// RMSNorm, the QKV epilogue (split-K sum, rotary embedding, paged-KV append),
// SwiGLU, and the per-step bookkeeping of a decode wave.
//
// Every kernel that consumes GEMM partials sums the K splits in split order,
// so the result does not depend on scheduling.  The residual stream is fp32;
// the outputs that feed a GEMM are written in the GEMM's operand layout
// (xoff) and, like the cached K/V, in the cache dtype (bf16 rounded to
// nearest-even on the bf16 path).
//
// KV pool layout (blk tokens per block): [layer][block][kv head][K: blk x hd | V: hd x blk];
// K is token-major, V is dimension-major so the attention kernel's P.V MFMA
// reads four consecutive tokens of one dimension as one 8-byte load.
#include <algorithm>

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

// x[m] += sum_s part[s][m]; out[m] = x[m] / sqrt(mean(x[m]^2) + eps) * gain  (GEMM operand layout)
template <typename T>
__global__ __launch_bounds__(1024) void k_residual_norm(const float* __restrict__ part, int splits, int M, int d,
                                                       float* __restrict__ x, const float* __restrict__ gain,
                                                       float eps, T* __restrict__ out) {
  __shared__ float red[32];
  const int m = blockIdx.x;
  const int Mb = (M + 15) >> 4;
  float* xr = x + (size_t)m * d;
  const int ng = d >> 3;
  float ss = 0.f;
  for (int g = threadIdx.x; g < ng; g += blockDim.x) {
    float v[8];
    ld8(xr, (size_t)g * 8, v);
    if (part) {
      float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll 4
      for (int s = 0; s < splits; ++s) {
        float p[8];
        ld8(part, ((size_t)s * M + m) * d + (size_t)g * 8, p);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += p[e];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += acc[e];
      st8(xr, (size_t)g * 8, v);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  const float tot = block_sum(ss, red);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  for (int g = threadIdx.x; g < ng; g += blockDim.x) {
    float v[8], gn[8];
    ld8(xr, (size_t)g * 8, v);
    ld8(gain, (size_t)g * 8, gn);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * gn[e];
    st8(out, xoff(out, m, g * 8, d, Mb), v);
  }
}

// The same for rows of at most 1024 groups of 8 columns (every model here): one thread per group keeps
// its eight values in registers from load to store, and its loads of x, the gain and up to MAXS split
// partials all go out at once (threads past the row repeat the last group's addresses and store nothing),
// so a row costs one memory round trip, the block reduction and the stores.
template <typename T, int MAXS>
__global__ __launch_bounds__(1024) void k_residual_norm_row(const float* __restrict__ part, int splits, int M, int d,
                                                            float* __restrict__ x, const float* __restrict__ gain,
                                                            float eps, T* __restrict__ out) {
  __shared__ float red[32];
  const int m = blockIdx.x;
  const int Mb = (M + 15) >> 4;
  const int ng = d >> 3;
  const bool act = (int)threadIdx.x < ng;
  const size_t c = (size_t)(act ? threadIdx.x : ng - 1) * 8;
  float* xr = x + (size_t)m * d;
  float v[8], gn[8];
  ld8(xr, c, v);
  ld8(gain, c, gn);
  if (part) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int s0 = 0; s0 < splits; s0 += MAXS) {
      float p[MAXS][8];
#pragma unroll
      for (int s = 0; s < MAXS; ++s) ld8(part, ((size_t)min(s0 + s, splits - 1) * M + m) * d + c, p[s]);
#pragma unroll
      for (int s = 0; s < MAXS; ++s)
        if (s0 + s < splits)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] += p[s][e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] += acc[e];
    if (act) st8(xr, c, v);
  }
  float ss = 0.f;
  if (act)
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  const float tot = block_sum(ss, red);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  if (act) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * gn[e];
    st8(out, xoff(out, m, (int)c, d, Mb), v);
  }
}

__device__ __forceinline__ void row_place(const RowMap& rm, int m, int* seq, int* pos) {
  if (rm.P > 0) {
    const int p = m / rm.P;
    *pos = m - p * rm.P;
    *seq = rm.seq0 + p * rm.G;
  } else {
    *seq = rm.seq0 + m;
    *pos = rm.ctx_len[m];
  }
}

// One wave per (row, head slot): slots [0, nh) are query heads, [nh, nh+nkv)
// key heads, [nh+nkv, nh+2nkv) value heads; slot s owns columns [s*hd, s*hd+hd)
// of the fused QKV output.  Query and key heads are rotated (rotate-half pairs
// (i, i + hd/2), angles cos/sin[pos][i]); keys and values are appended to the
// paged cache at the row's position.
template <typename T>
__global__ __launch_bounds__(64) void k_qkv_epilogue(Dims D, const float* __restrict__ part, int splits, int M,
                                                     RowMap rm, const float* __restrict__ rcos,
                                                     const float* __restrict__ rsin, T* __restrict__ q_out,
                                                     T* __restrict__ kv, int n_blocks,
                                                     const int32_t* __restrict__ tables, int max_blocks, int layer,
                                                     int32_t* __restrict__ err) {
  const int m = blockIdx.x, slot = blockIdx.y, tid = threadIdx.x;
  int seq, pos;
  row_place(rm, m, &seq, &pos);
  const int hd = D.hd, half = hd / 2;
  // prefill rows in the last, partly filled prompt block go to every sequence of the group
  const int copies = (rm.P > 0 && (pos / D.blk) * D.blk + D.blk > rm.P) ? rm.G : 1;
  const int n = D.nqkv;
  const size_t split_stride = (size_t)M * n;
  const float* pr = part + (size_t)m * n + (size_t)slot * hd;
  const size_t blk_elems = (size_t)D.blk * hd;
  const int kslot = slot - D.nh, vslot = slot - D.nh - D.nkv;
  if (vslot < 0) {
    const float* cs = rcos + (size_t)pos * half;
    const float* sn = rsin + (size_t)pos * half;
    for (int i = tid; i < half; i += 64) {
      float x1 = 0.f, x2 = 0.f;
      for (int s = 0; s < splits; ++s) {
        x1 += pr[s * split_stride + i];
        x2 += pr[s * split_stride + i + half];
      }
      const float o1 = x1 * cs[i] - x2 * sn[i];
      const float o2 = x2 * cs[i] + x1 * sn[i];
      if (kslot < 0) {
        stf(q_out, (size_t)m * D.qd + (size_t)slot * hd + i, o1);
        stf(q_out, (size_t)m * D.qd + (size_t)slot * hd + i + half, o2);
      } else {
        for (int c = 0; c < copies; ++c) {
          const int b = tables[(size_t)(seq + c) * max_blocks + pos / D.blk];
          if (b < 0 || b >= n_blocks) { atomicOr(err, 2); continue; }
          T* dst = kv + kv_offset(layer, b, kslot, n_blocks, D.nkv, 2 * blk_elems) + (size_t)(pos % D.blk) * hd;
          stf(dst, i, o1);
          stf(dst, i + half, o2);
        }
      }
    }
  } else {
    for (int i = tid; i < hd; i += 64) {
      float v = 0.f;
      for (int s = 0; s < splits; ++s) v += pr[s * split_stride + i];
      for (int c = 0; c < copies; ++c) {
        const int b = tables[(size_t)(seq + c) * max_blocks + pos / D.blk];
        if (b < 0 || b >= n_blocks) { atomicOr(err, 2); continue; }
        T* dst = kv + kv_offset(layer, b, vslot, n_blocks, D.nkv, 2 * blk_elems) + blk_elems + (size_t)i * D.blk +
                 (pos % D.blk);
        stf(dst, 0, v);
      }
    }
  }
}

// h[m][f] = silu(g) * u, gate column f at 2f and up column f at 2f + 1
template <typename T>
__global__ __launch_bounds__(256) void k_swiglu(const float* __restrict__ part, int splits, int M, int ff,
                                                T* __restrict__ h) {
  const int m = blockIdx.x;
  const int g = blockIdx.y * 256 + threadIdx.x;
  if (g >= (ff >> 3)) return;
  const int f = g * 8;
  const size_t n = 2 * (size_t)ff;
  float gu[16] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  for (int s = 0; s < splits; ++s) {
    float a[8], b[8];
    ld8(part, ((size_t)s * M + m) * n + 2 * f, a);
    ld8(part, ((size_t)s * M + m) * n + 2 * f + 8, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      gu[e] += a[e];
      gu[8 + e] += b[e];
    }
  }
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = gu[2 * e] / (1.0f + expf(-gu[2 * e])) * gu[2 * e + 1];
  st8(h, xoff(h, m, f, ff, (M + 15) >> 4), o);
}

// dst row p*G + g = src row p*P + P - 1 (last prompt position, replicated over the group), GEMM operand layout
template <typename T>
__global__ __launch_bounds__(256) void k_gather_rows(const T* __restrict__ src, int d, int P, int G, int M_src,
                                                     int M_dst, T* __restrict__ dst) {
  const int r = blockIdx.x;
  const int sr = (r / G) * P + P - 1;
  const int mb_s = (M_src + 15) >> 4, mb_d = (M_dst + 15) >> 4;
  for (int g = threadIdx.x; g < (d >> 3); g += blockDim.x) {
    float v[8];
    ld8(src, xoff(src, sr, g * 8, d, mb_s), v);
    st8(dst, xoff(dst, r, g * 8, d, mb_d), v);
  }
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

// Decode-step embedding fused with the first layer's RMSNorm: x[m] = E[token of row m] (fp32) and out[m] =
// rmsnorm(x[m]) * gain in the GEMM operand layout, with the arithmetic of k_residual_norm_row (same thread
// mapping and block sum), so the result is the embedding kernel followed by that norm.  One thread per group
// of 8 columns (d <= 8192); a token outside [0, V) sets err bit 1 and reads row 0.
template <typename T>
__global__ __launch_bounds__(1024) void k_embed_norm_row(const T* __restrict__ E, const int32_t* __restrict__ tokens,
                                                         int tok_stride, const int32_t* __restrict__ col, int M, int d,
                                                         int V, float* __restrict__ x, const float* __restrict__ gain,
                                                         float eps, T* __restrict__ out, int32_t* __restrict__ err) {
  __shared__ float red[32];
  const int m = blockIdx.x;
  const int Mb = (M + 15) >> 4;
  const int ng = d >> 3;
  const bool act = (int)threadIdx.x < ng;
  const size_t c = (size_t)(act ? threadIdx.x : ng - 1) * 8;
  int tok = tokens[(size_t)m * tok_stride + (col ? col[0] : 0)];
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0) atomicOr(err, 1);
    tok = 0;
  }
  float v[8], gn[8];
  ld8(E, (size_t)tok * d + c, v);
  ld8(gain, c, gn);
  if (act) st8(x + (size_t)m * d, c, v);
  float ss = 0.f;
  if (act)
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  const float tot = block_sum(ss, red);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  if (act) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * gn[e];
    st8(out, xoff(out, m, (int)c, d, Mb), v);
  }
}

hipError_t launch_embed_norm(hipStream_t s, int dtype, const void* E, const int32_t* tokens, int tok_stride,
                             const int32_t* col, int M, int d, int V, float* x, const float* gain, float eps, void* out,
                             int32_t* err) {
  if (M <= 0) return hipSuccess;
  const int ng = d >> 3;
  if (d % 8 || ng > 1024) return hipErrorInvalidValue;
  const int threads = (ng + 63) / 64 * 64;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_embed_norm_row<uint16_t>, dim3(M), dim3(threads), 0, s, (const uint16_t*)E, tokens,
                       tok_stride, col, M, d, V, x, gain, eps, (uint16_t*)out, err);
  else
    hipLaunchKernelGGL(k_embed_norm_row<float>, dim3(M), dim3(threads), 0, s, (const float*)E, tokens, tok_stride,
                       col, M, d, V, x, gain, eps, (float*)out, err);
  return hipGetLastError();
}

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
  const int ng = d >> 3;
  // one thread per group of 8 columns (up to 1024 threads per row)
  const int threads = std::min(1024, (ng + 63) / 64 * 64);
  if (ng <= 1024) {
    const bool bf = dtype == ROLLOUT_DTYPE_BF16;
#define ROLLOUT_NORM_ROW(S)                                                                                           \
  do {                                                                                                                \
    if (bf)                                                                                                           \
      hipLaunchKernelGGL((k_residual_norm_row<uint16_t, S>), dim3(M), dim3(threads), 0, s, part, splits, M, d, x,    \
                         gain, eps, (uint16_t*)out);                                                                  \
    else                                                                                                              \
      hipLaunchKernelGGL((k_residual_norm_row<float, S>), dim3(M), dim3(threads), 0, s, part, splits, M, d, x, gain, \
                         eps, (float*)out);                                                                           \
  } while (0)
    if (!part || splits <= 1) ROLLOUT_NORM_ROW(1);
    else if (splits <= 2) ROLLOUT_NORM_ROW(2);
    else if (splits <= 4) ROLLOUT_NORM_ROW(4);
    else ROLLOUT_NORM_ROW(8);
#undef ROLLOUT_NORM_ROW
    return hipGetLastError();
  }
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_residual_norm<uint16_t>, dim3(M), dim3(threads), 0, s, part, splits, M, d, x, gain, eps,
                       (uint16_t*)out);
  else
    hipLaunchKernelGGL(k_residual_norm<float>, dim3(M), dim3(threads), 0, s, part, splits, M, d, x, gain, eps,
                       (float*)out);
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue(hipStream_t s, const Dims& D, const float* part, int splits, int M, RowMap rm,
                               const float* rope_cos, const float* rope_sin, void* q_out, void* kv_pool, int n_blocks,
                               const int32_t* tables, int max_blocks, int layer, int32_t* err) {
  if (M <= 0) return hipSuccess;
  const dim3 grid(M, D.nh + 2 * D.nkv);
  if (D.dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_qkv_epilogue<uint16_t>, grid, dim3(64), 0, s, D, part, splits, M, rm, rope_cos, rope_sin,
                       (uint16_t*)q_out, (uint16_t*)kv_pool, n_blocks, tables, max_blocks, layer, err);
  else
    hipLaunchKernelGGL(k_qkv_epilogue<float>, grid, dim3(64), 0, s, D, part, splits, M, rm, rope_cos, rope_sin,
                       (float*)q_out, (float*)kv_pool, n_blocks, tables, max_blocks, layer, err);
  return hipGetLastError();
}

hipError_t launch_swiglu(hipStream_t s, int dtype, const float* part, int splits, int M, int ff, void* h) {
  if (M <= 0) return hipSuccess;
  const dim3 grid(M, ((ff >> 3) + 255) / 256);
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_swiglu<uint16_t>, grid, dim3(256), 0, s, part, splits, M, ff, (uint16_t*)h);
  else
    hipLaunchKernelGGL(k_swiglu<float>, grid, dim3(256), 0, s, part, splits, M, ff, (float*)h);
  return hipGetLastError();
}

// one workgroup per layer copies block src's 16-byte words to block dst
__global__ __launch_bounds__(256) void k_copy_kv_block(uint4* __restrict__ kv, size_t block_words, int n_blocks, int src,
                                                       int dst) {
  const size_t base = (size_t)blockIdx.x * n_blocks * block_words;
  const uint4* from = kv + base + (size_t)src * block_words;
  uint4* to = kv + base + (size_t)dst * block_words;
  for (size_t i = threadIdx.x; i < block_words; i += blockDim.x) to[i] = from[i];
}

hipError_t launch_copy_kv_block(hipStream_t s, void* kv_pool, int n_blocks, int L, size_t bytes_per_layer, int src,
                                int dst) {
  if (L <= 0 || bytes_per_layer % 16 || src < 0 || src >= n_blocks || dst < 0 || dst >= n_blocks)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_copy_kv_block, dim3(L), dim3(256), 0, s, (uint4*)kv_pool, bytes_per_layer / 16, n_blocks, src,
                     dst);
  return hipGetLastError();
}

hipError_t launch_gather_rows(hipStream_t s, int dtype, const void* src, int d, int P, int G, int n_prompts,
                              void* dst) {
  if (n_prompts <= 0) return hipSuccess;
  const int M_src = n_prompts * P, M_dst = n_prompts * G;
  if (dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_gather_rows<uint16_t>, dim3(M_dst), dim3(256), 0, s, (const uint16_t*)src, d, P, G, M_src,
                       M_dst, (uint16_t*)dst);
  else
    hipLaunchKernelGGL(k_gather_rows<float>, dim3(M_dst), dim3(256), 0, s, (const float*)src, d, P, G, M_src, M_dst,
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
