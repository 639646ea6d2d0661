// Paged grouped-query attention over the KV cache, split over the context.
//
// One workgroup per (row, KV head, context split).  All query heads that share
// the KV head (n_heads / n_kv_heads of them) are served by the same workgroup,
// so every K/V tile is read from HBM once per row and reused from LDS by the
// whole group.  Scores use the 1/sqrt(hd) scale; the softmax is the online
// (running max / running sum) form, and each split leaves an unnormalised
// output with its (max, sum) for the combine kernel, which merges the splits
// by log-sum-exp weights in split order.
//
// Cache layout (per block of `blk` tokens): [block][layer][kv head][K|V][blk][hd].
// A row sees keys 0 .. pos (causal): pos is its position in the sequence.
#include "internal.h"

namespace rollout {
namespace {

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

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn(Dims D, const T* __restrict__ q, const T* __restrict__ kv, int n_blocks,
                                              const int32_t* __restrict__ tables, int max_blocks, RowMap rm,
                                              int splits, int split_tokens, int layer, float* __restrict__ opart,
                                              float* __restrict__ ml, int32_t* __restrict__ err) {
  constexpr int TT = 32;
  constexpr int NACC = 16 * HD / 256;
  __shared__ float qs[16][HD];
  __shared__ float ks[TT][HD + 1];
  __shared__ float vs[TT][HD + 1];
  __shared__ float sc[16][TT];
  __shared__ float m_s[16], l_s[16], a_s[16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x % splits;
  const int kvh = (blockIdx.x / splits) % D.nkv;
  const int r = blockIdx.x / (splits * D.nkv);
  int seq, pos;
  row_place(rm, r, &seq, &pos);
  const int ctx = pos + 1;
  const int nrep = D.nh / D.nkv;
  const int t_begin = split * split_tokens;
  const int t_end = min(ctx, t_begin + split_tokens);
  const float scale = 1.0f / sqrtf((float)HD);
  const size_t blk_elems = (size_t)D.blk * HD;

  for (int i = tid; i < nrep * HD; i += 256) qs[i / HD][i % HD] = ldf(q, (size_t)r * D.qd + (size_t)kvh * nrep * HD + i);
  if (tid < 16) {
    m_s[tid] = -INFINITY;
    l_s[tid] = 0.f;
  }
  float acc[NACC];
#pragma unroll
  for (int j = 0; j < NACC; ++j) acc[j] = 0.f;
  __syncthreads();

  for (int t0 = t_begin; t0 < t_end; t0 += TT) {
    const int nt = min(TT, t_end - t0);
    for (int i = tid; i < nt * HD; i += 256) {
      const int t = i / HD, dd = i - t * HD;
      const int tok = t0 + t;
      const int b = tables[(size_t)seq * max_blocks + tok / D.blk];
      float kval = 0.f, vval = 0.f;
      if (b >= 0 && b < n_blocks) {
        const size_t base = (((size_t)b * D.L + layer) * D.nkv + kvh) * 2 * blk_elems + (size_t)(tok % D.blk) * HD + dd;
        kval = ldf(kv, base);
        vval = ldf(kv, base + blk_elems);
      } else if (dd == 0) {
        atomicOr(err, 4);
      }
      ks[t][dd] = kval;
      vs[t][dd] = vval;
    }
    __syncthreads();
    for (int i = tid; i < nrep * TT; i += 256) {
      const int h = i / TT, t = i - h * TT;
      float s = -INFINITY;
      if (t < nt) {
        float dot = 0.f;
#pragma unroll 8
        for (int dd = 0; dd < HD; ++dd) dot += qs[h][dd] * ks[t][dd];
        s = dot * scale;
      }
      sc[h][t] = s;
    }
    __syncthreads();
    for (int h = wave; h < nrep; h += 4) {
      const float s = lane < TT ? sc[h][lane] : -INFINITY;
      const float mt = wave_max(s);
      const float mold = m_s[h];
      const float mnew = fmaxf(mold, mt);
      const float p = (lane < TT && s != -INFINITY) ? expf(s - mnew) : 0.f;
      const float lt = wave_sum(p);
      if (lane < TT) sc[h][lane] = p;
      if (lane == 0) {
        const float a = (mold == -INFINITY) ? 0.f : expf(mold - mnew);
        a_s[h] = a;
        l_s[h] = l_s[h] * a + lt;
        m_s[h] = mnew;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NACC; ++j) {
      const int idx = tid + 256 * j;
      const int h = idx / HD, dd = idx - h * HD;
      if (h < nrep) {
        float o = acc[j] * a_s[h];
        for (int t = 0; t < nt; ++t) o += sc[h][t] * vs[t][dd];
        acc[j] = o;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < NACC; ++j) {
    const int idx = tid + 256 * j;
    const int h = idx / HD, dd = idx - h * HD;
    if (h < nrep) opart[(((size_t)r * D.nh + kvh * nrep + h) * splits + split) * HD + dd] = acc[j];
  }
  if (tid < nrep) {
    const size_t o = (((size_t)r * D.nh + kvh * nrep + tid) * splits + split) * 2;
    ml[o] = m_s[tid];
    ml[o + 1] = l_s[tid];
  }
}

template <typename T>
__global__ void k_attn_combine(const float* __restrict__ opart, const float* __restrict__ ml, int splits, int hd,
                               T* __restrict__ out) {
  const size_t rh = blockIdx.x;  // row * n_heads + head
  const int d = threadIdx.x;
  float mx = -INFINITY;
  for (int s = 0; s < splits; ++s) {
    const float l = ml[(rh * splits + s) * 2 + 1];
    if (l > 0.f) mx = fmaxf(mx, ml[(rh * splits + s) * 2]);
  }
  float num = 0.f, den = 0.f;
  for (int s = 0; s < splits; ++s) {
    const float m = ml[(rh * splits + s) * 2], l = ml[(rh * splits + s) * 2 + 1];
    if (l > 0.f) {
      const float w = expf(m - mx);
      num += w * opart[(rh * splits + s) * hd + d];
      den += w * l;
    }
  }
  stf(out, rh * hd + d, den > 0.f ? num / den : 0.f);
}

}  // namespace

int attn_splits(int max_ctx, int* split_tokens) {
  const int st = 256;
  *split_tokens = st;
  const int s = (max_ctx + st - 1) / st;
  return s < 1 ? 1 : s;
}

hipError_t launch_attention(hipStream_t s, const Dims& D, const void* q, const void* kv_pool, int n_blocks,
                            const int32_t* tables, int max_blocks, RowMap rm, int R, int splits, int split_tokens,
                            int layer, float* opart, float* ml, int32_t* err) {
  if (R <= 0) return hipSuccess;
  const dim3 grid((unsigned)R * D.nkv * splits);
#define ROLLOUT_ATTN(T, HD)                                                                                   \
  hipLaunchKernelGGL((k_attn<T, HD>), grid, dim3(256), 0, s, D, (const T*)q, (const T*)kv_pool, n_blocks, tables, \
                     max_blocks, rm, splits, split_tokens, layer, opart, ml, err)
  if (D.dtype == ROLLOUT_DTYPE_BF16) {
    if (D.hd == 128) ROLLOUT_ATTN(uint16_t, 128);
    else if (D.hd == 64) ROLLOUT_ATTN(uint16_t, 64);
    else ROLLOUT_ATTN(uint16_t, 32);
  } else {
    if (D.hd == 128) ROLLOUT_ATTN(float, 128);
    else if (D.hd == 64) ROLLOUT_ATTN(float, 64);
    else ROLLOUT_ATTN(float, 32);
  }
#undef ROLLOUT_ATTN
  return hipGetLastError();
}

hipError_t launch_attn_combine(hipStream_t s, const Dims& D, const float* opart, const float* ml, int R, int splits,
                               void* out) {
  if (R <= 0) return hipSuccess;
  const dim3 grid((unsigned)R * D.nh);
  if (D.dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_attn_combine<uint16_t>, grid, dim3(D.hd), 0, s, opart, ml, splits, D.hd, (uint16_t*)out);
  else
    hipLaunchKernelGGL(k_attn_combine<float>, grid, dim3(D.hd), 0, s, opart, ml, splits, D.hd, (float*)out);
  return hipGetLastError();
}

}  // namespace rollout
