// Internal declarations shared by the kernels and the host runtime of librollout.
// Not part of the public ABI (that is include/rollout.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "rollout.h"

namespace rollout {

// ---------------------------------------------------------------------------
// Model dimensions as the kernels see them.
// ---------------------------------------------------------------------------
struct Dims {
  int L, d, nh, nkv, hd, ff, V;
  int qd, kvd, nqkv;  // nh*hd, nkv*hd, qd + 2*kvd
  float eps, theta;
  int dtype;          // ROLLOUT_DTYPE_FP32 or _BF16: activations, cache, embedding and LM head
  bool wq4;           // layer projections stored as int4 groups (ROLLOUT_DTYPE_INT4; dtype is then BF16)
  int blk;            // tokens per KV block
  int max_ctx;        // max prompt + max new tokens
};

// Bytes of one cache element and one weight element.
inline size_t elem_bytes(int dtype) { return dtype == ROLLOUT_DTYPE_BF16 ? 2 : 4; }

// Physical layout of a weight matrix.
enum WLayout : int {
  W_ROWMAJOR = 0,  // [rows][cols]
  W_TILED = 1,     // MFMA operand fragments, four 16-row blocks interleaved per k-step (wfrag)
};

// How physical rows of a (possibly fused) matrix map to synthesis tensor ids.
enum WFuse : int {
  FUSE_NONE = 0,  // one tensor: id0, row = physical row
  FUSE_QKV = 1,   // rows [0,a) id0, [a,a+b) id1, [a+b,a+2b) id2
  FUSE_GU = 2,    // rows alternate id0 (gate row i at 2i) and id1 (up row i at 2i + 1)
};

struct WeightDesc {
  int rows, cols;
  int layout;  // WLayout
  int fuse;    // WFuse
  int id0, id1, id2;
  int a, b;    // FUSE_QKV split sizes (q rows, kv rows)
};

// Where each activation row of a prefill or decode pass lives in the cache.
//   decode  (P == 0): row m is sequence seq0 + m at position ctx_len[m].
//   prefill (P > 0):  row m is token t = m % P of prompt m / P; it belongs to
//                     sequence seq0 + (m / P) * G at position t, and its K/V go
//                     to all G sequences of the group when t lies in the last,
//                     partially filled prompt block (shared blocks otherwise).
struct RowMap {
  const int32_t* ctx_len;
  int P, G, seq0;
};

// ---------------------------------------------------------------------------
// Launchers (each enqueues on the given stream and returns hipGetLastError()).
// ---------------------------------------------------------------------------
hipError_t launch_synth(hipStream_t s, void* dst, int dtype, const WeightDesc& w, uint64_t seed, double std_);
hipError_t launch_fill(hipStream_t s, float* dst, size_t n, float value);
// int4 weight-only matrices (layer projections of the int4 model): packed codes, then fp32 scales,
// then uint8 zero points, q4_code_bytes + q4_sz_bytes in all; rows a multiple of 16, cols of 128.
// The code, scale and zero arrays start at byte offsets 0, rows*cols/2 and rows*cols/2 + 4*rows*cols/128.
size_t q4_code_bytes(int rows, int cols);
size_t q4_sz_bytes(int rows, int cols);
hipError_t launch_synth_q4(hipStream_t s, void* dst, const WeightDesc& w, uint64_t seed, double std_);
hipError_t launch_export_q4(hipStream_t s, const void* src, const WeightDesc& w, int which, int rows, float* out);
// bf16 MFMA-operand tiles hi = bf16(w), lo = bf16(w - hi) of an int4 matrix (each rows * cols bf16)
hipError_t launch_dequant_q4(hipStream_t s, const void* src, int rows, int cols, void* dst_hi, void* dst_lo);
hipError_t launch_export(hipStream_t s, const void* src, int dtype, const WeightDesc& w, int which, int rows,
                         float* out);

// out[split][m][n] = sum over the split's k range of X[m][k] * W[n][k] (fp32).
int gemm_splits(int dtype, int M, int N, int K, int max_splits);
hipError_t launch_gemm(hipStream_t s, int dtype, const void* X, int ldx, const void* W, float* out, int M,
                       int N, int K, int splits);

// Gate/up projection with SwiGLU applied to its own output (bf16, one K split;
// the ring kernel up to 64 rows, the tile kernel above): W holds gate row i at
// physical row 2i and up row i at 2i + 1; h[m][i] = silu(gate) * up in the down
// projection's operand layout.  int4 weights: the int4 ring, M <= kSwigluMaxRows.
constexpr int kSwigluMaxRows = 64;
hipError_t launch_gemm_swiglu(hipStream_t s, const void* X, const void* W, int M, int N, int K, void* h);
// The same two GEMMs over an int4 weight matrix (M <= 64; K a multiple of 128; partial splits as above).
int gemm_splits_q4(int M, int N, int K, int max_splits);
hipError_t launch_gemm_q4(hipStream_t s, const void* X, const void* W, float* out, int M, int N, int K, int splits);
hipError_t launch_gemm_swiglu_q4(hipStream_t s, const void* X, const void* W, int M, int N, int K, void* h);

hipError_t launch_embed(hipStream_t s, int dtype, const void* E, const int32_t* tokens, int tok_stride,
                        const int32_t* col, int M, int d, int V, float* x, int32_t* err);
// x[m] = E[token m] and out[m] = rmsnorm(x[m]) * gain in one kernel (d <= 8192, else hipErrorInvalidValue and
// nothing enqueued); the same values as launch_embed followed by launch_residual_norm with part NULL.
hipError_t launch_embed_norm(hipStream_t s, int dtype, const void* E, const int32_t* tokens, int tok_stride,
                             const int32_t* col, int M, int d, int V, float* x, const float* gain, float eps, void* out,
                             int32_t* err);
// x[m] += sum_s part[s][m] (part may be NULL); out[m] = rmsnorm(x[m]) * gain in the cache dtype.
hipError_t launch_residual_norm(hipStream_t s, int dtype, const float* part, int splits, int M, int d, float* x,
                                const float* gain, float eps, void* out);
hipError_t launch_qkv_epilogue(hipStream_t s, const Dims& D, const float* part, int splits, int M, RowMap rm,
                               const float* rope_cos, const float* rope_sin, void* q_out, void* kv_pool,
                               int n_blocks, const int32_t* tables, int max_blocks, int layer, int32_t* err);
hipError_t launch_swiglu(hipStream_t s, int dtype, const float* part, int splits, int M, int ff, void* h);
// Attention of R rows over the cache, written to out in the O-projection operand
// layout.  Paths that split the context use opart/ml (R x n_heads x splits) as scratch.
// With qkv_part (decode rows, attention_forms_qkv(D) only) the kernel forms q,
// k and v from the QKV projection's split partials itself (rotary embedding,
// cache append) instead of reading q and expecting the cache to hold the row's token.
int attn_splits(int max_ctx, int* split_tokens);
bool attention_forms_qkv(const Dims& D);
hipError_t launch_attention(hipStream_t s, const Dims& D, const void* q, void* kv_pool, int n_blocks,
                            const int32_t* tables, int max_blocks, RowMap rm, int R, int splits, int split_tokens,
                            int layer, float* opart, float* ml, void* out, int32_t* err, const float* qkv_part,
                            int qkv_splits, const float* rope_cos, const float* rope_sin);
// Decode attention with the group's shared prompt read once per group: a suffix pass over each row's own
// keys (p_shared .. pos; q/k/v formed from the QKV split partials as above, rotated q kept in q_keep,
// softmax state in st_o [R][nh][hd] / st_ml [R][nh][2]) and a prefix pass over the shared blocks that
// merges the state and writes out.  Rows are R / G whole groups in sequence order from rm.seq0.
bool attention_shares_prefix(const Dims& D);
hipError_t launch_attention_shared(hipStream_t s, const Dims& D, void* kv_pool, int n_blocks, const int32_t* tables,
                                   int max_blocks, RowMap rm, int R, int layer, int G, int p_shared, void* q_keep,
                                   float* st_o, float* st_ml, void* out, int32_t* err, const float* qkv_part,
                                   int qkv_splits, const float* rope_cos, const float* rope_sin);
// copies block src to block dst in every layer of the pool (n_blocks blocks, bytes_per_layer per block and
// layer: all KV heads, K and V), for a sequence that starts from a copy of a shared partial block
hipError_t launch_copy_kv_block(hipStream_t s, void* kv_pool, int n_blocks, int L, size_t bytes_per_layer, int src,
                                int dst);
hipError_t launch_gather_rows(hipStream_t s, int dtype, const void* src, int ld, int P, int G, int n_prompts,
                              void* dst);
hipError_t launch_advance(hipStream_t s, int32_t* ctx_len, int S, int32_t* cols);
// Continuous batching (batching.hip): per-slot completion index, next token column, ended flag, the
// slot's last draw and its staged uniform; all [S] in the arena.
struct CbState {
  int32_t* seq;
  int32_t* col;
  int32_t* done;
  int32_t* draw;
  float* u_slot;
};
hipError_t launch_stop_bitmap(hipStream_t s, uint32_t* bitmap, int V, const int32_t* ids, int n, int32_t* err);
hipError_t launch_cb_reset(hipStream_t s, int S, const CbState& cb);
hipError_t launch_cb_admit(hipStream_t s, const CbState& cb, int r0, int G, int seq0, int P, int N,
                           int32_t* ctx_len, int32_t* tokens_out);
hipError_t launch_cb_commit(hipStream_t s, const CbState& cb, int r0, int r1, int N, const uint32_t* stop,
                            const float* u, int32_t* ctx_len, int32_t* tokens_out, int32_t* lengths, bool advance);
hipError_t launch_length_rewards(hipStream_t s, const int32_t* lengths, int n, int target, float* rewards,
                                 long long* total);
hipError_t launch_seq_table(hipStream_t s, int32_t* tables, int max_blocks, int row, int rec, int n_shared,
                            bool has_partial, int own, int n_own);
hipError_t launch_seq_admit(hipStream_t s, const CbState& cb, int r, int seq_id, int P, int N, int32_t* ctx_len,
                            int32_t* tokens_out);
hipError_t launch_set_cols(hipStream_t s, int32_t* cols, int c0, int c1);
// Sampler scratch: stored e values of S rows plus per-chunk statistics.
size_t sample_scratch_bytes(int S, int V);
// largest row count whose sampler scratch fits in `bytes` (0 if not even one row does)
int sample_rows_fitting(size_t bytes, int V);
// sets the message rollout_last_error(NULL) returns on the calling thread
void set_last_error(const std::string& msg);
hipError_t launch_sample(hipStream_t s, const float* logits, int S, int V, float temperature, float top_p,
                         const float* u, int u_stride, const int32_t* col, int32_t* out, int out_stride,
                         void* scratch);
hipError_t launch_grpo(hipStream_t s, const float* r, int n_groups, int G, float eps, int ddof, float* adv,
                       int32_t* zero_var);

}  // namespace rollout

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
#ifdef __HIPCC__
namespace rollout {

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float ldf(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ldf(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void stf(float* p, size_t i, float v) { p[i] = v; }
__device__ __forceinline__ void stf(uint16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }

// bf16 weight matrices (the GEMMs' A operand) are stored as fragments of 16
// rows x 32 k (64 lanes x 8 values, lane = row%16 + 16*((k%32)/8)).  The
// fragments of four consecutive 16-row blocks at one k-step are adjacent,
// [ceil(N/64)][K/32][4][64][8] (a last group of r < 4 blocks holds r per
// k-step), so a wave that owns four blocks reads one contiguous 4 KB run per
// k-step.  wfrag: fragment index of block nb at k-step kb (nbt = N/16 blocks,
// kbt = K/32 k-steps); the fragment's 64 lanes follow it.
__host__ __device__ __forceinline__ int wgroup_blocks(int nb, int nbt) {
  const int r = nbt - (nb & ~3);
  return r < 4 ? r : 4;
}
__host__ __device__ __forceinline__ size_t wfrag(int nb, int kb, int nbt, int kbt) {
  return (size_t)(nb >> 2) * (size_t)kbt * 4 + (size_t)kb * (size_t)wgroup_blocks(nb, nbt) + (size_t)(nb & 3);
}
__host__ __device__ __forceinline__ void wfrag_inv(size_t t, int nbt, int kbt, int* nb, int* kb) {
  const size_t per = (size_t)kbt * 4;
  const int g = (int)(t / per);
  const int rem = (int)(t - (size_t)g * per);
  const int r = wgroup_blocks(4 * g, nbt);
  *kb = rem / r;
  *nb = 4 * g + rem % r;
}

// Element (m, k) of an M x K GEMM activation operand.  bf16 operands are kept
// in MFMA B-operand order, tiles of 32 k x 16 rows: [K/32][Mb][64 lanes][8],
// lane = m%16 + 16*((k%32)/8), Mb = ceil(M/16); fp32 operands are row-major.
// Eight consecutive k starting at a multiple of 8 are contiguous in both.
// KV pool layout: [layer][block][KV head][K: blk x hd | V: hd x blk] (elements).  One layer's blocks are
// contiguous, so the blocks a decode step's attention reads for one layer span the pool's 1/L share and
// not all of it (fewer address-translation pages per layer: 7B attention KV loop -8%).  head_elems is
// 2 * blk * hd; the offset is that of (layer, block, KV head).
__host__ __device__ __forceinline__ size_t kv_offset(int layer, int block, int kvh, int n_blocks, int nkv,
                                                     size_t head_elems) {
  return (((size_t)layer * n_blocks + block) * nkv + kvh) * head_elems;
}

__device__ __forceinline__ size_t xoff(const uint16_t*, int m, int k, int K, int Mb) {
  (void)K;
  return ((size_t)((k >> 5) * Mb + (m >> 4)) * 64 + (size_t)((m & 15) + ((k & 31) >> 3) * 16)) * 8 + (k & 7);
}
__device__ __forceinline__ size_t xoff(const float*, int m, int k, int K, int Mb) {
  (void)Mb;
  return (size_t)m * K + k;
}

// Eight consecutive values at element index i (i a multiple of 8).
__device__ __forceinline__ void st8(float* p, size_t i, const float* v) {
  reinterpret_cast<float4*>(p + i)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p + i)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void st8(uint16_t* p, size_t i, const float* v) {
  uint4 u;
  u.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  u.z = (uint32_t)f32_to_bf16(v[4]) | ((uint32_t)f32_to_bf16(v[5]) << 16);
  u.w = (uint32_t)f32_to_bf16(v[6]) | ((uint32_t)f32_to_bf16(v[7]) << 16);
  *reinterpret_cast<uint4*>(p + i) = u;
}
__device__ __forceinline__ void ld8(const float* p, size_t i, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p + i)[0], b = reinterpret_cast<const float4*>(p + i)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void ld8(const uint16_t* p, size_t i, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p + i);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
  }
}

// LDS barrier: this wave's LDS writes are complete, then every wave of the workgroup has arrived.  Written
// as one asm statement with a memory clobber so that no LDS access moves across it and no wait for
// outstanding global memory operations (a register prefetch, stores) is added.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over the whole block in a fixed order (deterministic); red holds >= 32 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

}  // namespace rollout
#endif
