// Host runtime of librollout: the C ABI, the planner that sizes sequences in
// flight to the HBM budget, the arena layout, the paged-KV block manager and
// the launch sequences of prefill, decode and whole rollouts.
//
// A GRPO step's rollout phase (section 3 of the paper) generates G
// completions for each of B prompts; the generation batch is kept a multiple
// of G (section 4.3), and the concurrency it runs at is the knob that moves
// power and throughput (section 6.4, Table 4).  Group size, sequences in
// flight, completion length, temperature and top-p are therefore arguments of
// every call, never state fixed at initialisation.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "internal.h"

using namespace rollout;

namespace {

thread_local std::string g_last_error = "";

constexpr size_t kAlign = 256;
constexpr int kPrefillRows = 4096;  // activation rows of one prefill chunk (whole prompts)
constexpr int kMaxSplits = 16;      // K splits of one projection GEMM

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Layer {
  size_t wqkv, wo, wgu, wdown, attn_norm, mlp_norm;
};

// Byte offsets of everything in the arena.
struct Layout {
  size_t embed = 0, lm_head = 0, final_norm = 0;
  std::vector<Layer> layers;
  size_t rope_cos = 0, rope_sin = 0;
  size_t weights_end = 0;  // weights + rope tables
  size_t x = 0, a = 0, q = 0, o = 0, h = 0, a_last = 0, part = 0, opart = 0, ml = 0, logits = 0;
  size_t tables = 0, ctx_len = 0, cols = 0, err = 0, samp = 0, wdq = 0;
  size_t cb = 0, stopmap = 0;  // continuous batching: 5 x [S] slot state, then the stop-token bitmap
  size_t work_end = 0;     // start of the KV pool
  size_t weight_bytes = 0, work_bytes = 0, kv_block_bytes = 0;
  int S = 0, R = 0, T_chunk = 0, max_blocks = 0, attn_splits_max = 1;
  size_t part_elems = 0;
};

Dims make_dims(const rollout_model_config& c) {
  Dims D;
  D.L = c.n_layers;
  D.d = c.d_model;
  D.nh = c.n_heads;
  D.nkv = c.n_kv_heads;
  D.hd = c.head_dim;
  D.ff = c.d_ff;
  D.V = c.vocab;
  D.qd = c.n_heads * c.head_dim;
  D.kvd = c.n_kv_heads * c.head_dim;
  D.nqkv = D.qd + 2 * D.kvd;
  D.eps = c.rms_eps;
  D.theta = c.rope_theta;
  D.dtype = c.dtype == ROLLOUT_DTYPE_INT4 ? ROLLOUT_DTYPE_BF16 : c.dtype;
  D.wq4 = c.dtype == ROLLOUT_DTYPE_INT4;
  D.blk = c.kv_block_size;
  D.max_ctx = c.max_prompt_len + c.max_new_tokens;
  return D;
}

// Returns ROLLOUT_OK or an error code with *msg set.
rollout_status validate_config(const rollout_model_config* c, std::string* msg) {
  if (!c) { *msg = "config is NULL"; return ROLLOUT_EINVAL; }
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 1 ||
      c->d_ff < 1 || c->vocab < 2) {
    *msg = "model dimensions must be positive (vocab >= 2)";
    return ROLLOUT_EINVAL;
  }
  if (c->dtype != ROLLOUT_DTYPE_FP32 && c->dtype != ROLLOUT_DTYPE_BF16 && c->dtype != ROLLOUT_DTYPE_INT4) {
    *msg = "dtype must be 0 (fp32), 1 (bf16) or 2 (int4 layer weights)";
    return ROLLOUT_EINVAL;
  }
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 1.f) || !(c->weight_std > 0.0)) {
    *msg = "rms_eps > 0, rope_theta > 1 and weight_std > 0 are required";
    return ROLLOUT_EINVAL;
  }
  if (c->max_prompt_len < 1 || c->max_new_tokens < 1 || c->max_seqs_in_flight < 1) {
    *msg = "max_prompt_len, max_new_tokens and max_seqs_in_flight must be >= 1";
    return ROLLOUT_EINVAL;
  }
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128) { *msg = "head_dim must be 32, 64 or 128"; return ROLLOUT_EUNSUPPORTED; }
  if (c->n_heads % c->n_kv_heads || c->n_heads / c->n_kv_heads > 16) {
    *msg = "n_heads must be a multiple of n_kv_heads, at most 16 query heads per KV head";
    return ROLLOUT_EUNSUPPORTED;
  }
  if (c->d_model % 32 || (c->n_heads * c->head_dim) % 32 || c->d_ff % 32 || c->vocab % 16) {
    *msg = "d_model, n_heads*head_dim and d_ff must be multiples of 32, vocab a multiple of 16";
    return ROLLOUT_EUNSUPPORTED;
  }
  if (c->dtype == ROLLOUT_DTYPE_INT4 && (c->d_model % 128 || (c->n_heads * c->head_dim) % 128 || c->d_ff % 128)) {
    *msg = "int4 weights need d_model, n_heads*head_dim and d_ff to be multiples of 128 (the quantisation group)";
    return ROLLOUT_EUNSUPPORTED;
  }
  if (c->kv_block_size != 8 && c->kv_block_size != 16 && c->kv_block_size != 32) {
    *msg = "kv_block_size must be 8, 16 or 32";
    return ROLLOUT_EUNSUPPORTED;
  }
  if (((int64_t)c->max_prompt_len + c->max_new_tokens + c->kv_block_size - 1) / c->kv_block_size > 16384) {
    *msg = "context longer than 16384 KV blocks";  // the attention kernel stages a sequence's block table in LDS
    return ROLLOUT_EUNSUPPORTED;
  }
  if ((int64_t)c->vocab * c->d_model > ((int64_t)1 << 31) - 1 || (int64_t)c->d_ff * 2 * c->d_model > ((int64_t)1 << 31) - 1) {
    *msg = "a weight matrix exceeds 2^31 elements";
    return ROLLOUT_EUNSUPPORTED;
  }
  return ROLLOUT_OK;
}

int prefill_chunk_rows(int max_prompt_len) {
  return std::max(max_prompt_len, kPrefillRows / max_prompt_len * max_prompt_len);
}

size_t max_part_elems(const Dims& D, int R) {
  size_t best = 0;
  const int Ns[4] = {D.nqkv, D.d, 2 * D.ff, D.d};
  const int Ks[4] = {D.d, D.qd, D.d, D.ff};
  for (int M = 1; M <= R; ++M)
    for (int j = 0; j < 4; ++j) {
      int s = gemm_splits(D.dtype, M, Ns[j], Ks[j], kMaxSplits);
      if (D.wq4)  // int4: the ring's splits, or two bf16 GEMMs (hi and lo) of up to half the splits each
        s = std::max(gemm_splits_q4(M, Ns[j], Ks[j], kMaxSplits), 2 * gemm_splits(D.dtype, M, Ns[j], Ks[j], kMaxSplits / 2));
      best = std::max(best, (size_t)s * (size_t)M * (size_t)Ns[j]);
    }
  return best;
}

// Layout of weights and work buffers for S sequences in flight; the KV pool follows work_end.
Layout make_layout(const Dims& D, int S, int max_prompt_len) {
  Layout Lo;
  const size_t eb = elem_bytes(D.dtype);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  // a layer projection of N outputs over K inputs
  auto proj_bytes = [&](int N, int K) {
    return D.wq4 ? q4_code_bytes(N, K) + q4_sz_bytes(N, K) : (size_t)N * K * eb;
  };
  Lo.embed = take((size_t)D.V * D.d * eb);
  Lo.layers.resize(D.L);
  for (int l = 0; l < D.L; ++l) {
    Layer& y = Lo.layers[l];
    y.wqkv = take(proj_bytes(D.nqkv, D.d));
    y.wo = take(proj_bytes(D.d, D.qd));
    y.wgu = take(proj_bytes(2 * D.ff, D.d));
    y.wdown = take(proj_bytes(D.d, D.ff));
    y.attn_norm = take((size_t)D.d * 4);
    y.mlp_norm = take((size_t)D.d * 4);
  }
  Lo.final_norm = take((size_t)D.d * 4);
  Lo.lm_head = take((size_t)D.V * D.d * eb);
  Lo.weight_bytes = off;
  Lo.rope_cos = take((size_t)D.max_ctx * (D.hd / 2) * 4);
  Lo.rope_sin = take((size_t)D.max_ctx * (D.hd / 2) * 4);
  Lo.weights_end = off;

  Lo.S = S;
  Lo.T_chunk = prefill_chunk_rows(max_prompt_len);
  // activation operands are addressed in whole 16-row MFMA blocks
  Lo.R = (std::max(S, Lo.T_chunk) + 15) / 16 * 16;
  Lo.max_blocks = (D.max_ctx + D.blk - 1) / D.blk;
  int st;
  Lo.attn_splits_max = attn_splits(D.max_ctx, &st);
  Lo.part_elems = max_part_elems(D, Lo.R);
  const size_t R = Lo.R;
  Lo.x = take(R * D.d * 4);
  Lo.a = take(R * std::max(D.d, D.qd) * eb);
  Lo.q = take(R * D.qd * eb);
  Lo.o = take(R * D.qd * eb);
  Lo.h = take(R * D.ff * eb);
  Lo.a_last = take((size_t)(S + 15) / 16 * 16 * D.d * eb);
  Lo.part = take(Lo.part_elems * 4);
  Lo.opart = take(R * D.nh * Lo.attn_splits_max * D.hd * 4);
  Lo.ml = take(R * D.nh * Lo.attn_splits_max * 2 * 4);
  Lo.logits = take((size_t)S * D.V * 4);
  Lo.samp = take(sample_scratch_bytes(S, D.V));
  Lo.tables = take((size_t)S * Lo.max_blocks * 4 + (size_t)S * 4);  // block tables, then ctx_len
  Lo.ctx_len = Lo.tables + (size_t)S * Lo.max_blocks * 4;
  Lo.cols = take(64);
  Lo.err = take(64);
  Lo.cb = take((size_t)5 * S * 4);
  Lo.stopmap = take((size_t)(D.V + 31) / 32 * 4);
  // int4: batches above the ring GEMM's rows multiply bf16 hi and lo copies of one projection at a time
  if (D.wq4)
    Lo.wdq = take(std::max(std::max((size_t)D.nqkv * D.d, (size_t)D.d * D.qd), (size_t)2 * D.ff * D.d) * 4);
  Lo.work_end = off;
  Lo.work_bytes = Lo.work_end - Lo.weights_end;
  Lo.kv_block_bytes = (size_t)D.L * D.nkv * 2 * D.blk * D.hd * eb;
  return Lo;
}

// KV blocks for n_prompts groups of G sequences of up to ctx tokens whose first P tokens are shared.
int64_t blocks_needed(int n_prompts, int G, int P, int ctx, int blk) {
  const int64_t shared = P / blk;
  const int64_t per_seq = (ctx + blk - 1) / blk - shared;
  return (int64_t)n_prompts * shared + (int64_t)n_prompts * G * per_seq;
}

// roctx range over one entry point's host-side work (enqueueing, and the waits the call makes itself), so
// that a profiler's marker trace shows prefill, decode, sampling and advantages as named spans
struct Range {
  explicit Range(const char* name) { roctxRangePush(name); }
  ~Range() { roctxRangePop(); }
  Range(const Range&) = delete;
  Range& operator=(const Range&) = delete;
};

struct Prof {
  bool on = false;
  std::vector<hipEvent_t> ev;
  struct Rec { int cls; int e0, e1; double bytes, flops; };
  std::vector<Rec> recs;
};

}  // namespace

struct rollout_ctx {
  rollout_model_config cfg;
  Dims D;
  Layout Lo;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  char* arena = nullptr;
  uint64_t arena_bytes = 0;
  int n_blocks = 0;
  std::string err;

  // host staging (pinned) for block tables and context lengths: two buffers used in turn, each with an
  // event after the copy that reads it, so a wave's upload waits only for the copy of the upload before last
  int32_t* h_tables[2] = {nullptr, nullptr};
  hipEvent_t h_tables_ev[2] = {nullptr, nullptr};
  int h_tables_next = 0;
  // graph executables of finished waves whose replays may still be running, each with an event recorded
  // after its last replay; destroyed once that event has completed
  std::vector<std::pair<hipGraphExec_t, hipEvent_t>> retired;
  int32_t* h_done = nullptr;  // ended flags of the slots, read back at refill boundaries

  // current wave
  bool wave = false;
  bool seq_refill = false;  // the slots hold single completions of different groups (no shared-prefix attention)
  int S = 0, P = 0, G = 0, cur_len = 0, n_prompts = 0;

  Prof prof;

  template <typename T = void>
  T* at(size_t off) const { return reinterpret_cast<T*>(arena + off); }
};

namespace {

}  // namespace

// The calling thread's context-free error message (what rollout_last_error(NULL) returns).
void rollout::set_last_error(const std::string& msg) { g_last_error = msg; }

namespace {

rollout_status fail(rollout_ctx* c, rollout_status st, const std::string& msg) {
  if (c) c->err = msg;
  g_last_error = msg;
  return st;
}

rollout_status hip_fail(rollout_ctx* c, hipError_t e, const char* where) {
  return fail(c, ROLLOUT_EDEVICE, std::string(where) + ": " + hipGetErrorString(e));
}

// Destroy the graph executables of earlier waves whose last replay has finished (all of them, after waiting,
// when wait is set).
void reap_graphs(rollout_ctx* c, bool wait) {
  auto& r = c->retired;
  size_t keep = 0;
  for (size_t i = 0; i < r.size(); ++i) {
    const bool done = wait ? hipEventSynchronize(r[i].second) == hipSuccess : hipEventQuery(r[i].second) == hipSuccess;
    if (done || wait) {
      hipGraphExecDestroy(r[i].first);
      hipEventDestroy(r[i].second);
    } else {
      r[keep++] = r[i];
    }
  }
  r.resize(keep);
}

#define HIP_TRY(ctx, expr, where)                  \
  do {                                             \
    hipError_t e_ = (expr);                        \
    if (e_ != hipSuccess) return hip_fail(ctx, e_, where); \
  } while (0)

WeightDesc wdesc(int rows, int cols, int layout, int fuse, int id0, int id1 = 0, int id2 = 0, int a = 0, int b = 0) {
  WeightDesc w;
  w.rows = rows;
  w.cols = cols;
  w.layout = layout;
  w.fuse = fuse;
  w.id0 = id0;
  w.id1 = id1;
  w.id2 = id2;
  w.a = a;
  w.b = b;
  return w;
}

int matrix_layout(const Dims& D) { return D.dtype == ROLLOUT_DTYPE_BF16 ? W_TILED : W_ROWMAJOR; }

// ---------------------------------------------------------------------------
// profiling hooks (HIP events around launches on the context stream)
// ---------------------------------------------------------------------------
struct Scope {
  rollout_ctx* c;
  int cls;
  double bytes, flops;
  int e0 = -1;
  Scope(rollout_ctx* c_, int cls_, double bytes_, double flops_) : c(c_), cls(cls_), bytes(bytes_), flops(flops_) {
    if (!c->prof.on) return;
    e0 = (int)c->prof.recs.size() * 2;
    while ((int)c->prof.ev.size() < e0 + 2) {
      hipEvent_t e;
      hipEventCreate(&e);
      c->prof.ev.push_back(e);
    }
    hipEventRecord(c->prof.ev[e0], c->stream);
  }
  ~Scope() {
    if (!c->prof.on) return;
    hipEventRecord(c->prof.ev[e0 + 1], c->stream);
    c->prof.recs.push_back({cls, e0, e0 + 1, bytes, flops});
  }
};

rollout_status gemm(rollout_ctx* c, const void* X, const void* W, float* out, int M, int N, int K, int max_splits,
                    int* splits_out) {
  const Dims& D = c->D;
  const int s = gemm_splits(D.dtype, M, N, K, max_splits);
  if ((size_t)s * M * N > c->Lo.part_elems && out == c->at<float>(c->Lo.part))
    return fail(c, ROLLOUT_EINVAL, "internal: split-K workspace too small");
  const double eb = (double)elem_bytes(D.dtype);
  Scope sc(c, 0, (double)N * K * eb + (double)M * K * eb + (double)M * N * 4, 2.0 * M * N * K);
  HIP_TRY(c, launch_gemm(c->stream, D.dtype, X, K, W, out, M, N, K, s), "gemm");
  *splits_out = s;
  return ROLLOUT_OK;
}

// Gate/up GEMM with SwiGLU applied to its own output (bf16 weights: any M; int4: M <= kSwigluMaxRows).
rollout_status gemm_swiglu(rollout_ctx* c, const void* X, const void* W, int M, int N, int K, void* h) {
  const double eb = (double)elem_bytes(c->D.dtype);
  const double wb = c->D.wq4 ? (double)(q4_code_bytes(N, K) + q4_sz_bytes(N, K)) : (double)N * K * eb;
  Scope sc(c, 0, wb + (double)M * K * eb + (double)M * (N / 2) * eb, 2.0 * M * N * K);
  if (c->D.wq4)
    HIP_TRY(c, launch_gemm_swiglu_q4(c->stream, X, W, M, N, K, h), "gemm");
  else
    HIP_TRY(c, launch_gemm_swiglu(c->stream, X, W, M, N, K, h), "gemm");
  return ROLLOUT_OK;
}

// A layer projection.  int4 matrices take the int4 ring GEMM for decode batches; larger batches
// (prefill) dequantise the matrix into bf16 tiles first and take the bf16 GEMM.
rollout_status proj(rollout_ctx* c, const void* X, const void* W, float* out, int M, int N, int K, int* splits_out) {
  if (!c->D.wq4) return gemm(c, X, W, out, M, N, K, kMaxSplits, splits_out);
  const double wb = (double)(q4_code_bytes(N, K) + q4_sz_bytes(N, K));
  if (M <= kSwigluMaxRows) {
    const int s = gemm_splits_q4(M, N, K, kMaxSplits);
    if ((size_t)s * M * N > c->Lo.part_elems) return fail(c, ROLLOUT_EINVAL, "internal: split-K workspace too small");
    Scope sc(c, 0, wb + (double)M * K * 2 + (double)s * M * N * 4, 2.0 * M * N * K);
    HIP_TRY(c, launch_gemm_q4(c->stream, X, W, out, M, N, K, s), "gemm");
    *splits_out = s;
    return ROLLOUT_OK;
  }
  // w = hi + lo with hi = bf16(w), lo = bf16(w - hi): two bf16 GEMMs into consecutive split slots
  char* hi = c->at<char>(c->Lo.wdq);
  char* lo = hi + (size_t)N * K * 2;
  {
    Scope sc(c, 2, wb + (double)N * K * 4, 0);
    HIP_TRY(c, launch_dequant_q4(c->stream, W, N, K, hi, lo), "dequantise");
  }
  int s1 = 0, s2 = 0;
  rollout_status r = gemm(c, X, hi, out, M, N, K, kMaxSplits / 2, &s1);
  if (r) return r;
  if ((size_t)2 * s1 * M * N > c->Lo.part_elems) return fail(c, ROLLOUT_EINVAL, "internal: split-K workspace too small");
  if ((r = gemm(c, X, lo, out + (size_t)s1 * M * N, M, N, K, kMaxSplits / 2, &s2))) return r;
  *splits_out = s1 + s2;
  return ROLLOUT_OK;
}

// Whether a decode batch takes the shared-prefix attention (whole groups of G >= 2 sequences whose prompt
// fills at least one KV block).  By default only when G x shared prompt tokens >= 8192: below that the
// group's redundant prompt reads are served by the caches and the extra pass costs more than it saves.
// ROLLOUT_SHARED_PREFIX=0 never takes it, =2 always does (read per call).
bool use_shared_prefix(const rollout_ctx* c, int M, const RowMap& rm) {
  const char* v = std::getenv("ROLLOUT_SHARED_PREFIX");
  const int mode = v ? std::atoi(v) : 1;
  const int p_shared = c->P / c->D.blk * c->D.blk;
  if (mode == 0 || !c->wave || c->seq_refill || c->G < 2 || p_shared < c->D.blk || M % c->G || rm.seq0 % c->G) return false;
  return mode == 2 || (int64_t)c->G * p_shared >= 8192;
}

// One transformer pass over M rows (prefill chunk or decode batch). On return
// c->Lo.a holds the final-normed hidden states (cache dtype).
// normed: the first layer's norm output is already in place (decode steps embed and normalise in one kernel)
rollout_status forward_layers(rollout_ctx* c, int M, RowMap rm, int attn_ctx_max, double kv_tokens_read,
                              bool normed = false) {
  const Dims& D = c->D;
  const Layout& Lo = c->Lo;
  float* x = c->at<float>(Lo.x);
  void* a = c->at(Lo.a);
  void* q = c->at(Lo.q);
  void* o = c->at(Lo.o);
  void* h = c->at(Lo.h);
  float* part = c->at<float>(Lo.part);
  float* opart = c->at<float>(Lo.opart);
  float* ml = c->at<float>(Lo.ml);
  int32_t* err = c->at<int32_t>(Lo.err);
  const int32_t* tables = c->at<int32_t>(Lo.tables);
  char* kv = c->arena + Lo.work_end;
  const double eb = (double)elem_bytes(D.dtype);
  int st_tok;
  const int asplits = attn_splits(attn_ctx_max, &st_tok);
  if (!normed) {
    Scope sc(c, 2, (double)M * D.d * (4 + eb), 0);
    HIP_TRY(c, launch_residual_norm(c->stream, D.dtype, nullptr, 1, M, D.d, x, c->at<float>(Lo.layers[0].attn_norm),
                                    D.eps, a), "rmsnorm");
  }
  // decode rows of whole groups read their group's shared prompt blocks once per group (shared-prefix attention)
  const int p_shared = (rm.P == 0 && attention_shares_prefix(D) && use_shared_prefix(c, M, rm)) ? c->P / D.blk * D.blk : 0;
  for (int l = 0; l < D.L; ++l) {
    const Layer& y = Lo.layers[l];
    int s;
    rollout_status r = proj(c, a, c->at(y.wqkv), part, M, D.nqkv, D.d, &s);
    if (r) return r;
    // decode rows: attention rotates q/k and appends k/v itself, straight from the split partials
    const bool attn_qkv = rm.P == 0 && attention_forms_qkv(D);
    if (!attn_qkv) {
      Scope sc(c, 2, (double)s * M * D.nqkv * 4 + (double)M * (D.qd + 2 * D.kvd) * eb, 0);
      HIP_TRY(c, launch_qkv_epilogue(c->stream, D, part, s, M, rm, c->at<float>(Lo.rope_cos), c->at<float>(Lo.rope_sin),
                                     q, kv, c->n_blocks, tables, Lo.max_blocks, l, err), "qkv epilogue");
    }
    {
      const double kvb = kv_tokens_read * D.nkv * 2.0 * D.hd * eb;
      Scope sc(c, 1, kvb + (double)M * D.qd * (eb + eb), 4.0 * kv_tokens_read * D.nh * D.hd);
      if (attn_qkv && p_shared > 0)
        HIP_TRY(c, launch_attention_shared(c->stream, D, kv, c->n_blocks, tables, Lo.max_blocks, rm, M, l, c->G,
                                           p_shared, q, opart, ml, o, err, part, s, c->at<float>(Lo.rope_cos),
                                           c->at<float>(Lo.rope_sin)), "attention");
      else
        HIP_TRY(c, launch_attention(c->stream, D, q, kv, c->n_blocks, tables, Lo.max_blocks, rm, M, asplits, st_tok, l,
                                    opart, ml, o, err, attn_qkv ? part : nullptr, s, c->at<float>(Lo.rope_cos),
                                    c->at<float>(Lo.rope_sin)), "attention");
    }
    r = proj(c, o, c->at(y.wo), part, M, D.d, D.qd, &s);
    if (r) return r;
    {
      Scope sc(c, 2, (double)s * M * D.d * 4 + (double)M * D.d * (8 + eb), 0);
      HIP_TRY(c, launch_residual_norm(c->stream, D.dtype, part, s, M, D.d, x, c->at<float>(y.mlp_norm), D.eps, a),
              "residual norm");
    }
    // SwiGLU in the gate/up GEMM's epilogue; int4 weights only up to the int4 ring's rows
    if (D.dtype == ROLLOUT_DTYPE_BF16 && (!D.wq4 || M <= kSwigluMaxRows)) {
      if ((r = gemm_swiglu(c, a, c->at(y.wgu), M, 2 * D.ff, D.d, h))) return r;
    } else {
      if ((r = proj(c, a, c->at(y.wgu), part, M, 2 * D.ff, D.d, &s))) return r;
      Scope sc(c, 2, (double)s * M * 2 * D.ff * 4 + (double)M * D.ff * eb, 0);
      HIP_TRY(c, launch_swiglu(c->stream, D.dtype, part, s, M, D.ff, h), "swiglu");
    }
    r = proj(c, h, c->at(y.wdown), part, M, D.d, D.ff, &s);
    if (r) return r;
    {
      const float* next_gain = l + 1 < D.L ? c->at<float>(Lo.layers[l + 1].attn_norm) : c->at<float>(Lo.final_norm);
      Scope sc(c, 2, (double)s * M * D.d * 4 + (double)M * D.d * (8 + eb), 0);
      HIP_TRY(c, launch_residual_norm(c->stream, D.dtype, part, s, M, D.d, x, next_gain, D.eps, a), "residual norm");
    }
  }
  return ROLLOUT_OK;
}

rollout_status upload_wave(rollout_ctx* c, int n_prompts, int P, int G) {
  const Dims& D = c->D;
  const Layout& Lo = c->Lo;
  const int S = n_prompts * G;
  const int ctx = P + c->cfg.max_new_tokens;
  const int64_t need = blocks_needed(n_prompts, G, P, ctx, D.blk);
  if (need > c->n_blocks)
    return fail(c, ROLLOUT_ENOMEM, "wave needs " + std::to_string(need) + " KV blocks, pool has " +
                                       std::to_string(c->n_blocks));
  // the staging buffer used two uploads ago may still feed its copy: wait for that copy only
  const int buf = c->h_tables_next;
  c->h_tables_next ^= 1;
  HIP_TRY(c, hipEventSynchronize(c->h_tables_ev[buf]), "staging wait");
  int32_t* t = c->h_tables[buf];
  std::fill(t, t + (size_t)Lo.S * Lo.max_blocks, -1);
  const int shared = P / D.blk;
  const int nb_seq = (ctx + D.blk - 1) / D.blk;
  int next = 0;
  for (int p = 0; p < n_prompts; ++p) {
    for (int j = 0; j < shared; ++j) {
      for (int g = 0; g < G; ++g) t[(size_t)(p * G + g) * Lo.max_blocks + j] = next;
      ++next;
    }
    for (int g = 0; g < G; ++g)
      for (int j = shared; j < nb_seq; ++j) t[(size_t)(p * G + g) * Lo.max_blocks + j] = next++;
  }
  int32_t* ctxl = t + (size_t)Lo.S * Lo.max_blocks;
  for (int s = 0; s < Lo.S; ++s) ctxl[s] = s < S ? P : 0;
  HIP_TRY(c, hipMemcpyAsync(c->at(Lo.tables), t, (size_t)Lo.S * (Lo.max_blocks + 1) * 4, hipMemcpyHostToDevice,
                            c->stream), "block table upload");
  HIP_TRY(c, hipEventRecord(c->h_tables_ev[buf], c->stream), "staging event");
  c->wave = true;
  c->seq_refill = false;
  c->S = S;
  c->P = P;
  c->G = G;
  c->n_prompts = n_prompts;
  c->cur_len = P;
  return ROLLOUT_OK;
}

// Prefill n_prompts prompts.  Prompt i writes its K/V through the block-table rows row0 + i * G_kv ..
// + G_kv - 1 (tables already in place; the partial last prompt block goes to each of them); the last
// position's logits, replicated G_out times, go to d_logits [n_prompts * G_out, V].
rollout_status prefill_rows(rollout_ctx* c, const int32_t* d_prompts, int n_prompts, int P, int G_kv, int G_out,
                            int row0, float* d_logits) {
  const Dims& D = c->D;
  const Layout& Lo = c->Lo;
  const int per_chunk = std::max(1, Lo.T_chunk / P);
  for (int p0 = 0; p0 < n_prompts; p0 += per_chunk) {
    const int np = std::min(per_chunk, n_prompts - p0);
    const int M = np * P;
    {
      Scope sc(c, 2, (double)M * D.d * (4 + elem_bytes(D.dtype)), 0);
      HIP_TRY(c, launch_embed(c->stream, D.dtype, c->at(Lo.embed), d_prompts + (size_t)p0 * P, 1, nullptr, M, D.d, D.V,
                              c->at<float>(Lo.x), c->at<int32_t>(Lo.err)), "embed");
    }
    RowMap rm{nullptr, P, G_kv, row0 + p0 * G_kv};
    rollout_status r = forward_layers(c, M, rm, P, (double)np * P * (P + 1) / 2.0);
    if (r) return r;
    HIP_TRY(c, launch_gather_rows(c->stream, D.dtype, c->at(Lo.a), D.d, P, G_out, np, c->at(Lo.a_last)), "gather");
    int s;
    r = gemm(c, c->at(Lo.a_last), c->at(Lo.lm_head), d_logits + (size_t)p0 * G_out * D.V, np * G_out, D.V, D.d, 1,
             &s);
    if (r) return r;
  }
  return ROLLOUT_OK;
}

rollout_status do_prefill(rollout_ctx* c, const int32_t* d_prompts, int n_prompts, int P, int G, float* d_logits) {
  rollout_status r = upload_wave(c, n_prompts, P, G);
  if (r) return r;
  return prefill_rows(c, d_prompts, n_prompts, P, G, G, 0, d_logits);
}

// Enqueue one decode step of the current wave (no host-side state change).
rollout_status enqueue_decode(rollout_ctx* c, const int32_t* tokens, int tok_stride, const int32_t* col,
                              float* d_logits, int ctx_max, bool advance = true) {
  const Dims& D = c->D;
  const Layout& Lo = c->Lo;
  const int S = c->S;
  const bool fused = D.d % 8 == 0 && D.d / 8 <= 1024;  // embedding and the first norm in one kernel
  {
    Scope sc(c, 2, (double)S * D.d * (4 + elem_bytes(D.dtype)), 0);
    if (fused)
      HIP_TRY(c, launch_embed_norm(c->stream, D.dtype, c->at(Lo.embed), tokens, tok_stride, col, S, D.d, D.V,
                                   c->at<float>(Lo.x), c->at<float>(Lo.layers[0].attn_norm), D.eps, c->at(Lo.a),
                                   c->at<int32_t>(Lo.err)), "embed + norm");
    else
      HIP_TRY(c, launch_embed(c->stream, D.dtype, c->at(Lo.embed), tokens, tok_stride, col, S, D.d, D.V,
                              c->at<float>(Lo.x), c->at<int32_t>(Lo.err)), "embed");
  }
  RowMap rm{c->at<int32_t>(Lo.ctx_len), 0, 1, 0};
  rollout_status r = forward_layers(c, S, rm, ctx_max, (double)S * (c->cur_len + 1), fused);
  if (r) return r;
  int s;
  r = gemm(c, c->at(Lo.a), c->at(Lo.lm_head), d_logits, S, D.V, D.d, 1, &s);
  if (r) return r;
  if (advance) HIP_TRY(c, launch_advance(c->stream, c->at<int32_t>(Lo.ctx_len), S, nullptr), "advance");
  return ROLLOUT_OK;
}

void rope_tables(const Dims& D, std::vector<float>* cs, std::vector<float>* sn) {
  const int half = D.hd / 2;
  cs->resize((size_t)D.max_ctx * half);
  sn->resize((size_t)D.max_ctx * half);
  for (int i = 0; i < half; ++i) {
    const double inv = std::pow((double)D.theta, -(2.0 * i) / (double)D.hd);
    for (int p = 0; p < D.max_ctx; ++p) {
      const double ang = (double)p * inv;
      (*cs)[(size_t)p * half + i] = (float)std::cos(ang);
      (*sn)[(size_t)p * half + i] = (float)std::sin(ang);
    }
  }
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* rollout_last_error(const rollout_ctx* ctx) {
  if (ctx) return ctx->err.c_str();
  return g_last_error.c_str();
}

rollout_status rollout_plan(const rollout_model_config* cfg, int32_t group_size, rollout_plan_t* out) {
  std::string msg;
  rollout_status st = validate_config(cfg, &msg);
  if (st) return fail(nullptr, st, msg);
  if (group_size < 1) return fail(nullptr, ROLLOUT_EINVAL, "group_size must be >= 1");
  if (!out) return fail(nullptr, ROLLOUT_EINVAL, "out is NULL");
  const Dims D = make_dims(*cfg);
  uint64_t budget = cfg->hbm_budget_bytes;
  uint64_t reserve = 0;
  if (budget == 0) {
    size_t free_b = 0, total_b = 0;
    hipError_t e = hipMemGetInfo(&free_b, &total_b);
    if (e != hipSuccess) return fail(nullptr, ROLLOUT_EDEVICE, std::string("hipMemGetInfo: ") + hipGetErrorString(e));
    budget = free_b;
    reserve = (uint64_t)2 << 30;  // headroom for the caller's own allocations
  }
  const int ctx = cfg->max_prompt_len + cfg->max_new_tokens;
  // bytes of the arena for k whole groups in flight (weights + work for k*G rows + KV blocks)
  auto arena_for = [&](int64_t k, Layout* lo, int64_t* nb) {
    *lo = make_layout(D, (int)(k * group_size), cfg->max_prompt_len);
    *nb = blocks_needed((int)k, group_size, cfg->max_prompt_len, ctx, D.blk);
    return (uint64_t)lo->work_end + (uint64_t)*nb * lo->kv_block_bytes;
  };
  // the arena grows with the number of groups, so the largest fitting count is found by bisection
  int64_t lo_k = 0, hi_k = cfg->max_seqs_in_flight / group_size;
  Layout Lo;
  int64_t nb = 0;
  while (lo_k < hi_k) {
    const int64_t mid = (lo_k + hi_k + 1) / 2;
    if (arena_for(mid, &Lo, &nb) + reserve <= budget) lo_k = mid;
    else hi_k = mid - 1;
  }
  if (lo_k < 1)
    return fail(nullptr, ROLLOUT_ENOMEM, "not even one group of " + std::to_string(group_size) +
                                             " sequences fits in the HBM budget");
  const uint64_t total = arena_for(lo_k, &Lo, &nb);
  out->seqs_in_flight_max = (int32_t)(lo_k * group_size);
  out->kv_blocks = (int32_t)nb;
  out->arena_bytes = total;
  out->weight_bytes = Lo.weight_bytes;
  out->kv_block_bytes = Lo.kv_block_bytes;
  out->kv_bytes = (uint64_t)nb * Lo.kv_block_bytes;
  out->work_bytes = Lo.work_end - Lo.weight_bytes;
  return ROLLOUT_OK;
}

rollout_status rollout_init(const rollout_model_config* cfg, void* d_arena, uint64_t arena_bytes, void* hip_stream,
                            rollout_ctx** out) {
  std::string msg;
  rollout_status st = validate_config(cfg, &msg);
  if (st) return fail(nullptr, st, msg);
  if (!out || !d_arena) return fail(nullptr, ROLLOUT_EINVAL, "arena and out must be non-NULL");
  if ((uintptr_t)d_arena % kAlign) return fail(nullptr, ROLLOUT_EINVAL, "arena must be 256-byte aligned");
  const Dims D = make_dims(*cfg);
  Layout Lo = make_layout(D, cfg->max_seqs_in_flight, cfg->max_prompt_len);
  if (arena_bytes < Lo.work_end + Lo.kv_block_bytes * (uint64_t)Lo.max_blocks)
    return fail(nullptr, ROLLOUT_ENOMEM, "arena of " + std::to_string(arena_bytes) + " bytes holds no sequence (needs " +
                                             std::to_string(Lo.work_end + Lo.kv_block_bytes * Lo.max_blocks) + ")");
  const uint64_t nb = (arena_bytes - Lo.work_end) / Lo.kv_block_bytes;
  rollout_ctx* c = new rollout_ctx();
  c->cfg = *cfg;
  c->D = D;
  c->Lo = Lo;
  c->arena = (char*)d_arena;
  c->arena_bytes = arena_bytes;
  c->n_blocks = (int)std::min<uint64_t>(nb, (uint64_t)INT32_MAX);
  if (hip_stream) {
    c->stream = (hipStream_t)hip_stream;
  } else {
    hipError_t e = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking);
    if (e != hipSuccess) { delete c; return fail(nullptr, ROLLOUT_EDEVICE, std::string("stream: ") + hipGetErrorString(e)); }
    c->own_stream = true;
  }
  hipError_t e = hipSuccess;
  for (int b = 0; b < 2 && e == hipSuccess; ++b) {
    e = hipHostMalloc((void**)&c->h_tables[b], (size_t)Lo.S * (Lo.max_blocks + 1) * 4, hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->h_tables_ev[b], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(c->h_tables_ev[b], c->stream);
  }
  if (e == hipSuccess) e = hipHostMalloc((void**)&c->h_done, (size_t)Lo.S * 4, hipHostMallocDefault);
  if (e != hipSuccess) {
    rollout_destroy(c);
    return fail(nullptr, ROLLOUT_EDEVICE, std::string("pinned staging: ") + hipGetErrorString(e));
  }
  auto bad = [&](hipError_t err, const char* where) {
    std::string m = std::string(where) + ": " + hipGetErrorString(err);
    rollout_destroy(c);
    return fail(nullptr, ROLLOUT_EDEVICE, m);
  };
  // weights, straight into the layouts the kernels read
  const int lay = matrix_layout(D);
  const uint64_t seed = cfg->weight_seed;
  const double sd = cfg->weight_std;
  if ((e = launch_synth(c->stream, c->at(Lo.embed), D.dtype, wdesc(D.V, D.d, W_ROWMAJOR, FUSE_NONE, 0), seed, sd)))
    return bad(e, "synth embed");
  for (int l = 0; l < D.L; ++l) {
    const Layer& y = Lo.layers[l];
    const int b = 1 + 9 * l;
    // layer projections: int4 groups quantised from the same fp32 values, or the dtype's layout
    auto synth_proj = [&](void* dst, const WeightDesc& w) {
      return D.wq4 ? launch_synth_q4(c->stream, dst, w, seed, sd) : launch_synth(c->stream, dst, D.dtype, w, seed, sd);
    };
    if ((e = synth_proj(c->at(y.wqkv), wdesc(D.nqkv, D.d, lay, FUSE_QKV, b + 1, b + 2, b + 3, D.qd, D.kvd))) ||
        (e = synth_proj(c->at(y.wo), wdesc(D.d, D.qd, lay, FUSE_NONE, b + 4))) ||
        (e = synth_proj(c->at(y.wgu), wdesc(2 * D.ff, D.d, lay, FUSE_GU, b + 6, b + 7))) ||
        (e = synth_proj(c->at(y.wdown), wdesc(D.d, D.ff, lay, FUSE_NONE, b + 8))) ||
        (e = launch_fill(c->stream, c->at<float>(y.attn_norm), D.d, 1.0f)) ||
        (e = launch_fill(c->stream, c->at<float>(y.mlp_norm), D.d, 1.0f)))
      return bad(e, "synth layer");
  }
  if ((e = launch_fill(c->stream, c->at<float>(Lo.final_norm), D.d, 1.0f)) ||
      (e = launch_synth(c->stream, c->at(Lo.lm_head), D.dtype, wdesc(D.V, D.d, lay, FUSE_NONE, 2 + 9 * D.L), seed, sd)))
    return bad(e, "synth head");
  std::vector<float> cs, sn;
  rope_tables(D, &cs, &sn);
  if ((e = hipMemcpyAsync(c->at(Lo.rope_cos), cs.data(), cs.size() * 4, hipMemcpyHostToDevice, c->stream)) ||
      (e = hipMemcpyAsync(c->at(Lo.rope_sin), sn.data(), sn.size() * 4, hipMemcpyHostToDevice, c->stream)) ||
      (e = hipMemsetAsync(c->at(Lo.err), 0, 64, c->stream)) ||
      (e = hipMemsetAsync(c->at(Lo.cols), 0, 64, c->stream)) ||
      (e = hipStreamSynchronize(c->stream)))
    return bad(e, "init upload");
  *out = c;
  return ROLLOUT_OK;
}

void rollout_destroy(rollout_ctx* ctx) {
  if (!ctx) return;
  if (ctx->stream) hipStreamSynchronize(ctx->stream);
  reap_graphs(ctx, true);
  for (hipEvent_t e : ctx->prof.ev) hipEventDestroy(e);
  for (int b = 0; b < 2; ++b) {
    if (ctx->h_tables[b]) hipHostFree(ctx->h_tables[b]);
    if (ctx->h_tables_ev[b]) hipEventDestroy(ctx->h_tables_ev[b]);
  }
  if (ctx->h_done) hipHostFree(ctx->h_done);
  if (ctx->own_stream) hipStreamDestroy(ctx->stream);
  delete ctx;
}

rollout_status rollout_prefill(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts, int32_t prompt_len,
                               int32_t group_size, float* d_logits) {
  Range range("rollout_prefill");
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_prompts || !d_logits) return fail(ctx, ROLLOUT_EINVAL, "prompts and logits must be non-NULL");
  if (n_prompts < 1 || group_size < 1) return fail(ctx, ROLLOUT_EINVAL, "n_prompts and group_size must be >= 1");
  if (prompt_len < 1 || prompt_len > ctx->cfg.max_prompt_len)
    return fail(ctx, ROLLOUT_EINVAL, "prompt_len must be in [1, max_prompt_len]");
  if ((int64_t)n_prompts * group_size > ctx->Lo.S)
    return fail(ctx, ROLLOUT_ENOMEM, "n_prompts * group_size exceeds the sequences in flight of the context");
  ctx->wave = false;
  return do_prefill(ctx, d_prompts, n_prompts, prompt_len, group_size, d_logits);
}

rollout_status rollout_decode_step(rollout_ctx* ctx, const int32_t* d_tokens, float* d_logits) {
  Range range("rollout_decode_step");
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_tokens || !d_logits) return fail(ctx, ROLLOUT_EINVAL, "tokens and logits must be non-NULL");
  if (!ctx->wave) return fail(ctx, ROLLOUT_ESTATE, "decode before prefill");
  if (ctx->cur_len + 1 > ctx->P + ctx->cfg.max_new_tokens)
    return fail(ctx, ROLLOUT_ESTATE, "context full (max_prompt_len + max_new_tokens reached)");
  rollout_status r = enqueue_decode(ctx, d_tokens, 1, nullptr, d_logits, ctx->P + ctx->cfg.max_new_tokens);
  if (r) return r;
  ctx->cur_len += 1;
  return ROLLOUT_OK;
}

rollout_status rollout_sample(rollout_ctx* ctx, const float* d_logits, int32_t n_seqs, float temperature, float top_p,
                              const float* d_uniforms, int32_t* d_tokens_out) {
  Range range("rollout_sample");
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_logits || !d_uniforms || !d_tokens_out) return fail(ctx, ROLLOUT_EINVAL, "NULL buffer");
  if (n_seqs < 1) return fail(ctx, ROLLOUT_EINVAL, "n_seqs must be >= 1");
  if (!(temperature >= 0.f) || !std::isfinite(temperature)) return fail(ctx, ROLLOUT_EINVAL, "temperature must be >= 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(ctx, ROLLOUT_EINVAL, "top_p must be in (0, 1]");
  // rows go through the sampler scratch in batches of the context's sequence capacity
  for (int r0 = 0; r0 < n_seqs; r0 += ctx->Lo.S) {
    const int n = std::min(ctx->Lo.S, n_seqs - r0);
    Scope sc(ctx, 2, (double)n * ctx->D.V * 4, 0);
    HIP_TRY(ctx, launch_sample(ctx->stream, d_logits + (size_t)r0 * ctx->D.V, n, ctx->D.V, temperature, top_p,
                               d_uniforms + r0, 1, nullptr, d_tokens_out + r0, 1, ctx->at(ctx->Lo.samp)), "sample");
  }
  return ROLLOUT_OK;
}

rollout_status grpo_advantages(const float* d_rewards, int32_t n_groups, int32_t group_size, float eps,
                               int32_t std_ddof, float* d_adv, int32_t* d_zero_var_groups, void* hip_stream) {
  Range range("grpo_advantages");
  if (!d_rewards || !d_adv) return fail(nullptr, ROLLOUT_EINVAL, "rewards and advantages must be non-NULL");
  if (n_groups < 1 || group_size < 1) return fail(nullptr, ROLLOUT_EINVAL, "n_groups and group_size must be >= 1");
  if (std_ddof != 0 && std_ddof != 1) return fail(nullptr, ROLLOUT_EINVAL, "std_ddof must be 0 or 1");
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(nullptr, ROLLOUT_EINVAL, "eps must be >= 0");
  hipError_t e = launch_grpo((hipStream_t)hip_stream, d_rewards, n_groups, group_size, eps, std_ddof, d_adv,
                             d_zero_var_groups);
  if (e != hipSuccess) return fail(nullptr, ROLLOUT_EDEVICE, std::string("grpo: ") + hipGetErrorString(e));
  return ROLLOUT_OK;
}

rollout_status rollout_generate(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts, int32_t prompt_len,
                                int32_t group_size, int32_t seqs_in_flight, int32_t max_new_tokens, float temperature,
                                float top_p, const float* d_uniforms, int32_t* d_tokens_out) {
  Range range("rollout_generate");
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_prompts || !d_uniforms || !d_tokens_out) return fail(ctx, ROLLOUT_EINVAL, "NULL buffer");
  if (n_prompts < 1 || group_size < 1 || seqs_in_flight < 1)
    return fail(ctx, ROLLOUT_EINVAL, "n_prompts, group_size and seqs_in_flight must be >= 1");
  if (prompt_len < 1 || prompt_len > ctx->cfg.max_prompt_len)
    return fail(ctx, ROLLOUT_EINVAL, "prompt_len must be in [1, max_prompt_len]");
  if (max_new_tokens < 1 || max_new_tokens > ctx->cfg.max_new_tokens)
    return fail(ctx, ROLLOUT_EINVAL, "max_new_tokens must be in [1, config max_new_tokens]");
  if (!(temperature >= 0.f) || !std::isfinite(temperature)) return fail(ctx, ROLLOUT_EINVAL, "temperature must be >= 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(ctx, ROLLOUT_EINVAL, "top_p must be in (0, 1]");
  reap_graphs(ctx, false);
  const Dims& D = ctx->D;
  // sequences per wave: whole groups, within the context's rows and the KV pool
  int S = std::min<int64_t>(seqs_in_flight, ctx->Lo.S) / group_size * group_size;
  const int ctxlen = prompt_len + ctx->cfg.max_new_tokens;
  while (S >= group_size && blocks_needed(S / group_size, group_size, prompt_len, ctxlen, D.blk) > ctx->n_blocks)
    S -= group_size;
  if (S < group_size) return fail(ctx, ROLLOUT_ENOMEM, "one group does not fit in the context");
  const int per_wave = S / group_size;
  float* logits = ctx->at<float>(ctx->Lo.logits);
  int32_t* cols = ctx->at<int32_t>(ctx->Lo.cols);
  const int N = max_new_tokens;
  for (int p0 = 0; p0 < n_prompts; p0 += per_wave) {
    const int np = std::min(per_wave, n_prompts - p0);
    const int s0 = p0 * group_size;
    const int Sw = np * group_size;
    ctx->wave = false;
    rollout_status r = do_prefill(ctx, d_prompts + (size_t)p0 * prompt_len, np, prompt_len, group_size, logits);
    if (r) return r;
    int32_t* tok = d_tokens_out + (size_t)s0 * N;
    const float* uu = d_uniforms + (size_t)s0 * N;
    HIP_TRY(ctx, launch_sample(ctx->stream, logits, Sw, D.V, temperature, top_p, uu, N, nullptr, tok, N,
                               ctx->at(ctx->Lo.samp)), "sample");
    if (N == 1) continue;
    HIP_TRY(ctx, launch_set_cols(ctx->stream, cols, 0, 1), "set cols");
    const bool use_graph = !ctx->prof.on;
    // cols[0] = column of the token fed in, cols[1] = column drawn; both move on after the draw
    // the sequences' positions and the token columns move on together, in one launch after the draw
    auto step = [&]() -> rollout_status {
      rollout_status rr = enqueue_decode(ctx, tok, N, cols, logits, prompt_len + N, false);
      if (rr) return rr;
      HIP_TRY(ctx, launch_sample(ctx->stream, logits, Sw, D.V, temperature, top_p, uu, N, cols + 1, tok, N,
                                 ctx->at(ctx->Lo.samp)), "sample");
      HIP_TRY(ctx, launch_advance(ctx->stream, ctx->at<int32_t>(ctx->Lo.ctx_len), ctx->S, cols), "advance");
      return ROLLOUT_OK;
    };
    if (!use_graph) {
      for (int t = 1; t < N; ++t) {
        r = step();
        if (r) return r;
        ctx->cur_len += 1;
      }
      continue;
    }
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    HIP_TRY(ctx, hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal), "begin capture");
    r = step();
    hipError_t ce = hipStreamEndCapture(ctx->stream, &graph);
    if (r) {
      if (graph) hipGraphDestroy(graph);
      return r;
    }
    if (ce != hipSuccess) return hip_fail(ctx, ce, "end capture");
    hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    hipGraphDestroy(graph);
    if (ie != hipSuccess) return hip_fail(ctx, ie, "graph instantiate");
    {
      Range replay("rollout_generate: decode steps (graph replay)");
      for (int t = 1; t < N; ++t) {
        hipError_t le = hipGraphLaunch(exec, ctx->stream);
        if (le != hipSuccess) {
          hipStreamSynchronize(ctx->stream);
          hipGraphExecDestroy(exec);
          return hip_fail(ctx, le, "graph launch");
        }
        ctx->cur_len += 1;
      }
    }
    // the replays run on after the call returns: the executable is destroyed once they have finished
    hipEvent_t done = nullptr;
    hipError_t ee = hipEventCreateWithFlags(&done, hipEventDisableTiming);
    if (ee == hipSuccess) ee = hipEventRecord(done, ctx->stream);
    if (ee != hipSuccess) {
      hipStreamSynchronize(ctx->stream);
      hipGraphExecDestroy(exec);
      if (done) hipEventDestroy(done);
      return hip_fail(ctx, ee, "wave event");
    }
    ctx->retired.emplace_back(exec, done);
  }
  return ROLLOUT_OK;
}

rollout_status rollout_generate_eos(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts,
                                    int32_t prompt_len, int32_t group_size, int32_t seqs_in_flight,
                                    int32_t max_new_tokens, float temperature, float top_p, const float* d_uniforms,
                                    const int32_t* d_stop_ids, int32_t n_stop, int32_t refill_interval,
                                    int32_t whole_groups, int32_t* d_tokens_out, int32_t* d_lengths_out,
                                    int32_t* d_admit_step_out, int32_t* h_decode_steps_out) {
  Range range("rollout_generate_eos");
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_prompts || !d_uniforms || !d_tokens_out || !d_lengths_out) return fail(ctx, ROLLOUT_EINVAL, "NULL buffer");
  if (n_stop < 0 || (n_stop > 0 && !d_stop_ids)) return fail(ctx, ROLLOUT_EINVAL, "n_stop < 0 or stop ids NULL");
  if (refill_interval < 1) return fail(ctx, ROLLOUT_EINVAL, "refill_interval must be >= 1");
  if (whole_groups != 0 && whole_groups != 1) return fail(ctx, ROLLOUT_EINVAL, "whole_groups must be 0 or 1");
  if (n_prompts < 1 || group_size < 1 || seqs_in_flight < 1)
    return fail(ctx, ROLLOUT_EINVAL, "n_prompts, group_size and seqs_in_flight must be >= 1");
  if ((int64_t)n_prompts * group_size > INT32_MAX)
    return fail(ctx, ROLLOUT_EINVAL, "n_prompts * group_size exceeds the int32 completion index");
  if (prompt_len < 1 || prompt_len > ctx->cfg.max_prompt_len)
    return fail(ctx, ROLLOUT_EINVAL, "prompt_len must be in [1, max_prompt_len]");
  if (max_new_tokens < 1 || max_new_tokens > ctx->cfg.max_new_tokens)
    return fail(ctx, ROLLOUT_EINVAL, "max_new_tokens must be in [1, config max_new_tokens]");
  if (!(temperature >= 0.f) || !std::isfinite(temperature)) return fail(ctx, ROLLOUT_EINVAL, "temperature must be >= 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(ctx, ROLLOUT_EINVAL, "top_p must be in (0, 1]");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  const int G = group_size, P = prompt_len, N = max_new_tokens;
  const int n_seq = n_prompts * G;
  // KV blocks: a group's full prompt blocks are shared; positions from there on belong to a slot
  const int n_shared = P / D.blk;
  const bool partial = P % D.blk != 0;
  const int n_own = (P + N + D.blk - 1) / D.blk - n_shared;
  const int n_rec = n_shared + (partial ? 1 : 0);  // a prompt record: shared blocks + its partial block
  int S;
  if (whole_groups) {
    // whole groups, within the context's rows and the KV pool, no more ranges than prompts
    S = std::min<int64_t>(seqs_in_flight, Lo.S) / G * G;
    const int ctxlen = P + ctx->cfg.max_new_tokens;
    while (S >= G && blocks_needed(S / G, G, P, ctxlen, D.blk) > ctx->n_blocks) S -= G;
    if (S < G) return fail(ctx, ROLLOUT_ENOMEM, "one group does not fit in the context");
    S = std::min(S / G, (int)n_prompts) * G;
  } else {
    // a group's token-0 prefill and draw write G rows of logits and sampler scratch, sized for the context's rows
    if (G > Lo.S)
      return fail(ctx, ROLLOUT_ENOMEM, "group_size " + std::to_string(G) + " exceeds the context's " +
                                           std::to_string(Lo.S) + " rows (a group's first tokens are drawn together)");
    // single completions: one block-table row beyond the slots serves the prefills; up to S + 1 prompt
    // records are alive at once (a group per occupied slot, plus the one being admitted)
    S = std::min<int64_t>(std::min<int64_t>(seqs_in_flight, Lo.S - 1), n_seq);
    while (S >= 1 && (int64_t)(S + 1) * n_rec + (int64_t)S * n_own > ctx->n_blocks) --S;
    if (S < 1) return fail(ctx, ROLLOUT_ENOMEM, "one completion does not fit in the context");
  }
  ctx->wave = false;
  int32_t* tables = ctx->at<int32_t>(Lo.tables);
  int32_t* ctx_len = ctx->at<int32_t>(Lo.ctx_len);
  if (whole_groups) {
    // every range keeps its block-table rows for the whole call; a refilled range reuses them
    rollout_status r = upload_wave(ctx, S / G, P, G);
    if (r) return r;
  } else {
    HIP_TRY(ctx, hipStreamSynchronize(ctx->stream), "stream sync");
    ctx->wave = true;
    ctx->seq_refill = true;
    ctx->S = S;
    ctx->P = P;
    ctx->G = G;
    ctx->n_prompts = n_prompts;
    ctx->cur_len = P;
  }
  int32_t* base = ctx->at<int32_t>(Lo.cb);
  const CbState cb{base, base + S, base + 2 * S, base + 3 * S, reinterpret_cast<float*>(base + 4 * S)};
  uint32_t* stop = n_stop > 0 ? ctx->at<uint32_t>(Lo.stopmap) : nullptr;
  if (stop) HIP_TRY(ctx, launch_stop_bitmap(ctx->stream, stop, D.V, d_stop_ids, n_stop, ctx->at<int32_t>(Lo.err)), "stop set");
  HIP_TRY(ctx, launch_cb_reset(ctx->stream, S, cb), "slot reset");
  float* logits = ctx->at<float>(Lo.logits);
  void* samp = ctx->at(Lo.samp);
  std::vector<int32_t> admit_step(n_seq, -1);
  // host view of the slots: completion per slot (-1 none); whole groups use slot ranges of G
  std::vector<int> slot_seq(S, -1);
  int next = 0;  // next completion to admit, in order s = p * G + g
  // --- whole groups: a range takes the next prompt's group: reset its slots, prefill, draw token 0
  auto admit_group = [&](int k, int boundary) -> rollout_status {
    const int p = next / G;
    const int r0 = k * G, seq0 = p * G;
    for (int g = 0; g < G; ++g) {
      admit_step[seq0 + g] = boundary;
      slot_seq[r0 + g] = seq0 + g;
    }
    next += G;
    HIP_TRY(ctx, launch_cb_admit(ctx->stream, cb, r0, G, seq0, P, N, ctx_len, d_tokens_out), "admit");
    rollout_status rr = prefill_rows(ctx, d_prompts + (size_t)p * P, 1, P, G, G, r0, logits);
    if (rr) return rr;
    HIP_TRY(ctx, launch_sample(ctx->stream, logits, G, D.V, temperature, top_p, d_uniforms + (size_t)seq0 * N, N,
                               nullptr, cb.draw + r0, 1, samp), "sample");
    HIP_TRY(ctx, launch_cb_commit(ctx->stream, cb, r0, r0 + G, N, stop, d_uniforms, ctx_len, d_tokens_out,
                                  d_lengths_out, false), "commit");
    return ROLLOUT_OK;
  };
  // --- single completions: prompt records [0, S], own blocks of slot r after them
  std::vector<int> rec_free, rec_of(n_prompts, -1), ended_of(n_prompts, 0);
  for (int k = S; k >= 0; --k) rec_free.push_back(k);
  const int own0 = (S + 1) * n_rec;
  auto admit_seq = [&](int r, int boundary) -> rollout_status {
    const int s = next++, p = s / G, g = s % G;
    if (g == 0) {  // the group's first completion: prefill its prompt into a free record, draw every token 0
      if (rec_free.empty()) return fail(ctx, ROLLOUT_EINVAL, "internal: no free prompt record");
      const int k = rec_free.back();
      rec_free.pop_back();
      rec_of[p] = k;
      HIP_TRY(ctx, launch_seq_table(ctx->stream, tables, Lo.max_blocks, S, k * n_rec, n_shared, partial, -1, 0),
              "prefill table");
      rollout_status rr = prefill_rows(ctx, d_prompts + (size_t)p * P, 1, P, 1, G, S, logits);
      if (rr) return rr;
      HIP_TRY(ctx, launch_sample(ctx->stream, logits, G, D.V, temperature, top_p, d_uniforms + (size_t)p * G * N, N,
                                 nullptr, d_tokens_out + (size_t)p * G * N, N, samp), "sample");
    }
    const int k = rec_of[p];
    HIP_TRY(ctx, launch_seq_table(ctx->stream, tables, Lo.max_blocks, r, k * n_rec, n_shared, partial, own0 + r * n_own,
                                  n_own), "slot table");
    if (partial)  // the slot's first own block starts as the record's copy of the partial prompt block
      HIP_TRY(ctx, launch_copy_kv_block(ctx->stream, ctx->arena + Lo.work_end, ctx->n_blocks, D.L,
                                        Lo.kv_block_bytes / D.L, k * n_rec + n_shared, own0 + r * n_own),
              "partial block");
    HIP_TRY(ctx, launch_seq_admit(ctx->stream, cb, r, s, P, N, ctx_len, d_tokens_out), "admit");
    HIP_TRY(ctx, launch_cb_commit(ctx->stream, cb, r, r + 1, N, stop, d_uniforms, ctx_len, d_tokens_out, d_lengths_out,
                                  false), "commit");
    admit_step[s] = boundary;
    slot_seq[r] = s;
    return ROLLOUT_OK;
  };
  // one decode step over all slots: feed each slot's last draw, draw with its staged uniform, file the draws
  auto step = [&]() -> rollout_status {
    rollout_status rr = enqueue_decode(ctx, cb.draw, 1, nullptr, logits, P + N, false);
    if (rr) return rr;
    HIP_TRY(ctx, launch_sample(ctx->stream, logits, S, D.V, temperature, top_p, cb.u_slot, 1, nullptr, cb.draw, 1,
                               samp), "sample");
    HIP_TRY(ctx, launch_cb_commit(ctx->stream, cb, 0, S, N, stop, d_uniforms, ctx_len, d_tokens_out, d_lengths_out,
                                  true), "commit");
    return ROLLOUT_OK;
  };
  rollout_status r = ROLLOUT_OK;
  if (whole_groups) {
    for (int k = 0; k < S / G && !r; ++k) r = admit_group(k, 0);
  } else {
    for (int i = 0; i < S && !r; ++i) r = admit_seq(i, 0);
  }
  if (r) return r;
  hipGraphExec_t exec = nullptr;
  auto finish = [&](rollout_status st) {
    if (exec) {
      hipStreamSynchronize(ctx->stream);
      hipGraphExecDestroy(exec);
      exec = nullptr;
    }
    ctx->wave = false;  // the slots' state is not a wave that rollout_decode_step may continue
    return st;
  };
  if (!ctx->prof.on) {
    hipGraph_t graph = nullptr;
    HIP_TRY(ctx, hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal), "begin capture");
    r = step();
    hipError_t ce = hipStreamEndCapture(ctx->stream, &graph);
    if (r) {
      if (graph) hipGraphDestroy(graph);
      return finish(r);
    }
    if (ce != hipSuccess) return finish(hip_fail(ctx, ce, "end capture"));
    hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    hipGraphDestroy(graph);
    if (ie != hipSuccess) return finish(hip_fail(ctx, ie, "graph instantiate"));
  }
  int steps = 0;
  auto live = [&]() {
    for (int i = 0; i < S; ++i)
      if (slot_seq[i] >= 0) return true;
    return false;
  };
  while (live()) {
    for (int i = 0; i < refill_interval; ++i) {
      if (exec) {
        hipError_t le = hipGraphLaunch(exec, ctx->stream);
        if (le != hipSuccess) return finish(hip_fail(ctx, le, "graph launch"));
      } else if ((r = step())) {
        return finish(r);
      }
    }
    steps += refill_interval;
    hipError_t ce = hipMemcpyAsync(ctx->h_done, cb.done, (size_t)S * 4, hipMemcpyDeviceToHost, ctx->stream);
    if (ce == hipSuccess) ce = hipStreamSynchronize(ctx->stream);
    if (ce != hipSuccess) return finish(hip_fail(ctx, ce, "ended flags read"));
    if (whole_groups) {
      for (int k = 0; k < S / G; ++k) {
        if (slot_seq[k * G] < 0) continue;
        bool ended = true;
        for (int g = 0; g < G; ++g) ended = ended && ctx->h_done[k * G + g] != 0;
        if (!ended) continue;
        for (int g = 0; g < G; ++g) slot_seq[k * G + g] = -1;
        if (next < n_seq && (r = admit_group(k, steps))) return finish(r);
      }
    } else {
      for (int i = 0; i < S; ++i) {
        const int s = slot_seq[i];
        if (s < 0 || !ctx->h_done[i]) continue;
        slot_seq[i] = -1;
        if (++ended_of[s / G] == G) rec_free.push_back(rec_of[s / G]);
        if (next < n_seq && (r = admit_seq(i, steps))) return finish(r);
      }
    }
  }
  r = finish(ROLLOUT_OK);
  if (d_admit_step_out)
    HIP_TRY(ctx, hipMemcpy(d_admit_step_out, admit_step.data(), (size_t)n_seq * 4, hipMemcpyHostToDevice),
            "admission steps");
  if (h_decode_steps_out) *h_decode_steps_out = steps;
  return r;
}

rollout_status rollout_length_rewards(const int32_t* d_lengths, int32_t n, int32_t target, float* d_rewards,
                                      int64_t* d_total_tokens, void* hip_stream) {
  if (!d_lengths || !d_rewards) return fail(nullptr, ROLLOUT_EINVAL, "lengths and rewards must be non-NULL");
  if (n < 1 || target < 1) return fail(nullptr, ROLLOUT_EINVAL, "n and target must be >= 1");
  hipError_t e = launch_length_rewards((hipStream_t)hip_stream, d_lengths, n, target, d_rewards,
                                       reinterpret_cast<long long*>(d_total_tokens));
  if (e != hipSuccess) return fail(nullptr, ROLLOUT_EDEVICE, std::string("length rewards: ") + hipGetErrorString(e));
  return ROLLOUT_OK;
}

rollout_status rollout_sync(rollout_ctx* ctx) {
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  int32_t flag = 0;
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream), "stream sync");
  reap_graphs(ctx, true);
  HIP_TRY(ctx, hipMemcpy(&flag, ctx->at(ctx->Lo.err), 4, hipMemcpyDeviceToHost), "error flag read");
  if (flag) {
    HIP_TRY(ctx, hipMemset(ctx->at(ctx->Lo.err), 0, 4), "error flag clear");
    std::string m = "device error flag";
    if (flag & 1) m += ": token id outside [0, vocab)";
    if (flag & 2) m += ": KV write outside the block pool";
    if (flag & 4) m += ": KV read outside the block pool";
    return fail(ctx, ROLLOUT_EINVAL, m);
  }
  return ROLLOUT_OK;
}

rollout_status rollout_export_weight(rollout_ctx* ctx, int32_t tensor_id, float* d_out) {
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!d_out) return fail(ctx, ROLLOUT_EINVAL, "out is NULL");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  const int lay = matrix_layout(D);
  hipError_t e;
  if (tensor_id == 0) {
    e = launch_export(ctx->stream, ctx->at(Lo.embed), D.dtype, wdesc(D.V, D.d, W_ROWMAJOR, FUSE_NONE, 0), 0, D.V, d_out);
  } else if (tensor_id == 2 + 9 * D.L) {
    e = launch_export(ctx->stream, ctx->at(Lo.lm_head), D.dtype, wdesc(D.V, D.d, lay, FUSE_NONE, 0), 0, D.V, d_out);
  } else if (tensor_id >= 1 && tensor_id < 1 + 9 * D.L) {
    const int l = (tensor_id - 1) / 9, slot = (tensor_id - 1) % 9;
    const Layer& y = Lo.layers[l];
    // int4 projections export their dequantised values (q - z) * s, rounded once to fp32
    auto exp = [&](const void* src, const WeightDesc& w, int which, int rows) {
      return D.wq4 ? launch_export_q4(ctx->stream, src, w, which, rows, d_out)
                   : launch_export(ctx->stream, src, D.dtype, w, which, rows, d_out);
    };
    switch (slot) {
      case 1: case 2: case 3:
        e = exp(ctx->at(y.wqkv), wdesc(D.nqkv, D.d, lay, FUSE_QKV, 0, 0, 0, D.qd, D.kvd), slot - 1,
                slot == 1 ? D.qd : D.kvd);
        break;
      case 4: e = exp(ctx->at(y.wo), wdesc(D.d, D.qd, lay, FUSE_NONE, 0), 0, D.d); break;
      case 6: case 7: e = exp(ctx->at(y.wgu), wdesc(2 * D.ff, D.d, lay, FUSE_GU, 0), slot - 6, D.ff); break;
      case 8: e = exp(ctx->at(y.wdown), wdesc(D.d, D.ff, lay, FUSE_NONE, 0), 0, D.d); break;
      default: return fail(ctx, ROLLOUT_EINVAL, "tensor id names a norm gain, not a matrix");
    }
  } else {
    return fail(ctx, ROLLOUT_EINVAL, "tensor id out of range");
  }
  if (e != hipSuccess) return hip_fail(ctx, e, "export");
  return ROLLOUT_OK;
}

rollout_status rollout_profile_decode_step(rollout_ctx* ctx, const int32_t* d_tokens, float* d_logits,
                                           rollout_step_profile* out) {
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!out) return fail(ctx, ROLLOUT_EINVAL, "out is NULL");
  ctx->prof.recs.clear();
  ctx->prof.on = true;
  rollout_status r = rollout_decode_step(ctx, d_tokens, d_logits);
  ctx->prof.on = false;
  if (r) return r;
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream), "stream sync");
  std::memset(out, 0, sizeof(*out));
  for (const Prof::Rec& rec : ctx->prof.recs) {
    float ms = 0.f;
    HIP_TRY(ctx, hipEventElapsedTime(&ms, ctx->prof.ev[rec.e0], ctx->prof.ev[rec.e1]), "event time");
    out->ms[rec.cls] += ms;
    out->launches[rec.cls] += 1;
    out->bytes[rec.cls] += rec.bytes;
    out->flops[rec.cls] += rec.flops;
  }
  return ROLLOUT_OK;
}

rollout_status rollout_profile_projections(rollout_ctx* ctx, int32_t reps, float* d_logits,
                                           rollout_projection_profile* out) {
  if (!ctx) return fail(nullptr, ROLLOUT_EINVAL, "ctx is NULL");
  if (!out || !d_logits || reps < 1) return fail(ctx, ROLLOUT_EINVAL, "out and logits must be non-NULL, reps >= 1");
  if (!ctx->wave) return fail(ctx, ROLLOUT_ESTATE, "no wave (prefill first)");
  const Dims& D = ctx->D;
  const Layout& Lo = ctx->Lo;
  const int M = ctx->S;
  if (D.wq4 && M > kSwigluMaxRows)
    return fail(ctx, ROLLOUT_EINVAL, "int4 batches over " + std::to_string(kSwigluMaxRows) +
                                         " rows dequantise before their GEMMs: not one launch per projection");
  const bool fused = D.dtype == ROLLOUT_DTYPE_BF16;
  void* a = ctx->at(Lo.a);
  void* o = ctx->at(Lo.o);
  void* h = ctx->at(Lo.h);
  float* part = ctx->at<float>(Lo.part);
  const double eb = (double)elem_bytes(D.dtype);
  auto wbytes = [&](int N, int K) {
    return D.wq4 ? (double)(q4_code_bytes(N, K) + q4_sz_bytes(N, K)) : (double)N * K * eb;
  };
  double bytes = 0.0, flops = 0.0;
  int launches = 0;
  // the projection launches of forward_layers and enqueue_decode at M = S rows, in step order
  auto enqueue = [&]() -> rollout_status {
    int s = 0;
    rollout_status r;
    for (int l = 0; l < D.L; ++l) {
      const Layer& y = Lo.layers[l];
      if ((r = proj(ctx, a, ctx->at(y.wqkv), part, M, D.nqkv, D.d, &s))) return r;
      if ((r = proj(ctx, o, ctx->at(y.wo), part, M, D.d, D.qd, &s))) return r;
      if (fused) {
        if ((r = gemm_swiglu(ctx, a, ctx->at(y.wgu), M, 2 * D.ff, D.d, h))) return r;
      } else {
        if ((r = proj(ctx, a, ctx->at(y.wgu), part, M, 2 * D.ff, D.d, &s))) return r;
      }
      if ((r = proj(ctx, h, ctx->at(y.wdown), part, M, D.d, D.ff, &s))) return r;
    }
    return gemm(ctx, a, ctx->at(Lo.lm_head), d_logits, M, D.V, D.d, 1, &s);
  };
  for (int l = 0; l < D.L; ++l) {
    bytes += wbytes(D.nqkv, D.d) + (double)M * D.d * eb + (double)M * D.nqkv * 4;
    bytes += wbytes(D.d, D.qd) + (double)M * D.qd * eb + (double)M * D.d * 4;
    bytes += wbytes(2 * D.ff, D.d) + (double)M * D.d * eb + (fused ? (double)M * D.ff * eb : (double)M * 2 * D.ff * 4);
    bytes += wbytes(D.d, D.ff) + (double)M * D.ff * eb + (double)M * D.d * 4;
    flops += 2.0 * M * ((double)D.nqkv * D.d + (double)D.d * D.qd + 2.0 * D.ff * D.d + (double)D.d * D.ff);
    launches += 4;
  }
  bytes += (double)D.V * D.d * eb + (double)M * D.d * eb + (double)M * D.V * 4;
  flops += 2.0 * M * (double)D.V * D.d;
  launches += 1;
  Range range("rollout_profile_projections");
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  HIP_TRY(ctx, hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal), "begin capture");
  rollout_status r = enqueue();
  hipError_t ce = hipStreamEndCapture(ctx->stream, &graph);
  if (r) {
    if (graph) hipGraphDestroy(graph);
    return r;
  }
  if (ce != hipSuccess) return hip_fail(ctx, ce, "end capture");
  hipError_t e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (e != hipSuccess) return hip_fail(ctx, e, "graph instantiate");
  hipEvent_t e0 = nullptr, e1 = nullptr;
  e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipGraphLaunch(exec, ctx->stream);  // warm-up replay
  if (e == hipSuccess) e = hipEventRecord(e0, ctx->stream);
  for (int i = 0; i < reps && e == hipSuccess; ++i) e = hipGraphLaunch(exec, ctx->stream);
  if (e == hipSuccess) e = hipEventRecord(e1, ctx->stream);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  hipStreamSynchronize(ctx->stream);
  hipGraphExecDestroy(exec);
  if (e0) hipEventDestroy(e0);
  if (e1) hipEventDestroy(e1);
  if (e != hipSuccess) return hip_fail(ctx, e, "projection replay");
  out->launches = launches;
  out->avg_us = (double)ms * 1e3 / ((double)reps * launches);
  out->bytes_per_launch = bytes / launches;
  out->flops_per_launch = flops / launches;
  return ROLLOUT_OK;
}

}  // extern "C"
