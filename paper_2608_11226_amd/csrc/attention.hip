// Paged grouped-query attention over the KV cache.
//
// Every query row attends to keys 0 .. pos of its sequence (causal), with the
// 1/sqrt(hd) scale and a max-subtracted softmax (online form: running max and
// running sum, rescaled as new keys arrive).
//
// bf16 path, head_dim 64 or 128: one workgroup of NW waves per (row, KV
// head), covering the whole context.  All query heads of the KV head's group
// ride in one MFMA (up to 16 heads): with the scores computed transposed,
// S^T = K Q^T (16 tokens x 16 heads per v_mfma_f32_16x16x32_bf16 step over
// hd), each lane holds the scores of one head for four tokens, which is
// exactly the B-operand layout of the P V product, so O^T = V^T P^T
// (v_mfma_f32_16x16x16_bf16, one per 16 output dimensions) consumes the
// softmaxed tile straight from registers.  Softmax statistics need two
// cross-lane shuffles per 16-token tile.  Wave w takes tiles w, w+NW, ...
// of the context and keeps the next tile's K/V loads in flight while it
// computes the current one; at the end the waves merge their (max, sum,
// output) states through LDS and write the normalised output directly in the
// O-projection's operand layout, so no partial results leave the workgroup.
// K and V are read once per row and KV head.  P enters the MFMA as the sum of
// two bf16 terms (scores, softmax and accumulation are fp32).
//
// fp32 path (and head_dim 32): a VALU kernel split over the context that
// stages K/V tiles in LDS; a combine kernel merges its splits with
// log-sum-exp weights in split order.
//
// Cache layout: [layer][block][kv head][K: blk x hd | V: hd x blk] (kv_offset).
#include <cstdlib>

#include "internal.h"

namespace rollout {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef short short8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

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

__device__ __forceinline__ short f2bs(float f) { return (short)f32_to_bf16(f); }

// K (A operand) and V^T (A operand of P.V) fragments of one 16-token tile
template <int HD>
struct KVTile {
  bf16x8_t k[HD / 32];
  short4_t v[HD / 16];
};

// Loads one 16-token tile starting at tb.  Every load is issued unconditionally,
// with rows past the context clamped onto its last token (they are masked when
// the tile is used), so a wave can keep several tiles in flight without the
// compiler draining the load queue.  Block ids come from the LDS copy of the
// sequence's block table; an out-of-range id sets *bad and reads block 0.
template <int HD>
__device__ __forceinline__ void load_tile(KVTile<HD>& t, int tb, int t_end, int hh, int g, const int* s_tab, int blk,
                                          const uint16_t* kv, size_t block_stride, size_t layer_base,
                                          size_t blk_elems, int n_blocks, bool* bad) {
  const int tk = min(tb + hh, t_end - 1);            // key row supplied by this lane
  const int tv = min(tb + 4 * g, (t_end - 1) & ~3);  // four value tokens tv .. tv+3 (never straddle a block)
  int bk = s_tab[tk / blk], bv = s_tab[tv / blk];
  if ((unsigned)bk >= (unsigned)n_blocks) { *bad = true; bk = 0; }
  if ((unsigned)bv >= (unsigned)n_blocks) { *bad = true; bv = 0; }
  const uint16_t* kp = kv + (size_t)bk * block_stride + layer_base + (size_t)(tk % blk) * HD + 8 * g;
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) t.k[c] = *reinterpret_cast<const bf16x8_t*>(kp + 32 * c);
  const uint16_t* vp = kv + (size_t)bv * block_stride + layer_base + blk_elems + (tv % blk);
#pragma unroll
  for (int j = 0; j < HD / 16; ++j) t.v[j] = *reinterpret_cast<const short4_t*>(vp + (size_t)(16 * j + hh) * blk);
}

template <int HD>
__device__ __forceinline__ void attend_tile(KVTile<HD>& t, const bf16x8_t* qf, int tb, int t_end, int g, float scale,
                                            float& m_run, float& l_run, floatx4_t* o) {
  floatx4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(t.k[c], qf[c], s, 0, 0, 0);
  // s[i] = score of token tb + 4g + i for head lane%16; tokens past the context drop out here
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s[i] = (tb + 4 * g + i < t_end) ? s[i] * scale : -INFINITY;
    mx = fmaxf(mx, s[i]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(m_run, mx);
  const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
  float p[4], ps = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p[i] = (s[i] == -INFINITY) ? 0.f : expf(s[i] - m_new);
    ps += p[i];
  }
  ps += __shfl_xor(ps, 16, 64);
  ps += __shfl_xor(ps, 32, 64);
  l_run = l_run * alpha + ps;
  m_run = m_new;
  if (tb + 16 > t_end) {  // the clamped rows of the last tile may hold stale data: keep them out of the MFMA
    const int vm = t_end - (tb + 4 * g);
#pragma unroll
    for (int j = 0; j < HD / 16; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e >= vm) t.v[j][e] = 0;
  }
  // p enters the MFMA as hi + lo, two bf16 terms whose sum is p to about 2^-17 relative: a single bf16
  // rounding of p would be an extra rounding point, worth up to ~2.5e-2 in the logits at 7B width
  short4_t ph, pl;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ph[i] = f2bs(p[i]);
    pl[i] = f2bs(p[i] - __uint_as_float((uint32_t)(uint16_t)ph[i] << 16));
  }
#pragma unroll
  for (int j = 0; j < HD / 16; ++j) {
    o[j] *= alpha;
    o[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(t.v[j], ph, o[j], 0, 0, 0);
    o[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(t.v[j], pl, o[j], 0, 0, 0);
  }
}

// Two tiles per softmax update: one max and one sum reduction for 32 tokens, and P.V as one
// v_mfma_f32_16x16x32_bf16 per 16 output dimensions (twice the tokens of the 16x16x16 form at the same
// issue cost).  The 32 reduction indices of that MFMA are the lane's four tokens of tile a followed by its
// four tokens of tile c, in both operands: V^T is the two tiles' four-token fragments side by side and P
// is the two tiles' probabilities, exactly as the scores come out of the two QK^T products.
template <int HD>
__device__ __forceinline__ void mask_tail(KVTile<HD>& t, int tb, int t_end, int g) {
  if (tb + 16 > t_end) {  // the clamped rows of the last tile may hold stale data: keep them out of the MFMA
    const int vm = t_end - (tb + 4 * g);
#pragma unroll
    for (int j = 0; j < HD / 16; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e >= vm) t.v[j][e] = 0;
  }
}

template <int HD>
__device__ __forceinline__ void attend_pair(KVTile<HD>& ta, KVTile<HD>& tc, const bf16x8_t* qf, int tba, int tbc,
                                            int t_end, int g, float scale, float& m_run, float& l_run, floatx4_t* o) {
  floatx4_t sa = {0.f, 0.f, 0.f, 0.f}, sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) {
    sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ta.k[c], qf[c], sa, 0, 0, 0);
    sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tc.k[c], qf[c], sc, 0, 0, 0);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sa[i] = (tba + 4 * g + i < t_end) ? sa[i] * scale : -INFINITY;
    sc[i] = (tbc + 4 * g + i < t_end) ? sc[i] * scale : -INFINITY;
    mx = fmaxf(mx, fmaxf(sa[i], sc[i]));
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(m_run, mx);
  const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
  float p[8], ps = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p[i] = (sa[i] == -INFINITY) ? 0.f : expf(sa[i] - m_new);
    p[4 + i] = (sc[i] == -INFINITY) ? 0.f : expf(sc[i] - m_new);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) ps += p[i];
  ps += __shfl_xor(ps, 16, 64);
  ps += __shfl_xor(ps, 32, 64);
  l_run = l_run * alpha + ps;
  m_run = m_new;
  mask_tail<HD>(ta, tba, t_end, g);
  mask_tail<HD>(tc, tbc, t_end, g);
  // p as hi + lo, two bf16 terms (see attend_tile)
  short8_t ph, pl;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    ph[i] = f2bs(p[i]);
    pl[i] = f2bs(p[i] - __uint_as_float((uint32_t)(uint16_t)ph[i] << 16));
  }
  const bf16x8_t bh = __builtin_bit_cast(bf16x8_t, ph), bl = __builtin_bit_cast(bf16x8_t, pl);
#pragma unroll
  for (int j = 0; j < HD / 16; ++j) {
    const bf16x8_t v = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(ta.v[j], tc.v[j], 0, 1, 2, 3, 4, 5, 6, 7));
    o[j] *= alpha;
    o[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v, bh, o[j], 0, 0, 0);
    o[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v, bl, o[j], 0, 0, 0);
  }
}

// One pass of wave-strided tiles through a ring of DR tiles: tile k of this wave starts at first + STRIDE k.
// With pairs (U = 2), ring slots (d, d + 1) hold consecutive tiles of the wave and are attended together;
// the pair's two reloads then go out together, so no tile is in flight while a wave computes.  That pays
// where several waves share a SIMD (the one-group decode instance and the prefix pass, three workgroups
// per CU: 14B rollout +1.5%) and not at one wave per SIMD, which has nothing else to overlap (7B -0.6%;
// a ring of two pairs needs registers those instances do not have).
template <int HD, int DR, int U>
__device__ __forceinline__ void attend_ring(KVTile<HD>* ring, int n_w, int first, int STRIDE, int t_end, int hh, int g,
                                            const int* s_tab, int blk, const uint16_t* kv, size_t block_stride,
                                            size_t layer_base, size_t blk_elems, int n_blocks, bool* bad,
                                            const bf16x8_t* qf, float scale, float& m_run, float& l_run,
                                            floatx4_t* o) {
  constexpr int UU = DR % U == 0 ? U : 1;  // an odd ring attends single tiles
  for (int i = 0; i < n_w; i += DR) {
#pragma unroll
    for (int d = 0; d < DR; d += UU) {
      if (i + d < n_w) {
        if constexpr (UU == 2)
          attend_pair<HD>(ring[d], ring[d + 1], qf, first + STRIDE * (i + d), first + STRIDE * (i + d + 1), t_end, g,
                          scale, m_run, l_run, o);
        else
          attend_tile<HD>(ring[d], qf, first + STRIDE * (i + d), t_end, g, scale, m_run, l_run, o);
      }
#pragma unroll
      for (int u = 0; u < UU; ++u)
        load_tile<HD>(ring[d + u], first + STRIDE * min(i + d + u + DR, n_w - 1), t_end, hh, g, s_tab, blk, kv,
                      block_stride, layer_base, blk_elems, n_blocks, bad);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Decode rows may form their own q, k, v from the QKV projection's split-K
// partials (part[split][row][nqkv], summed in split order): rotary embedding
// on q and k, bf16 rounding, k and v appended to the cache.  The current token
// then enters the softmax as one more state beside the waves' states, so no
// wave reads the cache entry this workgroup is writing.
constexpr int kMaxQkvSplits = 16;  // most QKV split partials the attention kernel sums
constexpr int kQkvBatch = 8;       // of which the first this many are loaded with the block table
constexpr int kMaxTableBlocks = 16384;

struct AttnQKV {
  const float* part;  // NULL: q is read from the q buffer and the cache already holds the current token
  int splits;
  const float* rope_cos;
  const float* rope_sin;
  // shared-prefix decode (see k_attn_prefix): keys before t_begin are left to the prefix kernel, the
  // rotated q is kept in q_keep, and the unnormalised softmax state goes to st_o / st_ml
  int t_begin;
  uint16_t* q_keep;
  float* st_o;   // [row][head][HD]: sum of p * v relative to the state's max
  float* st_ml;  // [row][head][2]: max, sum of p
};

// ONE: every column group of the q/k/v formation fits one per thread ((nrep + 2) * HD / 4 <= NW * 64), so
// the partials of a single group are held (fewer registers, more workgroups per CU); else up to 16 query
// heads per KV head.  QBX: QKV split partials loaded with the block table (0: kQkvBatch, half for ONE); the
// launch takes 4 when the QKV projection has at most 4 splits, so no loads are spent on surplus partials.
template <int HD, int NW, int DR, bool FQ, bool SPLIT = false, bool ONE = false, int QBX = 0>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(ONE && NW == 4 ? 3 : 1)))
void k_attn_mfma(Dims D, const uint16_t* __restrict__ q,
                                                       uint16_t* __restrict__ kv, int n_blocks,
                                                       const int32_t* __restrict__ tables, int max_blocks, RowMap rm,
                                                       int R, int layer, AttnQKV Q, uint16_t* __restrict__ out,
                                                       int32_t* __restrict__ err) {
  constexpr int KC = HD / 32;  // QK^T k-steps
  constexpr int DT = HD / 16;  // P.V output tiles
  constexpr int NT = NW * 64;
  __shared__ float s_m[NW][16], s_l[NW][16];
  __shared__ float s_o[NW][16][HD + 4];
  __shared__ __align__(16) uint16_t s_q[FQ ? 16 : 1][HD];
  __shared__ float s_kv[FQ ? 2 : 1][HD];  // current token's k (rotated) and v, bf16 values
  __shared__ __align__(16) float s_raw[FQ ? 18 : 1][HD];  // split sums: q heads, then k, then v
  __shared__ float s_rope[FQ ? HD : 1];                   // cos (first half), sin (second half) at pos
  __shared__ float s_cur[16];             // current token's scaled score per head
  extern __shared__ int s_tab[];          // the sequence's block table (dynamic, max_blocks entries)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // XCD-aware order (workgroup b runs on XCD b % 8, and the grid is a multiple of 8): each XCD takes a
  // contiguous range of (row, KV head) items, so the rows of one group (or one prompt) -- which read the
  // same prompt KV blocks -- fetch them into one L2 instead of all eight
  const int item = (int)(blockIdx.x & 7) * (int)(gridDim.x >> 3) + (int)(blockIdx.x >> 3);
  if (item >= R * D.nkv) return;
  const int kvh = item % D.nkv;
  const int r = item / D.nkv;
  int seq, pos;
  row_place(rm, r, &seq, &pos);
  const int nrep = D.nh / D.nkv;
  const int hh = lane & 15, g = lane >> 4;
  const int blk = D.blk;
  const size_t blk_elems = (size_t)blk * HD;
  const size_t kv_head_stride = 2 * blk_elems;
  const size_t layer_base = kv_offset(layer, 0, kvh, n_blocks, D.nkv, kv_head_stride);
  const size_t block_stride = (size_t)D.nkv * kv_head_stride;
  const int32_t* trow = tables + (size_t)seq * max_blocks;
  const float scale = 1.0f / sqrtf((float)HD);
  bf16x8_t zero8;
#pragma unroll
  for (int e = 0; e < 8; ++e) zero8[e] = (__bf16)0.0f;

  int t_end = pos + 1;  // keys read from the cache
  if constexpr (FQ) t_end = pos;
  // One round trip for the block table, the row's rotary factors and the first QB QKV split
  // partials of this thread's column groups (float4 groups; every load in flight at once).  The table
  // goes to LDS as soon as it arrives and the first K/V tiles go out before the partials are summed, so
  // the waits on the partials (and the LDS-only barriers after them) leave the tile loads in flight.
  const int ntab = (t_end + blk - 1) / blk;
  constexpr int GI = ONE ? 1 : (18 * (HD / 4) + NT - 1) / NT;  // column groups per thread (nrep <= 16)
  constexpr int QB = QBX ? QBX : (ONE ? kQkvBatch / 2 : kQkvBatch);  // partials loaded with the table
  const int ng = (nrep + 2) * (HD / 4);
  const float* pr = FQ ? Q.part + (size_t)r * D.nqkv : nullptr;
  const size_t split_stride = (size_t)R * D.nqkv;
  const int s1 = FQ ? min(Q.splits, QB) : 1;
  float4 pv[FQ ? GI : 1][QB];
  auto group_col = [&](int gi) {
    const int slot = gi / (HD / 4), i4 = (gi % (HD / 4)) * 4;
    return (slot < nrep ? (kvh * nrep + slot) * HD : D.qd + (slot - nrep) * D.kvd + kvh * HD) + i4;
  };
  if constexpr (FQ) {
    // Every load here is unconditional (indices clamped; the clamped threads store the same value to
    // the same LDS word as their neighbour), so the compiler's waits stay per load: the table store
    // waits for the table alone and the partials stay in flight behind it.
    constexpr int half = HD / 2;
    for (int i = tid + NT; i < ntab; i += NT) s_tab[i] = trow[i];  // contexts of more than NT blocks
    const int ti = min(tid, max(ntab - 1, 0));
    const int tab0 = trow[ti];
    __builtin_amdgcn_sched_barrier(0);
    const int tr = min(tid, HD - 1);
    const float rope0 = tr < half ? Q.rope_cos[(size_t)pos * half + tr] : Q.rope_sin[(size_t)pos * half + tr - half];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int it = 0; it < GI; ++it) {
      const int c = group_col(min(tid + it * NT, ng - 1));
#pragma unroll
      for (int sp = 0; sp < QB; ++sp)
        pv[it][sp] = *reinterpret_cast<const float4*>(pr + (size_t)min(sp, s1 - 1) * split_stride + c);
    }
    __builtin_amdgcn_sched_barrier(0);
    s_tab[ti] = tab0;
    s_rope[tr] = rope0;
    lds_barrier();
  } else {
    for (int i = tid; i < ntab; i += NT) s_tab[i] = trow[i];
    __syncthreads();
  }

  // wave w: tiles w, w + NW, ...  They pass through a ring of DR tiles in
  // registers: while one is attended, the next DR - 1 are loading.  The first
  // DR loads go out before q/k/v are rotated, so they overlap that work.
  constexpr int STRIDE = 16 * NW;
  const int first = (SPLIT ? Q.t_begin : 0) + 16 * wave;
  const int n_w = t_end > first ? (t_end - first + STRIDE - 1) / STRIDE : 0;
  bool bad = false;
  KVTile<HD> ring[DR];
  // unconditional, so that no branch sits between these loads and the waits for the partials: a wave
  // with no tile here (n_w == 0) reloads tile 0's clamped rows and never uses them
  if (FQ || n_w > 0) {
#pragma unroll
    for (int d = 0; d < DR; ++d) {
      load_tile<HD>(ring[d], first + STRIDE * max(0, min(d, n_w - 1)), max(t_end, 1), hh, g, s_tab, blk, kv,
                    block_stride, layer_base, blk_elems, n_blocks, &bad);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (n_w == 0) bad = false;
  }

  // Q^T as the B operand: lane supplies head hh, dimensions 32c + 8g .. +7
  bf16x8_t qf[KC];
  if constexpr (FQ) {
    // split sums in split order: the first QB from registers (threads past the last column
    // group store group ng - 1 again), then any further partials, loaded now
    float4 acc[GI];
#pragma unroll
    for (int it = 0; it < GI; ++it) {
      acc[it] = pv[it][0];
#pragma unroll
      for (int sp = 1; sp < QB; ++sp) {
        if (sp < s1) {
          acc[it].x += pv[it][sp].x;
          acc[it].y += pv[it][sp].y;
          acc[it].z += pv[it][sp].z;
          acc[it].w += pv[it][sp].w;
        }
      }
    }
    for (int sp = QB; sp < Q.splits; ++sp) {
#pragma unroll
      for (int it = 0; it < GI; ++it) {
        const float4 t = *reinterpret_cast<const float4*>(pr + (size_t)sp * split_stride + group_col(min(tid + it * NT, ng - 1)));
        acc[it].x += t.x;
        acc[it].y += t.y;
        acc[it].z += t.z;
        acc[it].w += t.w;
      }
    }
#pragma unroll
    for (int it = 0; it < GI; ++it) {
      const int gi = min(tid + it * NT, ng - 1);
      *reinterpret_cast<float4*>(&s_raw[gi / (HD / 4)][(gi % (HD / 4)) * 4]) = acc[it];
    }
    lds_barrier();
    // rotary embedding of q and k, bf16 rounding, cache append of k and v
    constexpr int half = HD / 2;
    const float* cs = s_rope;
    const float* sn = s_rope + half;
    const int b = trow[pos / blk];
    const bool bok = b >= 0 && b < n_blocks;
    uint16_t* kdst = kv + (size_t)(bok ? b : 0) * block_stride + layer_base;
    const int npair = (nrep + 1) * half;
    for (int it = tid; it < npair + HD; it += NT) {
      if (it < npair) {
        const int h = it / half, i = it - h * half;
        const float x1 = s_raw[h][i], x2 = s_raw[h][i + half];
        const uint16_t b1 = f32_to_bf16(x1 * cs[i] - x2 * sn[i]);
        const uint16_t b2 = f32_to_bf16(x2 * cs[i] + x1 * sn[i]);
        if (h < nrep) {
          s_q[h][i] = b1;
          s_q[h][i + half] = b2;
          if constexpr (SPLIT) {
            uint16_t* qk = Q.q_keep + (size_t)r * D.qd + (size_t)(kvh * nrep + h) * HD;
            qk[i] = b1;
            qk[i + half] = b2;
          }
        } else {
          s_kv[0][i] = bf16_to_f32(b1);
          s_kv[0][i + half] = bf16_to_f32(b2);
          if (bok) {
            kdst[(size_t)(pos % blk) * HD + i] = b1;
            kdst[(size_t)(pos % blk) * HD + i + half] = b2;
          }
        }
      } else {
        const int i = it - npair;
        const uint16_t bv = f32_to_bf16(s_raw[nrep + 1][i]);
        s_kv[1][i] = bf16_to_f32(bv);
        if (bok) kdst[blk_elems + (size_t)i * blk + pos % blk] = bv;
      }
    }
    if (!bok && tid == 0) atomicOr(err, 2);
    for (int it = tid; it < (16 - nrep) * HD; it += NT) s_q[nrep + it / HD][it % HD] = 0;
    lds_barrier();  // LDS only: the tile loads and the cache stores stay in flight
#pragma unroll
    for (int c = 0; c < KC; ++c) qf[c] = *reinterpret_cast<const bf16x8_t*>(&s_q[hh][32 * c + 8 * g]);
    // score of the current token: one wave per head
    for (int h = wave; h < nrep; h += NW) {
      float acc = 0.f;
      for (int d = lane; d < HD; d += 64) acc += bf16_to_f32(s_q[h][d]) * s_kv[0][d];
      acc = wave_sum(acc);
      if (lane == 0) s_cur[h] = acc * scale;
    }
  } else {
    const uint16_t* qrow = q + (size_t)r * D.qd + (size_t)(kvh * nrep + hh) * HD;
#pragma unroll
    for (int c = 0; c < KC; ++c)
      qf[c] = hh < nrep ? *reinterpret_cast<const bf16x8_t*>(qrow + 32 * c + 8 * g) : zero8;
  }
  float m_run = -INFINITY, l_run = 0.f;
  floatx4_t o[DT];
#pragma unroll
  for (int j = 0; j < DT; ++j) o[j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  if (n_w > 0)
    attend_ring<HD, DR, ONE ? 2 : 1>(ring, n_w, first, STRIDE, t_end, hh, g, s_tab, blk, kv, block_stride,
                                     layer_base, blk_elems, n_blocks, &bad, qf, scale, m_run, l_run, o);
  if (bad) atomicOr(err, 4);

  // merge the waves: o[j][i] is head hh at dimension 16 j + 4 g + i
  if (g == 0) {
    s_m[wave][hh] = m_run;
    s_l[wave][hh] = l_run;
  }
#pragma unroll
  for (int j = 0; j < DT; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) s_o[wave][hh][16 * j + 4 * g + i] = o[j][i];
  __syncthreads();
  // each thread finishes 8 consecutive dimensions of one head
  const int Mb = (R + 15) >> 4;
  for (int item = tid; item < nrep * (HD / 8); item += NT) {
    const int h = item / (HD / 8), d0 = (item % (HD / 8)) * 8;
    float mx = FQ ? s_cur[h] : -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      if (s_l[w][h] > 0.f) mx = fmaxf(mx, s_m[w][h]);
    float num[8] = {0, 0, 0, 0, 0, 0, 0, 0}, den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (s_l[w][h] > 0.f) {
        const float wt = expf(s_m[w][h] - mx);
        den += wt * s_l[w][h];
#pragma unroll
        for (int e = 0; e < 8; ++e) num[e] += wt * s_o[w][h][d0 + e];
      }
    }
    if constexpr (FQ) {
      const float wt = expf(s_cur[h] - mx);
      den += wt;
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] += wt * s_kv[1][d0 + e];
    }
    if constexpr (SPLIT) {
      const size_t hr = (size_t)r * D.nh + kvh * nrep + h;
      float4* so = reinterpret_cast<float4*>(Q.st_o + hr * HD + d0);
      so[0] = make_float4(num[0], num[1], num[2], num[3]);
      so[1] = make_float4(num[4], num[5], num[6], num[7]);
      if (d0 == 0) {
        Q.st_ml[hr * 2] = mx;
        Q.st_ml[hr * 2 + 1] = den;
      }
    } else {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = den > 0.f ? num[e] / den : 0.f;
      st8(out, xoff(out, r, (kvh * nrep + h) * HD + d0, D.qd, Mb), v);
    }
  }
}

// Shared-prefix (group-aware) decode attention.  The G sequences of a group
// share the physical KV blocks of their prompt's full blocks, tokens
// [0, p_shared).  One workgroup per (group, KV head, block of 16 query
// columns), a column being one (sequence, query head) pair of the group, reads
// each shared K/V tile once for all 16 columns (the workgroups of one group and
// KV head are placed on one XCD, so their tile reads meet in its L2), merges
// its waves' softmax states with the state the suffix pass left for the
// column (keys p_shared .. pos, current token included) and writes the
// normalised output in the O-projection operand layout.
template <int HD, int NW, int DR>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW == 4 ? 3 : 1))) void k_attn_prefix(Dims D, const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ kv, int n_blocks,
                                                         const int32_t* __restrict__ tables, int max_blocks,
                                                         int layer, int seq0, int G, int n_groups, int p_shared,
                                                         const float* __restrict__ st_o,
                                                         const float* __restrict__ st_ml, int R,
                                                         uint16_t* __restrict__ out, int32_t* __restrict__ err) {
  constexpr int KC = HD / 32, DT = HD / 16, NT = NW * 64;
  __shared__ float s_m[NW][16], s_l[NW][16];
  __shared__ float s_o[NW][16][HD + 4];
  extern __shared__ int s_tab[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrep = D.nh / D.nkv;
  const int QB = (G * nrep + 15) / 16;
  // workgroup order: the QB column blocks of one (group, KV head) share an XCD (workgroup b runs on XCD b % 8)
  const int b = blockIdx.x;
  const int gk = (b / (8 * QB)) * 8 + b % 8, qb = (b / 8) % QB;
  if (gk >= n_groups * D.nkv) return;
  const int grp = gk / D.nkv, kvh = gk % D.nkv;
  const int hh = lane & 15, g = lane >> 4;
  const int blk = D.blk;
  const size_t blk_elems = (size_t)blk * HD;
  const size_t kv_head_stride = 2 * blk_elems;
  const size_t layer_base = kv_offset(layer, 0, kvh, n_blocks, D.nkv, kv_head_stride);
  const size_t block_stride = (size_t)D.nkv * kv_head_stride;
  const int32_t* trow = tables + (size_t)(seq0 + grp * G) * max_blocks;
  for (int i = tid; i < p_shared / blk; i += NT) s_tab[i] = trow[i];
  // this lane's query column: (row grp*G + c / nrep, head kvh*nrep + c % nrep)
  const int c = 16 * qb + hh;
  const bool cval = c < G * nrep;
  const int row = grp * G + (cval ? c / nrep : 0), head = kvh * nrep + (cval ? c % nrep : 0);
  bf16x8_t qf[KC];
  {
    bf16x8_t zero8;
#pragma unroll
    for (int e = 0; e < 8; ++e) zero8[e] = (__bf16)0.0f;
    const uint16_t* qrow = q + (size_t)row * D.qd + (size_t)head * HD;
#pragma unroll
    for (int cc = 0; cc < KC; ++cc) qf[cc] = cval ? *reinterpret_cast<const bf16x8_t*>(qrow + 32 * cc + 8 * g) : zero8;
  }
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)HD);
  float m_run = -INFINITY, l_run = 0.f;
  floatx4_t o[DT];
#pragma unroll
  for (int j = 0; j < DT; ++j) o[j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  constexpr int STRIDE = 16 * NW;
  const int first = 16 * wave;
  const int t_end = p_shared;
  const int n_w = t_end > first ? (t_end - first + STRIDE - 1) / STRIDE : 0;
  bool bad = false;
  if (n_w > 0) {
    KVTile<HD> ring[DR];
#pragma unroll
    for (int d = 0; d < DR; ++d) {
      load_tile<HD>(ring[d], first + STRIDE * min(d, n_w - 1), t_end, hh, g, s_tab, blk, kv, block_stride, layer_base,
                    blk_elems, n_blocks, &bad);
      __builtin_amdgcn_sched_barrier(0);
    }
    attend_ring<HD, DR, 2>(ring, n_w, first, STRIDE, t_end, hh, g, s_tab, blk, kv, block_stride, layer_base,
                           blk_elems, n_blocks, &bad, qf, scale, m_run, l_run, o);
  }
  if (bad) atomicOr(err, 4);
  if (g == 0) {
    s_m[wave][hh] = m_run;
    s_l[wave][hh] = l_run;
  }
#pragma unroll
  for (int j = 0; j < DT; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) s_o[wave][hh][16 * j + 4 * g + i] = o[j][i];
  __syncthreads();
  // each thread finishes 8 consecutive dimensions of one column, merging the suffix state
  const int Mb = (R + 15) >> 4;
  for (int item = tid; item < 16 * (HD / 8); item += NT) {
    const int cl = item / (HD / 8), d0 = (item % (HD / 8)) * 8;
    const int cc = 16 * qb + cl;
    if (cc >= G * nrep) continue;
    const int rr = grp * G + cc / nrep, hd_ = kvh * nrep + cc % nrep;
    const size_t hr = (size_t)rr * D.nh + hd_;
    const float sm = st_ml[hr * 2], sl = st_ml[hr * 2 + 1];
    float mx = sl > 0.f ? sm : -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      if (s_l[w][cl] > 0.f) mx = fmaxf(mx, s_m[w][cl]);
    float num[8], den = 0.f;
    {
      const float wt = sl > 0.f ? expf(sm - mx) : 0.f;
      const float4* so = reinterpret_cast<const float4*>(st_o + hr * HD + d0);
      const float4 a0 = so[0], a1 = so[1];
      den = wt * sl;
      num[0] = wt * a0.x; num[1] = wt * a0.y; num[2] = wt * a0.z; num[3] = wt * a0.w;
      num[4] = wt * a1.x; num[5] = wt * a1.y; num[6] = wt * a1.z; num[7] = wt * a1.w;
    }
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (s_l[w][cl] > 0.f) {
        const float wt = expf(s_m[w][cl] - mx);
        den += wt * s_l[w][cl];
#pragma unroll
        for (int e = 0; e < 8; ++e) num[e] += wt * s_o[w][cl][d0 + e];
      }
    }
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = den > 0.f ? num[e] / den : 0.f;
    st8(out, xoff(out, rr, hd_ * HD + d0, D.qd, Mb), v);
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_valu(Dims D, const T* __restrict__ q, const T* __restrict__ kv,
                                                   int n_blocks, const int32_t* __restrict__ tables, int max_blocks,
                                                   RowMap rm, int splits, int split_tokens, int layer,
                                                   float* __restrict__ opart, float* __restrict__ ml,
                                                   int32_t* __restrict__ err) {
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
  const int nrep = D.nh / D.nkv;
  const int t_begin = split * split_tokens;
  const int t_end = min(pos + 1, t_begin + split_tokens);
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
        const size_t base = kv_offset(layer, b, kvh, n_blocks, D.nkv, 2 * blk_elems);
        kval = ldf(kv, base + (size_t)(tok % D.blk) * HD + dd);
        vval = ldf(kv, base + blk_elems + (size_t)dd * D.blk + (tok % D.blk));
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

// out (O-projection operand layout) = sum_s w_s o_s / sum_s w_s l_s, w_s = exp(m_s - max m)
template <typename T>
__global__ __launch_bounds__(64) void k_attn_combine(const float* __restrict__ opart, const float* __restrict__ ml,
                                                     int R, int nh, int splits, int hd, T* __restrict__ out) {
  const int r = blockIdx.x;
  const int g = blockIdx.y * 64 + threadIdx.x;  // group of 8 output columns
  const int qd = nh * hd;
  if (g >= (qd >> 3)) return;
  const int h = (g * 8) / hd, d0 = (g * 8) % hd;
  const size_t rh = (size_t)r * nh + h;
  float mx = -INFINITY;
  for (int s = 0; s < splits; ++s)
    if (ml[(rh * splits + s) * 2 + 1] > 0.f) mx = fmaxf(mx, ml[(rh * splits + s) * 2]);
  float num[8] = {0, 0, 0, 0, 0, 0, 0, 0}, den = 0.f;
  for (int s = 0; s < splits; ++s) {
    const float m = ml[(rh * splits + s) * 2], l = ml[(rh * splits + s) * 2 + 1];
    if (l > 0.f) {
      const float w = expf(m - mx);
      float v[8];
      ld8(opart, (rh * splits + s) * hd + d0, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] += w * v[e];
      den += w * l;
    }
  }
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = den > 0.f ? num[e] / den : 0.f;
  st8(out, xoff(out, r, g * 8, qd, (R + 15) >> 4), o);
}


// whether the q/k/v column groups of one (row, KV head) fit one per thread of an NW-wave workgroup
bool one_group(const Dims& D, int nw) { return (D.nh / D.nkv + 2) * (D.hd / 4) <= nw * 64; }

bool mfma_attention(const Dims& D) { return D.dtype == ROLLOUT_DTYPE_BF16 && (D.hd == 128 || D.hd == 64); }

}  // namespace

// Waves per decode-attention workgroup: four once there is a workgroup per CU.  With that many
// workgroups the KV stream runs near the HBM rate either way, and four waves halve the merge of the
// waves' softmax states (7B, 256 workgroups: decode +1.6% over eight).  Eight for smaller grids, which
// need the loads of more waves in flight.  ROLLOUT_ATTN_WAVES=4 or 8 forces the choice (read per call).
int attn_waves(int n_workgroups) {
  const char* v = std::getenv("ROLLOUT_ATTN_WAVES");
  const int forced = v ? std::atoi(v) : 0;
  if (forced == 4 || forced == 8) return forced;
  return n_workgroups >= 256 ? 4 : 8;
}

// k_attn_mfma grid: one workgroup per (row, KV head), rounded up to a multiple of the 8 XCDs
static unsigned attn_grid(int R, const Dims& D) { return (unsigned)(R * D.nkv + 7) / 8 * 8; }

bool attention_shares_prefix(const Dims& D) { return mfma_attention(D); }

hipError_t launch_attention_shared(hipStream_t s, const Dims& D, void* kv_pool, int n_blocks, const int32_t* tables,
                                   int max_blocks, RowMap rm, int R, int layer, int G, int p_shared, void* q_keep,
                                   float* st_o, float* st_ml, void* out, int32_t* err, const float* qkv_part,
                                   int qkv_splits, const float* rope_cos, const float* rope_sin) {
  if (R <= 0) return hipSuccess;
  if (!mfma_attention(D) || rm.P != 0 || G < 1 || R % G || p_shared < D.blk || p_shared % D.blk ||
      qkv_splits < 1 || qkv_splits > kMaxQkvSplits || max_blocks > kMaxTableBlocks)
    return hipErrorInvalidValue;
  const AttnQKV Q{qkv_part, qkv_splits, rope_cos, rope_sin, p_shared, (uint16_t*)q_keep, st_o, st_ml};
  uint16_t* kk = (uint16_t*)kv_pool;
  uint16_t* oo = (uint16_t*)out;
  // suffix: keys p_shared .. pos of every row, q/k/v formed, state kept
  const size_t tab_bytes = (size_t)max_blocks * 4;
  const dim3 sgrid(attn_grid(R, D));
#define ROLLOUT_SUFFIX(HD, NW)                                                                                       \
  do {                                                                                                               \
    if (one_group(D, NW))                                                                                            \
      hipLaunchKernelGGL((k_attn_mfma<HD, NW, 2, true, true, true>), sgrid, dim3(NW * 64), tab_bytes, s, D,          \
                         (const uint16_t*)nullptr, kk, n_blocks, tables, max_blocks, rm, R, layer, Q, oo, err);      \
    else                                                                                                             \
      hipLaunchKernelGGL((k_attn_mfma<HD, NW, 2, true, true>), sgrid, dim3(NW * 64), tab_bytes, s, D,                \
                         (const uint16_t*)nullptr, kk, n_blocks, tables, max_blocks, rm, R, layer, Q, oo, err);      \
  } while (0)
  const int nws = attn_waves(R * D.nkv);
  if (D.hd == 128) {
    if (nws == 4) ROLLOUT_SUFFIX(128, 4);
    else ROLLOUT_SUFFIX(128, 8);
  } else {
    if (nws == 4) ROLLOUT_SUFFIX(64, 4);
    else ROLLOUT_SUFFIX(64, 8);
  }
#undef ROLLOUT_SUFFIX
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // prefix: the group's shared prompt blocks once per (group, KV head, 16 query columns), then the merge
  const int n_groups = R / G, nrep = D.nh / D.nkv, QB = (G * nrep + 15) / 16;
  const int gk = n_groups * D.nkv;
  const dim3 grid((unsigned)((gk + 7) / 8 * 8 * QB));
  const size_t ptab = (size_t)(p_shared / D.blk) * 4;
#define ROLLOUT_PREFIX(HD, NW)                                                                                       \
  hipLaunchKernelGGL((k_attn_prefix<HD, NW, 2>), grid, dim3(NW * 64), ptab, s, D, (const uint16_t*)q_keep,           \
                     (const uint16_t*)kv_pool, n_blocks, tables, max_blocks, layer, rm.seq0, G, n_groups, p_shared, \
                     (const float*)st_o, (const float*)st_ml, R, oo, err)
  const int nwp = attn_waves(gk * QB);
  if (D.hd == 128) {
    if (nwp == 4) ROLLOUT_PREFIX(128, 4);
    else ROLLOUT_PREFIX(128, 8);
  } else {
    if (nwp == 4) ROLLOUT_PREFIX(64, 4);
    else ROLLOUT_PREFIX(64, 8);
  }
#undef ROLLOUT_PREFIX
  return hipGetLastError();
}

int attn_splits(int max_ctx, int* split_tokens) {
  const int st = 256;
  *split_tokens = st;
  const int s = (max_ctx + st - 1) / st;
  return s < 1 ? 1 : s;
}

bool attention_forms_qkv(const Dims& D) { return mfma_attention(D); }

hipError_t launch_attention(hipStream_t s, const Dims& D, const void* q, void* kv_pool, int n_blocks,
                            const int32_t* tables, int max_blocks, RowMap rm, int R, int splits, int split_tokens,
                            int layer, float* opart, float* ml, void* out, int32_t* err, const float* qkv_part,
                            int qkv_splits, const float* rope_cos, const float* rope_sin) {
  if (R <= 0) return hipSuccess;
  if (qkv_part && (!mfma_attention(D) || rm.P != 0 || qkv_splits < 1 || qkv_splits > kMaxQkvSplits))
    return hipErrorInvalidValue;
  if (mfma_attention(D)) {
    if (max_blocks > kMaxTableBlocks) return hipErrorInvalidValue;  // the block table is staged in LDS
    const int nw = attn_waves(R * D.nkv);
    static const int dr = [] {
      const char* v = std::getenv("ROLLOUT_ATTN_RING");
      const int d = v ? std::atoi(v) : 2;
      return d == 3 || d == 4 ? d : 2;
    }();
    const dim3 grid(attn_grid(R, D));
    const AttnQKV Q{qkv_part, qkv_splits, rope_cos, rope_sin, 0, nullptr, nullptr, nullptr};
    const uint16_t* qq = (const uint16_t*)q;
    uint16_t* kk = (uint16_t*)kv_pool;
    uint16_t* oo = (uint16_t*)out;
    const size_t tab_bytes = (size_t)max_blocks * 4;
#define ROLLOUT_MFMA_ATTN(HD, NW, DR, FQ)                                                                              \
  do {                                                                                                                 \
    if constexpr (FQ && DR == 2) {                                                                                     \
      if (one_group(D, NW)) {                                                                                          \
        hipLaunchKernelGGL((k_attn_mfma<HD, NW, DR, FQ, false, true>), grid, dim3(NW * 64), tab_bytes, s, D, qq, kk,   \
                           n_blocks, tables, max_blocks, rm, R, layer, Q, oo, err);                                    \
        break;                                                                                                         \
      }                                                                                                                \
    }                                                                                                                  \
    if constexpr (FQ && DR == 2 && NW == 4) {                                                                      \
      if (qkv_splits <= 4) {                                                                                           \
        hipLaunchKernelGGL((k_attn_mfma<HD, NW, DR, FQ, false, false, 4>), grid, dim3(NW * 64), tab_bytes, s, D, qq,   \
                           kk, n_blocks, tables, max_blocks, rm, R, layer, Q, oo, err);                                \
        break;                                                                                                         \
      }                                                                                                                \
    }                                                                                                                  \
    hipLaunchKernelGGL((k_attn_mfma<HD, NW, DR, FQ>), grid, dim3(NW * 64), tab_bytes, s, D, qq, kk, n_blocks, tables,  \
                       max_blocks, rm, R, layer, Q, oo, err);                                                          \
  } while (0)
#define ROLLOUT_MFMA_ATTN_NW(HD, FQ)                    \
  do {                                                  \
    if (nw == 4) ROLLOUT_MFMA_ATTN(HD, 4, 2, FQ);         \
    else if (dr == 3) ROLLOUT_MFMA_ATTN(HD, 8, 3, FQ);    \
    else if (dr == 4) ROLLOUT_MFMA_ATTN(HD, 8, 4, FQ);    \
    else ROLLOUT_MFMA_ATTN(HD, 8, 2, FQ);                 \
  } while (0)
    if (D.hd == 128) {
      if (qkv_part) ROLLOUT_MFMA_ATTN_NW(128, true);
      else ROLLOUT_MFMA_ATTN_NW(128, false);
    } else {
      if (qkv_part) ROLLOUT_MFMA_ATTN_NW(64, true);
      else ROLLOUT_MFMA_ATTN_NW(64, false);
    }
#undef ROLLOUT_MFMA_ATTN_NW
#undef ROLLOUT_MFMA_ATTN
    return hipGetLastError();
  }
  const dim3 grid((unsigned)R * D.nkv * splits);
#define ROLLOUT_ATTN(T, HD)                                                                                        \
  hipLaunchKernelGGL((k_attn_valu<T, HD>), grid, dim3(256), 0, s, D, (const T*)q, (const T*)kv_pool, n_blocks, tables, \
                     max_blocks, rm, splits, split_tokens, layer, opart, ml, err)
  if (D.dtype == ROLLOUT_DTYPE_BF16) {
    ROLLOUT_ATTN(uint16_t, 32);
  } else {
    if (D.hd == 128) ROLLOUT_ATTN(float, 128);
    else if (D.hd == 64) ROLLOUT_ATTN(float, 64);
    else ROLLOUT_ATTN(float, 32);
  }
#undef ROLLOUT_ATTN
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // merge the context splits into the output
  const dim3 cgrid(R, ((D.qd >> 3) + 63) / 64);
  if (D.dtype == ROLLOUT_DTYPE_BF16)
    hipLaunchKernelGGL(k_attn_combine<uint16_t>, cgrid, dim3(64), 0, s, opart, ml, R, D.nh, splits, D.hd,
                       (uint16_t*)out);
  else
    hipLaunchKernelGGL(k_attn_combine<float>, cgrid, dim3(64), 0, s, opart, ml, R, D.nh, splits, D.hd, (float*)out);
  return hipGetLastError();
}

}  // namespace rollout
