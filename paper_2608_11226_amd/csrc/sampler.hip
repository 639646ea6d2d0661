// Token sampler: temperature, nucleus (top-p) truncation by radix select, and
// an inverse-CDF draw with a caller-supplied uniform.
//
// Definition (per row z, temperature T, top_p, uniform u):
//   T == 0: greedy arg max, lowest id among equal maxima.
//   y_i = fp32(z_i / T), m = max y, e_i = fp32 exp(y_i - m).
//   top_p < 1: keep the shortest prefix, in (e descending, id ascending)
//   order, whose mass reaches top_p of the total; otherwise keep all.
//   Walk the kept ids in ascending order and return the first whose running
//   mass exceeds u times the kept mass.
//
// Masses are fixed-point integers, floor(e * 2^40) (exact for e >= 2^-16,
// under 2^-40 of error each otherwise), so every sum, scan and comparison is
// exact integer arithmetic and the draw does not depend on scheduling.  The
// top-p threshold tau is a most-significant-digit radix select over the IEEE
// bit patterns of e (monotonic for e >= 0): four 8-bit digits, each digit
// chosen from mass histograms.  Ties at tau are kept lowest id first.
//
// Two implementations of the same integers.  Chunked (fewer rows): every
// pass over a row's V values runs as rows x chunks workgroups, a chunk being
// a whole number of 4096-id batches that a workgroup loads in one round trip
// (chunk max; exp stored once with the chunk mass and first-digit histogram; one
// histogram pass per remaining digit, the last one also leaving per chunk what
// its kept mass and its ties at tau are for either choice of the last digit).
// The chunks add their histogram bins into the row's histogram of each digit
// with integer atomics (the same sums in any order), and every workgroup of the
// next pass picks the digits chosen so far itself, with a parallel suffix scan
// over the row's 256 bins per digit, so no pass waits for a selection kernel.
// The final kernel per row selects tau the same way, takes the chunks' kept
// masses, finds the chunk holding the crossing, and walks only that chunk:
// one contiguous segment per wave, segment totals scanned across waves, then
// the crossing wave scans its segment 64 ids at a time.  Per row (from 128
// rows without top-p filtering, from 256 with it): one workgroup makes all of
// these passes over its row.
#include "internal.h"

#include <climits>
#include <type_traits>
#include <cstdlib>
#include <string>

namespace rollout {
namespace {

constexpr int CB = 256;  // threads of the per-chunk kernels
constexpr int CW = CB / 64;
constexpr int kMaxChunks = 64;  // chunks per row (sample_chunks caps nc here)
constexpr int kPer = 16;        // ids per thread in one batch of a chunk kernel
constexpr int kBatch = CB * kPer;  // ids per batch; a chunk is a whole number of batches
constexpr int RB = 1024;  // threads of the per-row draw kernel
constexpr int RW = RB / 64;
typedef unsigned long long u64;

// per-row selection state shared by the passes
struct RowSel {
  u64 total;   // mass of the row
  u64 target;  // ceil(top_p * total): mass the kept set must reach
  u64 above;   // mass of values strictly above the selected prefix
  unsigned prefix, mask;
  u64 kties;   // ties at tau that are kept (lowest ids first)
  u64 kept;    // kept mass
  float m;     // max of y
  int pad;
};

// floor(e * 2^40) for 0 <= e <= 1, by shifting the significand
__device__ __forceinline__ u64 fx40(float e) {
  const unsigned b = __float_as_uint(e);
  const int ex = (int)(b >> 23);
  if (ex == 0) return 0;
  const u64 mant = (u64)((b & 0x7FFFFFu) | 0x800000u);
  const int sh = ex - 110;  // e = mant * 2^(ex - 150)
  if (sh >= 0) return mant << sh;
  return sh > -24 ? mant >> (-sh) : 0;
}

// this lane's share of a row's nc (<= 64) chunk maxima: one vector load per lane (lanes past nc re-read the
// last); wave_max of it is the row maximum.  Uniform addresses would become scalar loads, at most 15 in
// flight, whose round trips would come before the chunk's own loads.
__device__ __forceinline__ float row_max_part(const float* cm, int nc) {
  return cm[min((int)(threadIdx.x & 63), nc - 1)];
}

// One batch of a chunk: thread t takes ids b + j * CB + t (j < kPer), all kPer loads in flight before
// the first is used.  Ids at or past hi read id hi - 1 (hi > b) and are masked where the values are used,
// unconditionally (a select, not a branch), so the compiler keeps the loads together.
__device__ __forceinline__ void load_batch(const float* __restrict__ row, int b, int hi, float* v) {
#pragma unroll
  for (int j = 0; j < kPer; ++j) v[j] = row[min(b + j * CB + (int)threadIdx.x, hi - 1)];
}

__device__ __forceinline__ u64 wave_sum_u64(u64 v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ u64 wave_incl_scan(u64 v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const u64 t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// the row's mass histograms of the four digits (bits 24..31, 16..23, 8..15, 0..7), each over the values
// that match the digits selected above it: rowhist[row][level][bin], level = (24 - shift) / 8
constexpr int kLevels = 4;

// Inclusive scan of one u64 per lane over the wave by DPP lane moves (no LDS): shifts of 1, 2, 4, 8 lanes
// within each row of 16, then row 0's total into row 1 and row 2's into row 3 (row_bcast:15), then the
// first two rows' total into rows 2 and 3 (row_bcast:31).  A lane with no source adds 0.
__device__ __forceinline__ u64 wave_incl_scan_dpp(u64 v) {
  auto step = [&](auto ctrl, auto row_mask) {
    constexpr int c = decltype(ctrl)::value, r = decltype(row_mask)::value;
    const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)v, c, r, 0xf, false);
    const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)(v >> 32), c, r, 0xf, false);
    v += ((u64)hi << 32) | lo;
  };
  step(std::integral_constant<int, 0x111>{}, std::integral_constant<int, 0xf>{});  // row_shr:1
  step(std::integral_constant<int, 0x112>{}, std::integral_constant<int, 0xf>{});  // row_shr:2
  step(std::integral_constant<int, 0x114>{}, std::integral_constant<int, 0xf>{});  // row_shr:4
  step(std::integral_constant<int, 0x118>{}, std::integral_constant<int, 0xf>{});  // row_shr:8
  step(std::integral_constant<int, 0x142>{}, std::integral_constant<int, 0xa>{});  // row_bcast:15
  step(std::integral_constant<int, 0x143>{}, std::integral_constant<int, 0xc>{});  // row_bcast:31
  return v;
}

__device__ __forceinline__ u64 readlane_u64(u64 v, int lane) {
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, lane);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), lane);
  return ((u64)hi << 32) | lo;
}

// Row state before the first digit, from the first digit's bins (lane l: h[k] = bin 255 - 4l - k): total
// mass and the mass the kept set must reach.
__device__ __forceinline__ RowSel select_init(const u64* h, float top_p) {
  const u64 total = readlane_u64(wave_incl_scan_dpp(h[0] + h[1] + h[2] + h[3]), 63);
  RowSel st;
  st.total = total;
  const u64 target = (u64)ceil((double)top_p * (double)total);
  st.target = target > total ? total : (target == 0 ? 1 : target);
  st.above = 0;
  st.prefix = 0;
  st.mask = 0;
  st.kties = 0;
  st.kept = 0;
  st.m = 0.f;
  st.pad = 0;
  return st;
}

// One digit of the selection, by one wave: lane l holds h[k] = bin 255 - 4l - k (k = 0..3) of the row's
// histogram at `shift`.  The digit is the largest d with above + sum_{j >= d} hist[j] >= target: suffix
// sums in descending digit order (within the lane, then across lanes by a scan), the first place where
// they reach the target.  At the last digit also the kept ties and the kept mass.  Every wave of every
// workgroup of a row computes the same integers, so no wave waits for another.
__device__ __forceinline__ void select_digit(const u64* h, int shift, RowSel& st) {
  const u64 c0 = h[0], c1 = c0 + h[1], c2 = c1 + h[2], c3 = c2 + h[3];
  const u64 excl = wave_incl_scan_dpp(c3) - c3;  // mass of the digits of the lanes before this one
  const bool r0 = st.above + excl + c0 >= st.target, r1 = st.above + excl + c1 >= st.target,
             r2 = st.above + excl + c2 >= st.target, r3 = st.above + excl + c3 >= st.target;
  const unsigned long long bal = __ballot(r3);
  if (!bal) return;
  const int first = __ffsll((long long)bal) - 1;  // the lane holding the selected digit
  const int k = r0 ? 0 : (r1 ? 1 : (r2 ? 2 : 3));
  const u64 ck = r0 ? c0 : (r1 ? c1 : (r2 ? c2 : c3));
  const u64 hk = r0 ? h[0] : (r1 ? h[1] : (r2 ? h[2] : h[3]));
  const int dsel = 255 - 4 * first - __builtin_amdgcn_readlane(k, first);
  st.above = readlane_u64(st.above + excl + ck - hk, first);  // mass of the digits above dsel
  st.prefix |= (unsigned)dsel << shift;
  st.mask |= 255u << shift;
  if (shift == 0) {
    const u64 ftau = fx40(__uint_as_float(st.prefix));
    const u64 need = st.target - st.above;
    st.kties = ftau ? (need + ftau - 1) / ftau : 0;
    st.kept = st.above + st.kties * ftau;
  }
}

// this lane's bins of the row histograms at levels 0 .. kLevels - 1 (level l clamped to lmax)
__device__ __forceinline__ void load_row_bins(const u64* __restrict__ rh, int lmax, u64 (*hb)[4]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int l = 0; l < kLevels; ++l)
#pragma unroll
    for (int k = 0; k < 4; ++k) hb[l][k] = rh[min(l, lmax) * 256 + 255 - 4 * lane - k];
}

// The row state after the digits of levels 0 .. levels - 1, selected again by every wave from the row
// histograms (a few scans; cheaper than a round trip to state left by the previous pass)
__device__ __forceinline__ RowSel select_above(const u64 (*hb)[4], int levels, float top_p) {
  RowSel st = select_init(hb[0], top_p);
#pragma unroll
  for (int l = 0; l < kLevels; ++l)
    if (l < levels) select_digit(hb[l], 24 - 8 * l, st);
  return st;
}

// A chunk's digit histogram into the row's: thread t adds bin t of its waves' LDS copies (bins with no
// mass are skipped)
__device__ __forceinline__ void add_row_bins(u64 (*hist)[256], u64* __restrict__ rh) {
  u64 t = 0;
#pragma unroll
  for (int j = 0; j < CW; ++j) t += hist[j][threadIdx.x];
  if (t) atomicAdd(rh + threadIdx.x, t);
}

// ---------------------------------------------------------------------------
// greedy
// ---------------------------------------------------------------------------
__device__ __forceinline__ void better(float& best, int& bi, float v, int i) {
  if (v > best || (v == best && i < bi)) { best = v; bi = i; }
}

__global__ __launch_bounds__(CB) void k_chunk_argmax(const float* __restrict__ logits, int V, int chunk,
                                                     float* __restrict__ cval, int* __restrict__ cidx) {
  __shared__ float rv[CW];
  __shared__ int ri[CW];
  const int row = blockIdx.x, c = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* z = logits + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  float best = -INFINITY;
  int bi = INT_MAX;
  for (int b = lo; b < hi; b += kBatch) {
    float v[kPer];
    load_batch(z, b, hi, v);
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = b + j * CB + tid;
      better(best, bi, i < hi ? v[j] : -INFINITY, i < hi ? i : INT_MAX);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) better(best, bi, __shfl_xor(best, o, 64), __shfl_xor(bi, o, 64));
  if (lane == 0) { rv[w] = best; ri[w] = bi; }
  __syncthreads();
  if (tid == 0) {
    for (int j = 1; j < CW; ++j) better(best, bi, rv[j], ri[j]);
    cval[(size_t)row * gridDim.y + c] = best;
    cidx[(size_t)row * gridDim.y + c] = bi;
  }
}

__global__ __launch_bounds__(64) void k_argmax_final(const float* __restrict__ cval, const int* __restrict__ cidx,
                                                     int nc, const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                                     int out_stride) {
  const int row = blockIdx.x, lane = threadIdx.x;
  float best = -INFINITY;
  int bi = INT_MAX;
  for (int c = lane; c < nc; c += 64) better(best, bi, cval[(size_t)row * nc + c], cidx[(size_t)row * nc + c]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) better(best, bi, __shfl_xor(best, o, 64), __shfl_xor(bi, o, 64));
  if (lane == 0) out[(size_t)row * out_stride + (col ? col[0] : 0)] = bi == INT_MAX ? 0 : bi;
}

// ---------------------------------------------------------------------------
// sampling
// ---------------------------------------------------------------------------
// cmax[row][c] = max over chunk c of z.  For T > 0 the rounded quotient fp32(z / T) does not decrease as
// z grows, so the largest y of the row is fp32(max z / T): the exp pass divides the row maximum once.
__global__ __launch_bounds__(CB) void k_chunk_max(const float* __restrict__ logits, int V, int chunk,
                                                  float* __restrict__ cmax, u64* __restrict__ rowhist) {
  __shared__ float red[CW];
  const int row = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  if (c == 0)  // the row's digit histograms start from zero in every call
    for (int i = tid; i < kLevels * 256; i += CB) rowhist[(size_t)row * kLevels * 256 + i] = 0;
  const float* z = logits + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  float mx = -INFINITY;
  for (int b = lo; b < hi; b += kBatch) {
    float v[kPer];
    load_batch(z, b, hi, v);
#pragma unroll
    for (int j = 0; j < kPer; ++j) mx = fmaxf(mx, b + j * CB + tid < hi ? v[j] : -INFINITY);
  }
  mx = wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  if (tid == 0) {
    for (int j = 1; j < CW; ++j) mx = fmaxf(mx, red[j]);
    cmax[(size_t)row * gridDim.y + c] = mx;
  }
}

// e = exp(y - m) stored; chunk mass; first-digit (bits 24..31) mass histogram when filtering
__global__ __launch_bounds__(CB) void k_chunk_exp(const float* __restrict__ logits, int V, int chunk, float T,
                                                  const float* __restrict__ cmax, float* __restrict__ escr,
                                                  u64* __restrict__ cmass, u64* __restrict__ rowhist, int filter) {
  __shared__ u64 hist[CW][256];
  __shared__ u64 red[CW];
  const int row = blockIdx.x, c = blockIdx.y, nc = gridDim.y, tid = threadIdx.x, w = tid >> 6;
  const float* z = logits + (size_t)row * V;
  float* e_row = escr + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  // the row's chunk maxima, then the chunk's first batch, then the wait for the maxima alone (the load
  // counter retires in issue order, so the batch stays in flight)
  const float mpart = row_max_part(cmax + (size_t)row * nc, nc);
  __builtin_amdgcn_sched_barrier(0);
  float v[kPer];
  load_batch(z, lo, hi, v);
  __builtin_amdgcn_sched_barrier(0);
  const float m = wave_max(mpart) / T;  // max of fp32(z / T) (see k_chunk_max)
  if (filter) {
    for (int i = tid; i < CW * 256; i += CB) (&hist[0][0])[i] = 0;
    __syncthreads();
  }
  u64 mass = 0;
  for (int b = lo; b < hi; b += kBatch) {
    if (b > lo) load_batch(z, b, hi, v);
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = b + j * CB + tid;
      const float e = expf(v[j] / T - m);
      const u64 f = i < hi ? fx40(e) : 0ull;
      mass += f;
      if (i < hi) {
        e_row[i] = e;
        if (filter) atomicAdd(&hist[w][__float_as_uint(e) >> 24], f);
      }
    }
  }
  mass = wave_sum_u64(mass);
  if ((tid & 63) == 0) red[w] = mass;
  __syncthreads();
  if (tid == 0) {
    u64 t = 0;
    for (int j = 0; j < CW; ++j) t += red[j];
    cmass[(size_t)row * nc + c] = t;
  }
  if (filter) add_row_bins(hist, rowhist + (size_t)row * kLevels * 256);
}

// mass histogram of the digit at `shift` over values matching the digits selected above it; each
// workgroup first selects those digits from the row's histograms (the same integers in every workgroup).
// LAST (the lowest digit, shift 0): the chunk also leaves what the draw needs to find its kept mass once
// the digit is chosen: the mass of its values above the selected 24-bit prefix (cabove), the suffix sums
// of its own digit histogram (csuf[d] = mass of its matching values with digit >= d) and its count per
// digit (ccnt), so the kept mass of the chunk is cabove + csuf[tau's digit + 1] and its ties at tau are
// ccnt[tau's digit].
template <bool LAST>
__global__ __launch_bounds__(CB) void k_chunk_hist(const float* __restrict__ escr, int V, int chunk, int shift,
                                                   float top_p, u64* __restrict__ rowhist, u64* __restrict__ cabove,
                                                   u64* __restrict__ csuf, unsigned* __restrict__ ccnt) {
  __shared__ u64 hist[CW][256];
  __shared__ unsigned cnt[LAST ? CW : 1][LAST ? 256 : 1];
  __shared__ u64 red[CW];
  const int row = blockIdx.x, c = blockIdx.y, nc = gridDim.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int level = (24 - shift) >> 3;  // 1..3; the digits above are levels 0 .. level - 1
  u64* rh = rowhist + (size_t)row * kLevels * 256;
  const float* e_row = escr + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  // this lane's bins of the digits above, then the chunk's first batch: waiting for the bins leaves the
  // batch in flight during the selection
  u64 hb[kLevels][4];
  load_row_bins(rh, level - 1, hb);
  float v[kPer];
  load_batch(e_row, lo, hi, v);
  for (int i = tid; i < CW * 256; i += CB) (&hist[0][0])[i] = 0;
  if constexpr (LAST)
    for (int i = tid; i < CW * 256; i += CB) (&cnt[0][0])[i] = 0;
  const RowSel st = select_above(hb, level, top_p);
  const unsigned prefix = st.prefix, mask = st.mask;
  __syncthreads();  // the cleared bins
  u64 above = 0;
  auto add = [&](int b0) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const unsigned b = __float_as_uint(v[j]);
      const bool ok = b0 + j * CB + tid < hi;
      if (ok && (b & mask) == prefix) {
        atomicAdd(&hist[w][(b >> shift) & 255u], fx40(v[j]));
        if constexpr (LAST) atomicAdd(&cnt[w][b & 255u], 1u);
      }
      if constexpr (LAST) above += ok && b > (prefix | 255u) ? fx40(v[j]) : 0ull;  // 24-bit prefix above
    }
  };
  add(lo);
  for (int b0 = lo + kBatch; b0 < hi; b0 += kBatch) {
    load_batch(e_row, b0, hi, v);
    add(b0);
  }
  __syncthreads();
  if constexpr (!LAST) {
    add_row_bins(hist, rh + level * 256);
  } else {
    // thread t holds digit t: its mass (added into the row's histogram) and count, then the chunk's
    // suffix sums over digits (within each wave by a scan, then the totals of the waves above)
    u64 t = 0;
    unsigned n = 0;
#pragma unroll
    for (int j = 0; j < CW; ++j) {
      t += hist[j][tid];
      n += cnt[j][tid];
    }
    if (t) atomicAdd(rh + level * 256 + tid, t);
    const u64 incl = wave_incl_scan_dpp(t);
    const u64 wtot = readlane_u64(incl, 63);
    above = wave_sum_u64(above);
    __syncthreads();  // every wave has read hist; reuse it for the wave totals and the above masses
    if (lane == 0) {
      hist[0][w] = wtot;
      red[w] = above;
    }
    __syncthreads();
    u64 suf = wtot - incl + t;
#pragma unroll
    for (int j = 0; j < CW; ++j)
      if (j > w) suf += hist[0][j];
    const size_t ci = (size_t)row * nc + c;
    csuf[ci * 256 + tid] = suf;
    ccnt[ci * 256 + tid] = n;
    if (tid == 0) {
      u64 a = 0;
#pragma unroll
      for (int j = 0; j < CW; ++j) a += red[j];
      cabove[ci] = a;
    }
  }
}

// the ordered draw: locate the crossing chunk from chunk totals, then walk that chunk only
__global__ __launch_bounds__(RB) void k_draw(const float* __restrict__ escr, int V, int chunk, int nc, int filter,
                                             float top_p, const u64* __restrict__ rowhist,
                                             const u64* __restrict__ cabove, const u64* __restrict__ csuf,
                                             const unsigned* __restrict__ ccnt, const u64* __restrict__ cmass,
                                             const float* __restrict__ u, int u_stride,
                                             const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                             int out_stride) {
  __shared__ u64 s_mass[RW], s_ties[RW];
  __shared__ int s_chunk, s_tok;
  __shared__ u64 s_excl, s_ties_before, s_thresh;
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c_out = col ? col[0] : 0;
  const float* e_row = escr + (size_t)row * V;
  unsigned tau = 0;
  u64 ftau = 0, kties = 0, kept = 0;
  if (filter) {
    // tau and the kept ties from the row's four digit histograms (every wave selects the same integers)
    u64 hb[kLevels][4];
    load_row_bins(rowhist + (size_t)row * kLevels * 256, kLevels - 1, hb);
    const RowSel st = select_above(hb, kLevels, top_p);
    tau = st.prefix;
    ftau = fx40(__uint_as_float(tau));
    kties = st.kties;
    kept = st.kept;
  } else {
    // the row's total mass: one chunk per lane (nc <= 64), then a wave sum
    const u64 cm = cmass[(size_t)row * nc + min(lane, nc - 1)];
    kept = wave_sum_u64(lane < nc ? cm : 0ull);
  }
  if (w == 0) {
    // chunk scan in one wave (nc <= 64): kept mass per chunk = gt + its kept ties, where gt is the mass of
    // its values above tau (with filtering: above tau's 24-bit prefix, plus its digits above tau's digit;
    // without: the whole chunk) and ti its values equal to tau
    const size_t ci = (size_t)row * nc + min(lane, nc - 1);
    const unsigned d = tau & 255u;
    u64 gt = filter ? cabove[ci] + (d < 255u ? csuf[ci * 256 + d + 1] : 0ull) : cmass[ci];
    u64 ti = filter ? (u64)ccnt[ci * 256 + d] : 0ull;
    if (lane >= nc) gt = ti = 0;
    const u64 ties_incl = wave_incl_scan(ti, lane);
    const u64 ties_before = ties_incl - ti;
    const u64 kt = filter ? (kties > ties_before ? min(kties - ties_before, ti) : 0) : 0;
    const u64 km = gt + kt * ftau;
    const u64 incl = wave_incl_scan(km, lane);
    // thresh < kept always (u < 1 and kept >= 2^40), so some chunk holds the crossing
    const u64 thresh = (u64)((double)u[(size_t)row * u_stride + c_out] * (double)kept);
    const unsigned long long hit = __ballot(lane < nc && km > 0 && incl > thresh);
    const int first = hit ? __ffsll((long long)hit) - 1 : max(0, nc - 1);
    if (lane == first) {
      s_chunk = lane;
      s_excl = incl - km;
      s_ties_before = ties_before;
      s_thresh = thresh;
    }
    if (lane == 0) s_tok = -1;
  }
  __syncthreads();
  const int c = s_chunk;
  const u64 thresh = s_thresh;
  // segments of the crossing chunk, one per wave
  const int lo_c = c * chunk, hi_c = min(V, lo_c + chunk);
  const int seg = ((hi_c - lo_c + RW - 1) / RW + 63) / 64 * 64;
  const int lo = min(hi_c, lo_c + w * seg), hi = min(hi_c, lo + seg);
  u64 gt = 0, ties = 0;
  // four 64-id steps of the segment per round trip (clamped to the segment's last id, masked at use)
  for (int b0 = lo; b0 < hi; b0 += 4 * 64) {
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = e_row[min(b0 + j * 64 + lane, hi - 1)];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = b0 + j * 64 + lane < hi;
      const unsigned b = __float_as_uint(v[j]);
      const u64 f = fx40(v[j]);
      gt += ok && (!filter || b > tau) ? f : 0ull;
      ties += ok && filter && b == tau ? 1ull : 0ull;
    }
  }
  gt = wave_sum_u64(gt);
  ties = wave_sum_u64(ties);
  if (lane == 0) { s_mass[w] = gt; s_ties[w] = ties; }
  __syncthreads();
  u64 ties_before = s_ties_before, excl = s_excl;
  for (int j = 0; j < w; ++j) ties_before += s_ties[j];
  const u64 my_kept_ties = filter ? (kties > ties_before ? min(kties - ties_before, ties) : 0) : 0;
  // kept mass before this wave's segment within the chunk
  for (int j = 0; j < w; ++j) {
    u64 tb = s_ties_before;
    for (int i = 0; i < j; ++i) tb += s_ties[i];
    const u64 ktj = filter ? (kties > tb ? min(kties - tb, s_ties[j]) : 0) : 0;
    excl += s_mass[j] + ktj * ftau;
  }
  const u64 my_mass = gt + my_kept_ties * ftau;
  if (my_mass > 0 && excl <= thresh && thresh < excl + my_mass) {
    u64 carry = excl, tie_carry = 0;
    bool found = false;
    for (int b0 = lo; b0 < hi && !found; b0 += 4 * 64) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = e_row[min(b0 + j * 64 + lane, hi - 1)];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int base = b0 + j * 64;
        if (found || base >= hi) break;  // wave-uniform
        const int i = base + lane;
        const float e = i < hi ? v[j] : 0.f;
        const unsigned b = __float_as_uint(e);
        bool keep = i < hi && (!filter || b > tau);
        if (filter) {
          const bool is_tie = i < hi && b == tau;
          const u64 tie_incl = wave_incl_scan(is_tie ? 1ull : 0ull, lane);
          if (is_tie && tie_carry + tie_incl - 1 < my_kept_ties) keep = true;
          tie_carry += __shfl(tie_incl, 63, 64);
        }
        const u64 cum = carry + wave_incl_scan(keep ? fx40(e) : 0ull, lane);
        const unsigned long long hit = __ballot(keep && cum > thresh);
        if (hit) {
          if (lane == __ffsll((long long)hit) - 1) s_tok = i;
          found = true;
        } else {
          carry = __shfl(cum, 63, 64);
        }
      }
    }
  }
  __syncthreads();
  if (tid == 0) out[(size_t)row * out_stride + c_out] = s_tok < 0 ? 0 : s_tok;
}

// ---------------------------------------------------------------------------
// One workgroup per row
// ---------------------------------------------------------------------------
// Rows of at most kRowMaxV ids (V a multiple of 4) are sampled by one
// workgroup of SR threads that makes every pass above itself, so a step costs
// one launch instead of up to eleven and no pass waits for another kernel.
// The row is cut into segments of 256 ids; wave w takes segments w, w + SRW,
// ..., each lane four consecutive ids (one 16-byte load).  Masses, histograms,
// the digit selection, the tie rule and the draw are the same integers as in
// the chunked kernels (segments play the role of chunks), so both paths give
// the same token.
constexpr int SR = 1024;
constexpr int SRW = SR / 64;
constexpr int kSeg = 256;
constexpr int kRowMaxSeg = SR;  // one segment per thread in the scans
constexpr int kRowMaxV = kRowMaxSeg * kSeg;

// inclusive scan of one u64 per thread over the SR threads; *tot receives the total
__device__ __forceinline__ u64 block_incl_scan(u64 v, u64* wtot, u64* tot) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_incl_scan(v, lane);
  __syncthreads();
  if (lane == 63) wtot[w] = v;
  __syncthreads();
  u64 before = 0, all = 0;
  for (int j = 0; j < SRW; ++j) {
    if (j < w) before += wtot[j];
    all += wtot[j];
  }
  *tot = all;
  return v + before;
}

// Segments are visited four at a time per wave (sg0 + j * SRW, j < 4): the four 16-byte loads are
// unconditional (ids past the row read its last four values and are masked at use), so they are all in
// flight before the first is used.
constexpr int kSegBatch = 4;
__device__ __forceinline__ void load_seg_batch(const float* row, int V, int sg0, int lane, float4* a, bool* ok) {
#pragma unroll
  for (int j = 0; j < kSegBatch; ++j) {
    const int i = (sg0 + j * SRW) * kSeg + 4 * lane;
    ok[j] = i < V;
    a[j] = *reinterpret_cast<const float4*>(row + min(i, V - 4));
  }
}

__global__ __launch_bounds__(SR) void k_sample_row(const float* __restrict__ logits, int V, float T, float top_p,
                                                   int filter, float* __restrict__ escr, const float* __restrict__ u,
                                                   int u_stride, const int32_t* __restrict__ col,
                                                   int32_t* __restrict__ out, int out_stride) {
  __shared__ u64 hist[SRW][256];
  __shared__ u64 s_gt[kRowMaxSeg], s_ties[kRowMaxSeg];
  __shared__ u64 wtot[SRW];
  __shared__ float s_redf[SRW];
  __shared__ int wcnt[4];
  __shared__ u64 s_above, s_target, s_excl, s_ties_before;
  __shared__ unsigned s_prefix, s_mask;
  __shared__ int s_seg, s_tok;
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c_out = col ? col[0] : 0;
  const float* z = logits + (size_t)row * V;
  float* e_row = escr + (size_t)row * V;
  const int nseg = (V + kSeg - 1) / kSeg;

  // m = max of y = fp32(z / T)
  float mx = -INFINITY;
  for (int sg0 = w; sg0 < nseg; sg0 += kSegBatch * SRW) {
    float4 a[kSegBatch];
    bool ok[kSegBatch];
    load_seg_batch(z, V, sg0, lane, a, ok);
#pragma unroll
    for (int j = 0; j < kSegBatch; ++j)
      if (ok[j]) mx = fmaxf(mx, fmaxf(fmaxf(a[j].x / T, a[j].y / T), fmaxf(a[j].z / T, a[j].w / T)));
  }
  mx = wave_max(mx);
  if (lane == 0) s_redf[w] = mx;
  for (int i = tid; i < SRW * 256; i += SR) (&hist[0][0])[i] = 0;
  if (tid == 0) {
    s_seg = INT_MAX;
    s_tok = -1;
  }
  __syncthreads();
  float m = -INFINITY;
  for (int j = 0; j < SRW; ++j) m = fmaxf(m, s_redf[j]);

  // e = exp(y - m), stored; per-segment mass; first-digit (bits 24..31) mass histogram when filtering
  for (int sg0 = w; sg0 < nseg; sg0 += kSegBatch * SRW) {
    float4 a[kSegBatch];
    bool ok[kSegBatch];
    load_seg_batch(z, V, sg0, lane, a, ok);
#pragma unroll
    for (int j = 0; j < kSegBatch; ++j) {
      const int sg = sg0 + j * SRW;
      u64 f = 0;
      if (ok[j]) {
        const float e[4] = {expf(a[j].x / T - m), expf(a[j].y / T - m), expf(a[j].z / T - m), expf(a[j].w / T - m)};
        *reinterpret_cast<float4*>(e_row + sg * kSeg + 4 * lane) = make_float4(e[0], e[1], e[2], e[3]);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const u64 fq = fx40(e[q]);
          f += fq;
          if (filter) atomicAdd(&hist[w][__float_as_uint(e[q]) >> 24], fq);
        }
      }
      f = wave_sum_u64(f);
      if (lane == 0 && sg < nseg) {
        s_gt[sg] = f;
        s_ties[sg] = 0;
      }
    }
  }
  __syncthreads();
  u64 total;
  block_incl_scan(tid < nseg ? s_gt[tid] : 0, wtot, &total);

  unsigned tau = 0;
  u64 ftau = 0, kties = 0, kept = total;
  if (filter) {
    if (tid == 0) {
      const u64 target = (u64)ceil((double)top_p * (double)total);
      s_target = target > total ? total : (target == 0 ? 1 : target);
      s_above = 0;
      s_prefix = 0;
      s_mask = 0;
    }
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (shift != 24) {
        // mass histogram of the digit at shift over the values matching the selected prefix
        __syncthreads();
        for (int i = tid; i < SRW * 256; i += SR) (&hist[0][0])[i] = 0;
        __syncthreads();
        const unsigned prefix = s_prefix, mask = s_mask;
        for (int sg0 = w; sg0 < nseg; sg0 += kSegBatch * SRW) {
          float4 a[kSegBatch];
          bool ok[kSegBatch];
          load_seg_batch(e_row, V, sg0, lane, a, ok);
#pragma unroll
          for (int j = 0; j < kSegBatch; ++j) {
            if (!ok[j]) continue;
            const float e[4] = {a[j].x, a[j].y, a[j].z, a[j].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const unsigned b = __float_as_uint(e[q]);
              if ((b & mask) == prefix) atomicAdd(&hist[w][(b >> shift) & 255u], fx40(e[q]));
            }
          }
        }
      }
      __syncthreads();
      // the largest digit d with above + (mass of digits >= d) >= target; threads 0..255, thread t owning
      // digit 255 - t, so the suffix sum is an inclusive scan in thread order
      const int d = 255 - tid;
      u64 h = 0, inc = 0;
      if (tid < 256) {
        for (int j = 0; j < SRW; ++j) h += hist[j][d];
        inc = wave_incl_scan(h, lane);
        if (lane == 63) wtot[w] = inc;
      }
      __syncthreads();
      const u64 above = s_above, target = s_target;
      if (tid < 256) {
        for (int j = 0; j < w; ++j) inc += wtot[j];
        const unsigned long long bal = __ballot(above + inc >= target);
        if (lane == 0) wcnt[w] = __popcll(bal);
      }
      __syncthreads();
      if (tid < 256 && d == wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3] - 1) {
        s_above = above + inc - h;
        s_prefix |= (unsigned)d << shift;
        s_mask |= 255u << shift;
      }
    }
    __syncthreads();
    tau = s_prefix;
    ftau = fx40(__uint_as_float(tau));
    const u64 need = s_target - s_above;
    kties = ftau ? (need + ftau - 1) / ftau : 0;
    kept = s_above + kties * ftau;
    // per segment: mass of the values above tau and the count of ties at tau
    for (int sg0 = w; sg0 < nseg; sg0 += kSegBatch * SRW) {
      float4 a[kSegBatch];
      bool ok[kSegBatch];
      load_seg_batch(e_row, V, sg0, lane, a, ok);
#pragma unroll
      for (int j = 0; j < kSegBatch; ++j) {
        const int sg = sg0 + j * SRW;
        u64 gt = 0, ties = 0;
        if (ok[j]) {
          const float e[4] = {a[j].x, a[j].y, a[j].z, a[j].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const unsigned b = __float_as_uint(e[q]);
            if (b > tau) gt += fx40(e[q]);
            else if (b == tau) ties += 1;
          }
        }
        gt = wave_sum_u64(gt);
        ties = wave_sum_u64(ties);
        if (lane == 0 && sg < nseg) {
          s_gt[sg] = gt;
          s_ties[sg] = ties;
        }
      }
    }
    __syncthreads();
  }

  // kept mass per segment (ties at tau kept lowest id first), its scan, and the segment holding the crossing
  const u64 gt = tid < nseg ? s_gt[tid] : 0, ti = tid < nseg ? s_ties[tid] : 0;
  u64 unused;
  const u64 ties_before = block_incl_scan(ti, wtot, &unused) - ti;
  const u64 kt = filter ? (kties > ties_before ? min(kties - ties_before, ti) : 0) : 0;
  const u64 km = gt + kt * ftau;
  const u64 incl = block_incl_scan(km, wtot, &unused);
  // thresh < kept always (u < 1 and kept >= 2^40), so some segment holds the crossing
  const u64 thresh = (u64)((double)u[(size_t)row * u_stride + c_out] * (double)kept);
  if (tid < nseg && km > 0 && incl > thresh) atomicMin(&s_seg, tid);
  __syncthreads();
  const int c = s_seg == INT_MAX ? nseg - 1 : s_seg;
  if (tid == c) {
    s_excl = incl - km;
    s_ties_before = ties_before;
  }
  __syncthreads();
  if (w == 0) {
    // walk the crossing segment 64 ids at a time
    const int lo = c * kSeg, hi = min(V, lo + kSeg);
    const u64 tb = s_ties_before, seg_ties = s_ties[c];
    const u64 my_kept_ties = filter ? (kties > tb ? min(kties - tb, seg_ties) : 0) : 0;
    u64 carry = s_excl, tie_carry = 0;
    for (int base = lo; base < hi; base += 64) {
      const int i = base + lane;
      const float e = i < hi ? e_row[i] : 0.f;
      const unsigned b = __float_as_uint(e);
      bool keep = i < hi && (!filter || b > tau);
      if (filter) {
        const bool is_tie = i < hi && b == tau;
        const u64 tie_incl = wave_incl_scan(is_tie ? 1ull : 0ull, lane);
        if (is_tie && tie_carry + tie_incl - 1 < my_kept_ties) keep = true;
        tie_carry += __shfl(tie_incl, 63, 64);
      }
      const u64 cum = carry + wave_incl_scan(keep ? fx40(e) : 0ull, lane);
      const unsigned long long hit = __ballot(keep && cum > thresh);
      if (hit) {
        if (lane == __ffsll((long long)hit) - 1) s_tok = i;
        break;
      }
      carry = __shfl(cum, 63, 64);
    }
  }
  __syncthreads();
  if (tid == 0) out[(size_t)row * out_stride + c_out] = s_tok < 0 ? 0 : s_tok;
}

// Which path samples S rows: one workgroup per row from a row count that depends on filtering (its time is
// set by one workgroup's passes over its row, so it barely grows with S; the chunked kernels grow with S
// and win below).  Measured at V = 152064, row / chunked: top-p 0.95: S = 64: 206 / 94 us, S = 128:
// 210 / 147 us, S = 256: 245 / 258 us; top-p 1 (no digit passes): S = 64: 79 / 60 us, S = 128: 80 / 88 us,
// S = 256: 90 / 152 us.  ROLLOUT_SAMPLE_PATH=row or =chunked forces a path (read per call; the row path
// still needs V % 4 == 0 and V <= kRowMaxV).
constexpr int kRowMinRows = 128, kRowMinRowsFiltered = 256;
bool use_row_sampler(int S, int V, bool filter) {
  if (V % 4 != 0 || V > kRowMaxV) return false;
  const char* v = std::getenv("ROLLOUT_SAMPLE_PATH");
  if (v && std::string(v) == "row") return true;
  if (v && std::string(v) == "chunked") return false;
  return S >= (filter ? kRowMinRowsFiltered : kRowMinRows);
}

}  // namespace

// Ids per chunk: the fewest whole batches that keep a row within kMaxChunks chunks.
int sample_chunk_ids(int V) {
  const long long per = ((long long)V + kMaxChunks - 1) / kMaxChunks;
  const long long b = (per + kBatch - 1) / kBatch;
  return (int)((b < 1 ? 1 : b) * kBatch);
}

int sample_chunks(int V) {
  const int c = (int)(((long long)V + sample_chunk_ids(V) - 1) / sample_chunk_ids(V));
  return c < 1 ? 1 : c;
}

size_t sample_scratch_bytes(int S, int V) {
  const int nc = sample_chunks(V);
  return (size_t)S * V * 4 + (size_t)S * nc * (4 + 4 + 8 + 8 + 256 * 8 + 256 * 4) + (size_t)S * kLevels * 256 * 8 +
         4096;
}

int sample_rows_fitting(size_t bytes, int V) {
  const size_t one = sample_scratch_bytes(1, V);
  if (one > bytes) return 0;
  const size_t per_row = sample_scratch_bytes(2, V) - one;
  size_t r = 1 + (bytes - one) / per_row;
  if (r > (size_t)INT_MAX) r = INT_MAX;
  while (r > 1 && sample_scratch_bytes((int)r, V) > bytes) --r;
  return (int)r;
}

hipError_t launch_sample(hipStream_t s, const float* logits, int S, int V, float temperature, float top_p,
                         const float* u, int u_stride, const int32_t* col, int32_t* out, int out_stride,
                         void* scratch) {
  if (S <= 0) return hipSuccess;
  const int nc = sample_chunks(V);
  const int chunk = sample_chunk_ids(V);
  char* p = (char*)scratch;
  auto take = [&](size_t bytes) {
    char* q = p;
    p += (bytes + 255) / 256 * 256;
    return q;
  };
  float* escr = (float*)take((size_t)S * V * 4);
  float* cmax = (float*)take((size_t)S * nc * 4);
  int* cidx = (int*)take((size_t)S * nc * 4);
  u64* cmass = (u64*)take((size_t)S * nc * 8);
  u64* cabove = (u64*)take((size_t)S * nc * 8);
  u64* csuf = (u64*)take((size_t)S * nc * 256 * 8);
  unsigned* ccnt = (unsigned*)take((size_t)S * nc * 256 * 4);
  u64* rowhist = (u64*)take((size_t)S * kLevels * 256 * 8);
  const dim3 rc(S, nc);
  if (temperature == 0.0f) {
    hipLaunchKernelGGL(k_chunk_argmax, rc, dim3(CB), 0, s, logits, V, chunk, cmax, cidx);
    hipLaunchKernelGGL(k_argmax_final, dim3(S), dim3(64), 0, s, cmax, cidx, nc, col, out, out_stride);
    return hipGetLastError();
  }
  const int filter = top_p < 1.0f;
  if (use_row_sampler(S, V, filter)) {
    hipLaunchKernelGGL(k_sample_row, dim3(S), dim3(SR), 0, s, logits, V, temperature, top_p, filter, escr, u, u_stride,
                       col, out, out_stride);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_chunk_max, rc, dim3(CB), 0, s, logits, V, chunk, cmax, rowhist);
  hipLaunchKernelGGL(k_chunk_exp, rc, dim3(CB), 0, s, logits, V, chunk, temperature, cmax, escr, cmass, rowhist,
                     filter);
  if (filter) {
    for (int shift = 16; shift >= 8; shift -= 8)
      hipLaunchKernelGGL(k_chunk_hist<false>, rc, dim3(CB), 0, s, escr, V, chunk, shift, top_p, rowhist, nullptr,
                         nullptr, nullptr);
    hipLaunchKernelGGL(k_chunk_hist<true>, rc, dim3(CB), 0, s, escr, V, chunk, 0, top_p, rowhist, cabove, csuf,
                       ccnt);
  }
  hipLaunchKernelGGL(k_draw, dim3(S), dim3(RB), 0, s, escr, V, chunk, nc, filter, top_p, rowhist, cabove, csuf, ccnt,
                     cmass, u,
                     u_stride, col, out, out_stride);
  return hipGetLastError();
}

}  // namespace rollout
