// Token sampler: temperature, nucleus (top-p) truncation by radix select, and
// an inverse-CDF draw with a caller-supplied uniform.  One workgroup of 1024
// threads (16 waves) per row of logits.
//
// Definition (per row z, temperature T, top_p, uniform u):
//   T == 0: greedy arg max, lowest id among equal maxima.
//   y_i = fp32(z_i / T), m = max y, e_i = fp32 exp(y_i - m).
//   top_p < 1: keep the shortest prefix, in (e descending, id ascending)
//   order, whose mass reaches top_p of the total; otherwise keep all.
//   Walk the kept ids in ascending order and return the first whose running
//   mass exceeds u times the kept mass.
//
// Masses are fixed-point integers, e * 2^40 truncated (exact for e >= 2^-16,
// under 2^-40 of error each otherwise), so every sum, scan and comparison is
// exact integer arithmetic and the draw does not depend on scheduling.  The
// top-p threshold is a most-significant-digit radix select over the IEEE bit
// patterns of e (monotonic for e >= 0): four 8-bit digits, mass histograms in
// LDS, one private histogram per wave to keep atomic contention inside a wave.
// Every pass over the row is coalesced: strided passes for max, mass and the
// histograms; for the ordered draw each wave owns a contiguous segment of ids,
// segment totals are scanned across waves, and only the wave whose segment
// holds the crossing walks it, 64 ids at a time with a wave-wide scan.
#include "internal.h"

#include <climits>

namespace rollout {
namespace {

constexpr int SB = 1024;
constexpr int NW = SB / 64;
typedef unsigned long long u64;

__device__ __forceinline__ u64 fx40(float e) { return (u64)(e * 1099511627776.0f); }

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

__global__ __launch_bounds__(SB) void k_sample(const float* __restrict__ logits, int V, float T, float top_p,
                                               const float* __restrict__ u, int u_stride,
                                               const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                               int out_stride) {
  __shared__ float redf[NW];
  __shared__ int redi[NW];
  __shared__ u64 redu[NW], redt[NW];
  __shared__ u64 hist[NW][256];
  __shared__ u64 sh_above;
  __shared__ unsigned sh_prefix;
  __shared__ int sh_tok;

  const int row = blockIdx.x;
  const float* z = logits + (size_t)row * V;
  const int c = col ? col[0] : 0;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int32_t* dst = out + (size_t)row * out_stride + c;

  if (T == 0.0f) {
    float best = -INFINITY;
    int bi = INT_MAX;
    for (int i = tid; i < V; i += SB) {
      const float v = z[i];
      if (v > best) { best = v; bi = i; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
    }
    if (lane == 0) { redf[w] = best; redi[w] = bi; }
    __syncthreads();
    if (tid == 0) {
      for (int i = 1; i < NW; ++i)
        if (redf[i] > best || (redf[i] == best && redi[i] < bi)) { best = redf[i]; bi = redi[i]; }
      *dst = bi == INT_MAX ? 0 : bi;
    }
    return;
  }

  // max of y = z / T
  float mx = -INFINITY;
  for (int i = tid; i < V; i += SB) mx = fmaxf(mx, z[i] / T);
  mx = wave_max(mx);
  if (lane == 0) redf[w] = mx;
  __syncthreads();
  mx = redf[0];
  for (int i = 1; i < NW; ++i) mx = fmaxf(mx, redf[i]);

  // total mass
  u64 part = 0;
  for (int i = tid; i < V; i += SB) part += fx40(expf(z[i] / T - mx));
  part = wave_sum_u64(part);
  if (lane == 0) redu[w] = part;
  __syncthreads();
  u64 total = 0;
  for (int i = 0; i < NW; ++i) total += redu[i];

  const bool filter = top_p < 1.0f;
  unsigned tau = 0;
  u64 ftau = 0, kties = 0, kept = total;
  if (filter) {
    u64 target = (u64)ceil((double)top_p * (double)total);
    if (target > total) target = total;
    if (target == 0) target = 1;
    unsigned prefix = 0, mask = 0;
    u64 above = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < NW * 256; i += SB) (&hist[0][0])[i] = 0;
      __syncthreads();
      for (int i = tid; i < V; i += SB) {
        const float e = expf(z[i] / T - mx);
        const unsigned b = __float_as_uint(e);
        if ((b & mask) == prefix) atomicAdd(&hist[w][(b >> shift) & 255u], fx40(e));
      }
      __syncthreads();
      if (tid < 256) {  // fold the per-wave histograms into hist[0]
        u64 t = 0;
        for (int j = 0; j < NW; ++j) t += hist[j][tid];
        hist[0][tid] = t;
      }
      __syncthreads();
      if (tid == 0) {
        u64 cum = above;
        int sel = 0;
        for (int dgt = 255; dgt >= 0; --dgt) {
          if (cum + hist[0][dgt] >= target) { sel = dgt; break; }
          cum += hist[0][dgt];
        }
        sh_above = cum;
        sh_prefix = prefix | ((unsigned)sel << shift);
      }
      __syncthreads();
      above = sh_above;
      prefix = sh_prefix;
      mask |= 255u << shift;
    }
    tau = prefix;
    ftau = fx40(__uint_as_float(tau));
    const u64 need = target - above;
    kties = ftau ? (need + ftau - 1) / ftau : (u64)V;
    kept = above + kties * ftau;
  }

  // ordered draw: wave w owns ids [w*seg, w*seg + seg)
  const int seg = ((V + NW - 1) / NW + 63) / 64 * 64;
  const int lo = min(V, w * seg), hi = min(V, lo + seg);
  u64 gt_mass = 0, ties = 0;
  for (int i = lo + lane; i < hi; i += 64) {
    const float e = expf(z[i] / T - mx);
    const unsigned b = __float_as_uint(e);
    if (!filter || b > tau) gt_mass += fx40(e);
    else if (b == tau) ties += 1;
  }
  gt_mass = wave_sum_u64(gt_mass);
  ties = wave_sum_u64(ties);
  if (lane == 0) { redt[w] = ties; }
  if (tid == 0) sh_tok = -1;
  __syncthreads();
  u64 ties_before = 0;
  for (int j = 0; j < w; ++j) ties_before += redt[j];
  const u64 my_kept_ties = filter ? (kties > ties_before ? min(kties - ties_before, ties) : 0) : 0;
  const u64 my_mass = gt_mass + my_kept_ties * ftau;
  if (lane == 0) redu[w] = my_mass;
  __syncthreads();
  u64 excl = 0;
  for (int j = 0; j < w; ++j) excl += redu[j];
  const double uval = (double)u[(size_t)row * u_stride + c];
  const u64 thresh = (u64)(uval * (double)kept);
  if (my_mass > 0 && excl <= thresh && thresh < excl + my_mass) {
    u64 carry = excl, tie_carry = 0;
    for (int base = lo; base < hi; base += 64) {
      const int i = base + lane;
      float e = 0.f;
      unsigned b = 0;
      if (i < hi) {
        e = expf(z[i] / T - mx);
        b = __float_as_uint(e);
      }
      bool keep = i < hi && (!filter || b > tau);
      const bool is_tie = filter && i < hi && b == tau;
      if (filter) {
        const u64 tie_incl = wave_incl_scan(is_tie ? 1ull : 0ull, lane);
        const u64 rank = tie_carry + tie_incl - (is_tie ? 1 : 0);
        if (is_tie && rank < my_kept_ties) keep = true;
        tie_carry += __shfl(tie_incl, 63, 64);
      }
      const u64 mass = keep ? fx40(e) : 0;
      const u64 cum = carry + wave_incl_scan(mass, lane);
      const unsigned long long hit = __ballot(keep && cum > thresh);
      if (hit) {
        const int first = __ffsll((long long)hit) - 1;
        if (lane == first) sh_tok = i;
        break;
      }
      carry = __shfl(cum, 63, 64);
    }
  }
  // largest kept id, for the case rounding leaves no crossing
  int last = -1;
  for (int i = tid; i < V; i += SB) {
    const unsigned b = __float_as_uint(expf(z[i] / T - mx));
    if (!filter || b > tau || (b == tau && kties > 0)) last = i;
  }
  last = max(last, __shfl_xor(last, 32, 64));
  last = max(last, __shfl_xor(last, 16, 64));
  last = max(last, __shfl_xor(last, 8, 64));
  last = max(last, __shfl_xor(last, 4, 64));
  last = max(last, __shfl_xor(last, 2, 64));
  last = max(last, __shfl_xor(last, 1, 64));
  if (lane == 0) redi[w] = last;
  __syncthreads();
  if (tid == 0) {
    int tok = sh_tok;
    if (tok < 0) {
      for (int j = 0; j < NW; ++j) tok = max(tok, redi[j]);
      tok = max(tok, 0);
    }
    *dst = tok;
  }
}

}  // namespace

hipError_t launch_sample(hipStream_t s, const float* logits, int S, int V, float temperature, float top_p,
                         const float* u, int u_stride, const int32_t* col, int32_t* out, int out_stride) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_sample, dim3(S), dim3(SB), 0, s, logits, V, temperature, top_p, u, u_stride, col, out,
                     out_stride);
  return hipGetLastError();
}

}  // namespace rollout
