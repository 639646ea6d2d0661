// Token sampler: temperature, nucleus (top-p) truncation by radix select, and
// an inverse-CDF draw with a caller-supplied uniform.  One workgroup of 1024
// threads per row of logits.
//
// Definition (per row z, temperature T, top_p, uniform u):
//   T == 0: greedy arg max, lowest id among equal maxima.
//   y_i = fp32(z_i / T), m = max y, e_i = fp32 exp(y_i - m).
//   top_p < 1: keep the shortest prefix, in (e descending, id ascending)
//   order, whose mass reaches top_p of the total; otherwise keep all.
//   Walk the kept ids in ascending order and return the first whose running
//   mass exceeds u times the kept mass.
//
// Masses are accumulated as fixed-point integers, e * 2^40 truncated (exact
// for e >= 2^-16, below 2^-40 of error each otherwise), so every sum, scan
// and comparison is exact integer arithmetic and the draw does not depend on
// thread scheduling.  The top-p threshold is found by a most-significant-digit
// radix select over the IEEE bit patterns of e (monotonic for e >= 0), four
// 8-bit digits, with mass (not count) histograms in LDS.
#include "internal.h"

#include <climits>

namespace rollout {
namespace {

constexpr int SB = 1024;
typedef unsigned long long u64;

__device__ __forceinline__ u64 fx40(float e) { return (u64)(e * 1099511627776.0f); }

__device__ __forceinline__ float block_max_f(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = red[0];
  for (int i = 1; i < SB / 64; ++i) t = fmaxf(t, red[i]);
  return t;
}

__device__ __forceinline__ u64 wave_incl_scan(u64 v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const u64 t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// Exclusive prefix sum over the block in thread order; *total receives the sum.
__device__ __forceinline__ u64 block_excl_scan(u64 v, u64* red, u64* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const u64 inc = wave_incl_scan(v);
  __syncthreads();
  if (lane == 63) red[w] = inc;
  __syncthreads();
  u64 before = 0, all = 0;
  for (int i = 0; i < SB / 64; ++i) {
    if (i < w) before += red[i];
    all += red[i];
  }
  *total = all;
  return before + inc - v;
}

__global__ __launch_bounds__(SB) void k_sample(const float* __restrict__ logits, int V, float T, float top_p,
                                               const float* __restrict__ u, int u_stride,
                                               const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                               int out_stride) {
  __shared__ float redf[SB / 64];
  __shared__ int redi[SB / 64];
  __shared__ u64 redu[SB / 64];
  __shared__ u64 hist[256];
  __shared__ u64 sh_above;
  __shared__ unsigned sh_prefix;
  __shared__ int sh_found, sh_last;

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
      for (int i = 1; i < SB / 64; ++i)
        if (redf[i] > best || (redf[i] == best && redi[i] < bi)) { best = redf[i]; bi = redi[i]; }
      *dst = bi == INT_MAX ? 0 : bi;
    }
    return;
  }

  // max of y = z / T
  float mx = -INFINITY;
  for (int i = tid; i < V; i += SB) mx = fmaxf(mx, z[i] / T);
  mx = block_max_f(mx, redf);

  // total mass
  u64 part = 0;
  for (int i = tid; i < V; i += SB) part += fx40(expf(z[i] / T - mx));
  u64 total;
  (void)block_excl_scan(part, redu, &total);

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
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < V; i += SB) {
        const float e = expf(z[i] / T - mx);
        const unsigned b = __float_as_uint(e);
        if ((b & mask) == prefix) atomicAdd(&hist[(b >> shift) & 255u], fx40(e));
      }
      __syncthreads();
      if (tid == 0) {
        u64 cum = above;
        int sel = 0;
        for (int dgt = 255; dgt >= 0; --dgt) {
          if (cum + hist[dgt] >= target) { sel = dgt; break; }
          cum += hist[dgt];
        }
        sh_above = cum;
        sh_prefix = prefix | ((unsigned)sel << shift);
      }
      __syncthreads();
      above = sh_above;
      prefix = sh_prefix;
      mask |= 255u << shift;
      __syncthreads();
    }
    tau = prefix;
    ftau = fx40(__uint_as_float(tau));
    const u64 need = target - above;
    kties = ftau ? (need + ftau - 1) / ftau : (u64)V;
    kept = above + kties * ftau;
  }

  // draw: contiguous id ranges per thread, exact scans of tie counts and kept mass
  const int chunk = (V + SB - 1) / SB;
  const int lo = min(V, tid * chunk), hi = min(V, lo + chunk);
  u64 mine = 0, nt = 0;
  int last_kept = -1;
  for (int i = lo; i < hi; ++i) {
    const float e = expf(z[i] / T - mx);
    const unsigned b = __float_as_uint(e);
    if (!filter || b > tau) { mine += fx40(e); last_kept = i; }
    else if (b == tau) nt += 1;
  }
  u64 all_ties;
  const u64 ties_before = block_excl_scan(nt, redu, &all_ties);
  if (filter) {
    const u64 kt = kties > ties_before ? min(kties - ties_before, nt) : 0;
    mine += kt * ftau;
    if (kt > 0) {  // the kept ties of this range are its first kt ties; find the last one
      u64 seen = 0;
      for (int i = lo; i < hi && seen < kt; ++i)
        if (__float_as_uint(expf(z[i] / T - mx)) == tau) { ++seen; last_kept = max(last_kept, i); }
    }
  }
  u64 kept_sum;
  const u64 excl = block_excl_scan(mine, redu, &kept_sum);
  (void)kept_sum;
  const double uval = (double)u[(size_t)row * u_stride + c];
  const u64 thresh = (u64)(uval * (double)kept);
  if (tid == 0) { sh_found = 0; sh_last = -1; }
  __syncthreads();
  atomicMax(&sh_last, last_kept);
  if (mine > 0 && excl <= thresh && thresh < excl + mine) {
    u64 cum = excl, seen = ties_before;
    for (int i = lo; i < hi; ++i) {
      const float e = expf(z[i] / T - mx);
      const unsigned b = __float_as_uint(e);
      bool keep = !filter || b > tau;
      if (filter && b == tau) keep = seen++ < kties;
      if (keep) {
        cum += fx40(e);
        if (cum > thresh) {
          *dst = i;
          sh_found = 1;
          break;
        }
      }
    }
  }
  __syncthreads();
  if (tid == 0 && !sh_found) *dst = sh_last < 0 ? 0 : sh_last;
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
