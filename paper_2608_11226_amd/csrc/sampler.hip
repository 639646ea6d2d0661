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
// top-p threshold is a most-significant-digit radix select over the IEEE bit
// patterns of e (monotonic for e >= 0): four 8-bit digits with mass
// histograms.
//
// Three launches per batch of rows: (1) per-chunk maxima of y, (2) e_i
// computed once and stored, with per-chunk masses and first-digit histograms
// (rows x chunks workgroups keep every CU busy), (3) one workgroup per row
// finishes the radix select and the ordered draw reading only the stored e.
// Every pass over a row is coalesced: for the ordered draw each wave owns a
// contiguous segment of ids, segment totals are scanned across waves, and only
// the wave whose segment holds the crossing walks it, 64 ids at a time.
#include "internal.h"

#include <climits>

namespace rollout {
namespace {

constexpr int SB = 1024;  // threads of the per-row kernels
constexpr int NW = SB / 64;
constexpr int CB = 256;   // threads of the per-chunk kernels
typedef unsigned long long u64;

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

__global__ __launch_bounds__(SB) void k_argmax(const float* __restrict__ logits, int V,
                                               const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                               int out_stride) {
  __shared__ float redf[NW];
  __shared__ int redi[NW];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* z = logits + (size_t)row * V;
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
    out[(size_t)row * out_stride + (col ? col[0] : 0)] = bi == INT_MAX ? 0 : bi;
  }
}

// (1) cmax[row][c] = max over chunk c of fp32(z / T)
__global__ __launch_bounds__(CB) void k_chunk_max(const float* __restrict__ logits, int V, int chunk, float T,
                                                  float* __restrict__ cmax) {
  __shared__ float red[CB / 64];
  const int row = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  const float* z = logits + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  float mx = -INFINITY;
  for (int i = lo + tid; i < hi; i += CB) mx = fmaxf(mx, z[i] / T);
  mx = wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  if (tid == 0) {
    for (int j = 1; j < CB / 64; ++j) mx = fmaxf(mx, red[j]);
    cmax[(size_t)row * gridDim.y + c] = mx;
  }
}

// (2) e = exp(y - m) stored; per-chunk mass; first-digit mass histogram when filtering
__global__ __launch_bounds__(CB) void k_chunk_exp(const float* __restrict__ logits, int V, int chunk, float T,
                                                  const float* __restrict__ cmax, float* __restrict__ escr,
                                                  u64* __restrict__ cmass, u64* __restrict__ chist, int filter) {
  __shared__ u64 hist[CB / 64][256];
  __shared__ u64 red[CB / 64];
  const int row = blockIdx.x, c = blockIdx.y, nc = gridDim.y, tid = threadIdx.x, w = tid >> 6;
  float m = -INFINITY;
  for (int j = 0; j < nc; ++j) m = fmaxf(m, cmax[(size_t)row * nc + j]);
  const float* z = logits + (size_t)row * V;
  float* e_row = escr + (size_t)row * V;
  const int lo = c * chunk, hi = min(V, lo + chunk);
  if (filter) {
    for (int i = tid; i < (CB / 64) * 256; i += CB) (&hist[0][0])[i] = 0;
    __syncthreads();
  }
  u64 mass = 0;
  for (int i = lo + tid; i < hi; i += CB) {
    const float e = expf(z[i] / T - m);
    e_row[i] = e;
    const u64 f = fx40(e);
    mass += f;
    if (filter) atomicAdd(&hist[w][__float_as_uint(e) >> 24], f);
  }
  mass = wave_sum_u64(mass);
  if ((tid & 63) == 0) red[w] = mass;
  __syncthreads();
  if (tid == 0) {
    u64 t = 0;
    for (int j = 0; j < CB / 64; ++j) t += red[j];
    cmass[(size_t)row * nc + c] = t;
  }
  if (filter) {
    u64 t = 0;
    for (int j = 0; j < CB / 64; ++j) t += hist[j][tid];
    chist[((size_t)row * nc + c) * 256 + tid] = t;
  }
}

// (3) finish the radix select and draw, one workgroup per row
__global__ __launch_bounds__(SB) void k_select_draw(const float* __restrict__ escr, int V, int nc, float top_p,
                                                    const u64* __restrict__ cmass, const u64* __restrict__ chist,
                                                    const float* __restrict__ u, int u_stride,
                                                    const int32_t* __restrict__ col, int32_t* __restrict__ out,
                                                    int out_stride) {
  __shared__ u64 hist[NW][256];
  __shared__ u64 redu[NW], redt[NW];
  __shared__ u64 sh_above;
  __shared__ unsigned sh_prefix;
  __shared__ int sh_tok;
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* e_row = escr + (size_t)row * V;
  const int c = col ? col[0] : 0;

  u64 total = 0;
  for (int j = 0; j < nc; ++j) total += cmass[(size_t)row * nc + j];

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
      if (shift == 24) {
        if (tid < 256) {
          u64 t = 0;
          for (int j = 0; j < nc; ++j) t += chist[((size_t)row * nc + j) * 256 + tid];
          hist[0][tid] = t;
        }
        __syncthreads();
      } else {
        for (int i = tid; i < NW * 256; i += SB) (&hist[0][0])[i] = 0;
        __syncthreads();
        for (int i = tid; i < V; i += SB) {
          const float e = e_row[i];
          const unsigned b = __float_as_uint(e);
          if ((b & mask) == prefix) atomicAdd(&hist[w][(b >> shift) & 255u], fx40(e));
        }
        __syncthreads();
        if (tid < 256) {
          u64 t = 0;
          for (int j = 0; j < NW; ++j) t += hist[j][tid];
          hist[0][tid] = t;
        }
        __syncthreads();
      }
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
      __syncthreads();
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
    const float e = e_row[i];
    const unsigned b = __float_as_uint(e);
    if (!filter || b > tau) gt_mass += fx40(e);
    else if (b == tau) ties += 1;
  }
  gt_mass = wave_sum_u64(gt_mass);
  ties = wave_sum_u64(ties);
  if (lane == 0) redt[w] = ties;
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
  // thresh < kept always (u < 1 and kept >= 2^40), so some kept id crosses it
  const u64 thresh = (u64)((double)u[(size_t)row * u_stride + c] * (double)kept);
  if (my_mass > 0 && excl <= thresh && thresh < excl + my_mass) {
    u64 carry = excl, tie_carry = 0;
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
        if (lane == __ffsll((long long)hit) - 1) sh_tok = i;
        break;
      }
      carry = __shfl(cum, 63, 64);
    }
  }
  __syncthreads();
  if (tid == 0) out[(size_t)row * out_stride + c] = sh_tok < 0 ? 0 : sh_tok;
}

}  // namespace

int sample_chunks(int V) {
  const int c = (V + 4095) / 4096;
  return c < 1 ? 1 : (c > 64 ? 64 : c);
}

size_t sample_scratch_bytes(int S, int V) {
  const int nc = sample_chunks(V);
  return (size_t)S * V * 4 + (size_t)S * nc * (4 + 8 + 256 * 8) + 1024;
}

hipError_t launch_sample(hipStream_t s, const float* logits, int S, int V, float temperature, float top_p,
                         const float* u, int u_stride, const int32_t* col, int32_t* out, int out_stride,
                         void* scratch) {
  if (S <= 0) return hipSuccess;
  if (temperature == 0.0f) {
    hipLaunchKernelGGL(k_argmax, dim3(S), dim3(SB), 0, s, logits, V, col, out, out_stride);
    return hipGetLastError();
  }
  const int nc = sample_chunks(V);
  const int chunk = (V + nc - 1) / nc;
  char* p = (char*)scratch;
  float* escr = (float*)p;
  p += ((size_t)S * V * 4 + 255) / 256 * 256;
  u64* cmass = (u64*)p;
  p += ((size_t)S * nc * 8 + 255) / 256 * 256;
  float* cmax = (float*)p;
  p += ((size_t)S * nc * 4 + 255) / 256 * 256;
  u64* chist = (u64*)p;
  const int filter = top_p < 1.0f;
  hipLaunchKernelGGL(k_chunk_max, dim3(S, nc), dim3(CB), 0, s, logits, V, chunk, temperature, cmax);
  hipLaunchKernelGGL(k_chunk_exp, dim3(S, nc), dim3(CB), 0, s, logits, V, chunk, temperature, cmax, escr, cmass,
                     chist, filter);
  hipLaunchKernelGGL(k_select_draw, dim3(S), dim3(SB), 0, s, escr, V, nc, top_p, cmass, chist, u, u_stride, col,
                     out, out_stride);
  return hipGetLastError();
}

}  // namespace rollout
