// Projection GEMMs: y[m][n] = sum_k X[m][k] * W[n][k], fp32 accumulation.
//
// bf16 path (CDNA4 MFMA, v_mfma_f32_16x16x32_bf16).  Both operands live in
// HBM in MFMA operand order, so every global load is a fully coalesced
// 16-byte-per-lane read:
//   W (A operand): fragments of 16 weight rows x 32 k (64 lanes x 8, lane =
//                  row%16 + 16*((k%32)/8)), the four fragments of 4
//                  consecutive row blocks adjacent at each k-step (wfrag) --
//                  written once at synthesis;
//   X (B operand): tiles of 32 k x 16 activation rows, [K/32][M/16][64][8],
//                  lane = m%16 + 16*((k%32)/8) -- written by the producing
//                  kernel (norm, SwiGLU, attention).
// Weights are read exactly once per step, with non-temporal loads (keeping
// them out of the caches leaves room for the activations).
//
// k_gemm_ring (decode, M <= 64 rows): a workgroup owns NBW 16-row weight
// blocks and one K split; its one or two waves each take a share of the split.
// Weight and activation fragments stream through a D-deep register ring with
// no LDS and no barriers; every load is unconditional (addresses clamped into
// range, surplus steps masked at the MFMA), so the compiler keeps D - 1 ring
// stages in flight instead of draining the load queue at every step.  X is
// read from L2 by every wave, which costs M/(16 NBW) of the weight bytes in L2
// traffic and nothing in HBM.  Two waves add their sums through LDS once, at
// the end.  With several K splits each writes a partial [split][M][N] that
// the consumer sums in split order.  The SwiGLU variant (gate/up, one split) finishes in
// registers: gate row i and up row i are adjacent weight rows, so the lane
// that holds one also holds the other, and h goes straight to the down
// projection's operand layout.
//
// Gate/up with SwiGLU at decode batches whose weight blocks give every CU 4 to 10 of them (7B) takes a
// balanced grid instead: one workgroup of two waves per CU, the blocks shared out evenly (BAL below); so
// does the LM head, with four one-wave workgroups per CU.
//
// k_gemm_wlds (decode batches of 129..256 rows): one workgroup holds all activation rows, so each weight
// byte enters one CU; the weights of a k-step are staged in LDS for the four waves and each wave reads its
// own activation rows straight from L2 (details at the kernel).
//
// k_gemm_tile (prefill, and batches of 65..128 or more than 256 rows): a workgroup of four
// waves owns 256 weight rows x 128 activation rows; each wave owns its own 64
// weight rows against all 128 activation rows (4 x 8 MFMA tiles, 128
// accumulator registers, two waves per SIMD).  The weights never touch LDS:
// each wave streams its own weight fragments from global memory straight into
// a three-deep register ring (no two waves read the same weight fragment).
// The activation fragments are shared by the four waves through a double LDS
// buffer, staged global -> registers -> LDS three k-steps ahead.  Per k-step
// a wave reads 8 KB from LDS for 32 MFMAs; one barrier per k-step.  All waits
// are compiler-placed on loads issued a step or more earlier.  Workgroup order
// is XCD-aware: the M tiles of one N tile run on one XCD, so its weight tile
// is fetched into that XCD's L2 once and served to the rest from there.
//
// k_gemm_q4 (decode with int4 layer weights, M <= 64): weights as 4-bit codes
// in groups of 128 inputs with an fp32 scale and a zero point per row and
// group; the group's scale multiplies its integer dot product in fp32, so the
// weights are never rounded.  The codes enter the MFMA as exact bf16 integers
// (128 + q); a workgroup of four waves shares each group's activation
// fragments and their sums through LDS.  Larger batches with int4 weights
// dequantise a projection into two bf16 tile matrices (hi + lo) and take the
// tile kernel twice.
//
// fp32 path: a plain LDS-tiled VALU GEMM over row-major X and W (the fp32
// path exists for exact parity on small models, not for speed).
#include <algorithm>
#include <cstdlib>

#include "internal.h"

namespace rollout {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// Tile kernel: 4 waves; a workgroup owns NB 16-row weight blocks per wave against MBW 16-row activation
// blocks (NB = 4, MBW = 8: 256 weight rows x 128 activation rows, each wave 64 x 128).
constexpr int kTileWaves = 4;
constexpr int kTileNB = 4, kTileMB = 8;

// SWI: gate/up with SwiGLU applied to the output (one K split): h in the down projection's operand layout
// XD: activation register stages (each k-step's X fragments are loaded XD steps before they are staged
// into LDS); OCC: waves per SIMD the registers are sized for.  Batches above 256 rows (prefill, MFMA-bound)
// take XD = 3 at two waves per SIMD; decode-sized batches, one wave per SIMD anyway, take XD = 6.
// Workgroups run in XCD-aware order: the M tiles of one N tile share one XCD and its L2.
template <int NB, int MBW, bool SWI, int XD, int OCC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void k_gemm_tile(const bf16x8_t* __restrict__ XF, const bf16x8_t* __restrict__ W, float* __restrict__ out,
                 int M, int N, int K, int kslice, uint16_t* __restrict__ h) {
  constexpr int XPW = MBW / kTileWaves;  // activation fragments each wave stages per k-step
  __shared__ bf16x8_t xs[2][MBW][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nbt = N >> 4, kbt = K >> 5, Mb = (M + 15) >> 4;
  const int Mt = (Mb + MBW - 1) / MBW, Nt = (nbt + NB * kTileWaves - 1) / (NB * kTileWaves);
  // XCD-aware order (workgroup b runs on XCD b % 8): the M tiles of N tile nt share one XCD and its L2
  const int b = blockIdx.x;
  const int grp = b / (8 * Mt), rem = b % (8 * Mt);
  const int nt = grp * 8 + rem % 8, mt = rem / 8;
  if (nt >= Nt) return;
  // the workgroup's first weight block and its block count, its first activation block
  const int wb0 = nt * NB * kTileWaves, wbc = min(NB * kTileWaves, nbt - wb0), mb0 = mt * MBW;
  const int lb0 = wave * NB;  // the wave's first block within the workgroup's
  const int kb0 = (int)blockIdx.y * (kslice >> 5);
  const int nk = min(kbt, kb0 + (kslice >> 5)) - kb0;
  floatx4_t acc[NB][MBW];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int i = 0; i < MBW; ++i) acc[j][i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  if (nk > 0) {
    // every load is unconditional: block and k indices are clamped into range, surplus k-steps are not computed
    const bf16x8_t* wp[NB];
    int ws[NB];  // k-step stride of each block's fragments
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int nb = wb0 + min(lb0 + j, wbc - 1);
      wp[j] = W + wfrag(nb, kb0, nbt, kbt) * 64 + lane;
      ws[j] = wgroup_blocks(nb, nbt) * 64;
    }
    const bf16x8_t* xp[XPW];
#pragma unroll
    for (int i = 0; i < XPW; ++i)
      xp[i] = XF + ((size_t)kb0 * Mb + min(mb0 + XPW * wave + i, Mb - 1)) * 64 + lane;
    const size_t xstride = (size_t)Mb * 64;
    static_assert(6 % XD == 0, "the k-step loop is unrolled by 6");
    bf16x8_t wr[3][NB], xg[XD][XPW];
    auto load_w = [&](int slot, int st) {
      const size_t kk = (size_t)min(st, nk - 1);
#pragma unroll
      for (int j = 0; j < NB; ++j) wr[slot][j] = wp[j][kk * ws[j]];
    };
    auto load_x = [&](int slot, int st) {
      const size_t kk = (size_t)min(st, nk - 1);
#pragma unroll
      for (int i = 0; i < XPW; ++i) xg[slot][i] = xp[i][kk * xstride];
    };
    auto stage_x = [&](int buf, int slot) {
#pragma unroll
      for (int i = 0; i < XPW; ++i) xs[buf][XPW * wave + i][lane] = xg[slot][i];
    };
    // k-step st computes from LDS buffer st % 2 and weight slot st % 3.  Before it, the step loads
    // W(st + 2), writes X(st + 1) (loaded XD steps earlier, register slot (st + 1) % XD) into the other LDS
    // buffer and loads X(st + 1 + XD) into that slot; every wait the compiler inserts is then on loads
    // issued at least one step earlier.
    load_w(0, 0);
    load_w(1, 1);
#pragma unroll
    for (int d = 0; d < XD; ++d) load_x(d, d);
    stage_x(0, 0);
    load_x(0, XD);
    lds_barrier();
    for (int s0 = 0; s0 < nk; s0 += 6) {
#pragma unroll
      for (int u = 0; u < 6; ++u) {
        const int st = s0 + u;
        load_w((u + 2) % 3, st + 2);
        stage_x((u + 1) & 1, (u + 1) % XD);
        load_x((u + 1) % XD, st + 1 + XD);
        if (st < nk) {
#pragma unroll
          for (int i = 0; i < MBW; ++i) {
            const bf16x8_t xf = xs[u & 1][i][lane];
#pragma unroll
            for (int j = 0; j < NB; ++j)
              acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[u % 3][j], xf, acc[j][i], 0, 0, 0);
          }
          // two LDS fragment reads ahead of the MFMAs, then one more per fragment's NB MFMAs
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
          for (int i = 0; i < MBW - 2; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, NB, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
        }
        lds_barrier();
      }
    }
  }
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
  float* o = out + (size_t)blockIdx.y * M * N;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (lb0 + j >= wbc) continue;
    const int n = (wb0 + lb0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < MBW; ++i) {
      const int m = (mb0 + i) * 16 + (lane & 15);
      if (m >= M) continue;
      if constexpr (SWI) {
        // rows n, n+1 are (gate, up) of output f = n/2; rows n+2, n+3 of output f + 1
        const float g0 = acc[j][i][0], u0 = acc[j][i][1], g1 = acc[j][i][2], u1 = acc[j][i][3];
        const float h0 = g0 / (1.0f + expf(-g0)) * u0, h1 = g1 / (1.0f + expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(h + xoff(h, m, n >> 1, N >> 1, Mb)) = pack_bf16x2(h0, h1);
      } else {
        *reinterpret_cast<float4*>(o + (size_t)m * N + n) = make_float4(acc[j][i][0], acc[j][i][1], acc[j][i][2], acc[j][i][3]);
      }
    }
  }
}

// Tall decode batches (129..256 rows), weights staged in LDS: a workgroup of four waves owns up to
// kWldsBlocks weight blocks (128 rows; the grid shares the blocks out evenly, floor(nbt / grid) or one more
// each) and all 16 activation blocks; wave w owns activation blocks 4w .. 4w + 3 against every weight block
// of the workgroup (8 x 4 MFMA tiles).  A k-step's weight fragments (8 KB) are streamed from HBM once per
// workgroup -- each wave stages two of them, global -> registers (three steps ahead) -> LDS (double
// buffered) -- and read from LDS by all four waves, while each wave loads its own activation fragments
// from L2 straight into registers, XD steps ahead.  Per k-step and CU: 40 KB of LDS traffic for 128 MFMAs
// (staging the 16 KB activation tile instead would take 80 KB), and every weight byte enters one CU.
// One LDS barrier per k-step; loads are unconditional (indices clamped, surplus steps not computed).
constexpr int kWldsBlocks = 8;
template <bool SWI, int XD, int WD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_gemm_wlds(const bf16x8_t* __restrict__ XF, const bf16x8_t* __restrict__ W, float* __restrict__ out, int M,
                 int N, int K, int kslice, uint16_t* __restrict__ h) {
  constexpr int NBG = kWldsBlocks;           // weight blocks per workgroup
  constexpr int MBV = 4;                     // activation blocks per wave
  constexpr int WPW = NBG / kTileWaves;      // weight fragments each wave stages per k-step
  __shared__ bf16x8_t wl[2][NBG][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nbt = N >> 4, kbt = K >> 5, Mb = (M + 15) >> 4;
  const int wb0 = (int)((long long)blockIdx.x * nbt / gridDim.x);
  const int wbc = (int)((long long)(blockIdx.x + 1) * nbt / gridDim.x) - wb0;
  const int kb0 = (int)blockIdx.y * (kslice >> 5);
  const int nk = min(kbt, kb0 + (kslice >> 5)) - kb0;
  floatx4_t acc[NBG][MBV];
#pragma unroll
  for (int j = 0; j < NBG; ++j)
#pragma unroll
    for (int i = 0; i < MBV; ++i) acc[j][i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  if (nk > 0) {
    const bf16x8_t* wp[WPW];
    int wsd[WPW];  // k-step stride of each staged block's fragments
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int nb = wb0 + min(WPW * wave + j, wbc - 1);
      wp[j] = W + wfrag(nb, kb0, nbt, kbt) * 64 + lane;
      wsd[j] = wgroup_blocks(nb, nbt) * 64;
    }
    const bf16x8_t* xp[MBV];
#pragma unroll
    for (int i = 0; i < MBV; ++i) xp[i] = XF + ((size_t)kb0 * Mb + min(MBV * wave + i, Mb - 1)) * 64 + lane;
    const size_t xstride = (size_t)Mb * 64;
    static_assert(6 % XD == 0 && 6 % WD == 0 && WD >= 3, "the k-step loop is unrolled by 6");
    bf16x8_t wg[WD][WPW], xr[XD][MBV], wf[2][NBG];
    auto load_w = [&](int slot, int st) {
      const size_t kk = (size_t)min(st, nk - 1);
#pragma unroll
      for (int j = 0; j < WPW; ++j) wg[slot][j] = __builtin_nontemporal_load(wp[j] + kk * wsd[j]);
    };
    auto store_w = [&](int buf, int slot) {
#pragma unroll
      for (int j = 0; j < WPW; ++j) wl[buf][WPW * wave + j][lane] = wg[slot][j];
    };
    auto read_w = [&](int reg, int buf) {
#pragma unroll
      for (int j = 0; j < NBG; ++j) wf[reg][j] = wl[buf][j][lane];
    };
    auto load_x = [&](int slot, int st) {
      const size_t kk = (size_t)min(st, nk - 1);
#pragma unroll
      for (int i = 0; i < MBV; ++i) xr[slot][i] = xp[i][kk * xstride];
    };
    // W(k) passes through global register slot k % WD, LDS buffer k % 2 and fragment registers wf[k % 2].
    // k-step st multiplies wf[st % 2] (read from LDS during step st - 1) with activation slot st % XD, and
    // meanwhile reads W(st + 1) out of LDS, writes W(st + 2) into the LDS buffer W(st) came from (every wave
    // finished reading it before the barrier that ended step st - 1), loads W(st + 2 + WD) into the freed
    // register slot and X(st + XD) into its slot.  WD - 2 steps of weights stay in flight; one barrier per
    // step.
#pragma unroll
    for (int d = 0; d < WD; ++d) load_w(d, d);
#pragma unroll
    for (int d = 0; d < XD; ++d) load_x(d, d);
    store_w(0, 0);
    store_w(1, 1);
    load_w(0, WD);
    load_w(1, WD + 1);
    lds_barrier();
    read_w(0, 0);
    lds_barrier();  // every wave holds W(0) before step 0 overwrites LDS buffer 0
    for (int s0 = 0; s0 < nk; s0 += 6) {
#pragma unroll
      for (int u = 0; u < 6; ++u) {
        const int st = s0 + u;
        read_w((u + 1) & 1, (u + 1) & 1);
        store_w(u & 1, (u + 2) % WD);
        load_w((u + 2) % WD, st + 2 + WD);
        if (st < nk) {
#pragma unroll
          for (int j = 0; j < NBG; ++j)
#pragma unroll
            for (int i = 0; i < MBV; ++i)
              acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[u & 1][j], xr[u % XD][i], acc[j][i], 0, 0, 0);
        }
        load_x(u % XD, st + XD);
        lds_barrier();
      }
    }
  }
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
  float* o = out + (size_t)blockIdx.y * M * N;
#pragma unroll
  for (int j = 0; j < NBG; ++j) {
    if (j >= wbc) continue;
    const int n = (wb0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < MBV; ++i) {
      const int m = (MBV * wave + i) * 16 + (lane & 15);
      if (m >= M) continue;
      if constexpr (SWI) {
        // rows n, n+1 are (gate, up) of output f = n/2; rows n+2, n+3 of output f + 1
        const float g0 = acc[j][i][0], u0 = acc[j][i][1], g1 = acc[j][i][2], u1 = acc[j][i][3];
        const float h0 = g0 / (1.0f + expf(-g0)) * u0, h1 = g1 / (1.0f + expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(h + xoff(h, m, n >> 1, N >> 1, Mb)) = pack_bf16x2(h0, h1);
      } else {
        *reinterpret_cast<float4*>(o + (size_t)m * N + n) = make_float4(acc[j][i][0], acc[j][i][1], acc[j][i][2], acc[j][i][3]);
      }
    }
  }
}

// MB = ceil(M/16) row blocks of X; NBW weight blocks per wave; D ring stages; KW waves per workgroup, which
// split the workgroup's K slice between them and add their sums through LDS (in wave order) before the
// epilogue, so a workgroup writes one partial however many waves it has.
// BAL: the grid's workgroups share the N/16 weight blocks out evenly, floor(nbt / grid) or one more each
// (at most NBW), so that a grid of one workgroup per CU gives every CU the same work; otherwise workgroup x
// owns blocks NBW x .. NBW x + NBW - 1.  A workgroup with fewer than NBW blocks loads its last block again
// for the missing ones (a cache hit) and stores nothing for them.
template <int MB, int NBW, int D, bool SWI, int KW, bool BAL = false>
__global__ __launch_bounds__(64 * KW) void k_gemm_ring(const bf16x8_t* __restrict__ XF, const bf16x8_t* __restrict__ W,
                                                       float* __restrict__ out, int M, int N, int K, int kslice,
                                                       uint16_t* __restrict__ h) {
  const int lane = threadIdx.x & 63;
  const int wave = KW > 1 ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) : 0;
  const int nbt = N >> 4, kbt = K >> 5;
  int nb0, nbc;  // the workgroup's first weight block and its block count (>= 1)
  if constexpr (BAL) {
    nb0 = (int)((long long)blockIdx.x * nbt / gridDim.x);
    nbc = (int)((long long)(blockIdx.x + 1) * nbt / gridDim.x) - nb0;
  } else {
    nb0 = blockIdx.x * NBW;
    nbc = min(NBW, nbt - nb0);
  }
  const int kw0 = (int)blockIdx.y * (kslice >> 5);         // the workgroup's first k-step
  const int nkw = min(kbt, kw0 + (kslice >> 5)) - kw0;    // and its k-steps (none in a surplus split)
  const int per = (nkw + KW - 1) / KW;
  const int kb0 = kw0 + wave * per;
  const int nk = min(kw0 + nkw, kb0 + per) - kb0;         // this wave's k-steps; an empty share adds zeros
  if constexpr (KW == 1) {
    if (nk <= 0) {  // an empty K split contributes zeros
      if constexpr (!SWI) {
        for (int j = 0; j < nbc; ++j)
          for (int m = lane & 15; m < M; m += 16)
            *reinterpret_cast<float4*>(out + ((size_t)blockIdx.y * M + m) * N + (nb0 + j) * 16 + 4 * (lane >> 4)) =
                make_float4(0.f, 0.f, 0.f, 0.f);
      }
      return;
    }
  }
  floatx4_t acc[NBW][MB];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  if (nk > 0) {
    const bf16x8_t* wp[NBW];
    int ws[NBW];  // k-step stride of each block's fragments
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int nb = nb0 + min(j, nbc - 1);
      wp[j] = W + wfrag(nb, kb0, nbt, kbt) * 64 + lane;
      ws[j] = wgroup_blocks(nb, nbt) * 64;
    }
    const bf16x8_t* xp = XF + (size_t)kb0 * MB * 64 + lane;
    bf16x8_t wr[D][NBW], xr[D][MB];
    // ring stage d holds k-step min(i, nk - 1); steps past nk reload the last one and are not used
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const size_t kk = (size_t)min(d, nk - 1);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) xr[d][mb] = xp[(kk * MB + mb) * 64];
#pragma unroll
      for (int j = 0; j < NBW; ++j) wr[d][j] = __builtin_nontemporal_load(wp[j] + kk * ws[j]);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int i = 0; i < nk; i += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        if (i + d < nk) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < NBW; ++j)
              acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[d][j], xr[d][mb], acc[j][mb], 0, 0, 0);
        }
        const size_t kk = (size_t)min(i + d + D, nk - 1);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) xr[d][mb] = xp[(kk * MB + mb) * 64];
#pragma unroll
        for (int j = 0; j < NBW; ++j) wr[d][j] = __builtin_nontemporal_load(wp[j] + kk * ws[j]);
        // keeps the ring order through scheduling, so each stage waits only for its own loads
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  if constexpr (KW > 1) {
    // weight block j is finished by wave j % KW; the other waves hand it their sums through LDS
    static_assert(NBW % KW == 0, "weight blocks are shared out evenly");
    __shared__ floatx4_t red[KW - 1][NBW][MB][64];
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int o = j % KW;
      if (wave != o) {
        const int sl = wave < o ? wave : wave - 1;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) red[sl][j][mb][lane] = acc[j][mb];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int o = j % KW;
      if (wave == o) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          floatx4_t t = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int w = 0; w < KW; ++w) t += (w == o) ? acc[j][mb] : red[w < o ? w : w - 1][j][mb][lane];
          acc[j][mb] = t;
        }
      }
    }
  }
  // D layout of the 16x16 MFMA: lane holds rows 4*(lane/16)+r (weight rows n) of column lane%16 (row m of X)
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (j % KW != wave || j >= nbc) continue;
    const int n = (nb0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = mb * 16 + (lane & 15);
      if (m >= M) continue;
      if constexpr (SWI) {
        // rows n, n+1 are (gate, up) of output f = n/2; rows n+2, n+3 of output f + 1
        const float g0 = acc[j][mb][0], u0 = acc[j][mb][1], g1 = acc[j][mb][2], u1 = acc[j][mb][3];
        const float h0 = g0 / (1.0f + expf(-g0)) * u0, h1 = g1 / (1.0f + expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(h + xoff(h, m, n >> 1, N >> 1, MB)) = pack_bf16x2(h0, h1);
      } else {
        float* o = out + (size_t)blockIdx.y * M * N;
        *reinterpret_cast<float4*>(o + (size_t)m * N + n) =
            make_float4(acc[j][mb][0], acc[j][mb][1], acc[j][mb][2], acc[j][mb][3]);
      }
    }
  }
}

// int4 weights (format in synth.hip: codes [N/16][K/128][64][4 words] in AWQ nibble order, then fp32
// scales and uint8 zeros [N/16][K/128][16]), scaled per group: for a 128-input group g of row n,
//   y[m] += s[n,g] * sum_k (q[n,k] - z[n,g]) x[m,k].
// A code q enters the MFMA as the exact bf16 integer 128 + q (the nibble in the mantissa of 128: one
// shift and one and-or per pair of codes), so a group's MFMA partial is P = sum_k (128 + q) x.  One
// all-ones MFMA per group gives X = sum_k x[m,k], shared by the wave's weight blocks, and the group's
// epilogue adds s * (P - (128 + z) * X) to the fp32 accumulator.  The weights are never rounded.
// Ring over groups as in k_gemm_ring: per group and weight block one 16-byte code load, a 16-byte load
// of the four scales of the lane's accumulator rows and a 4-byte load of their zeros.
__device__ __forceinline__ bf16x8_t q4_operand(uint32_t w) {
  u32x4_t d;
  d[0] = (w & 0x000F000Fu) | 0x43004300u;
  d[1] = ((w >> 4) & 0x000F000Fu) | 0x43004300u;
  d[2] = ((w >> 8) & 0x000F000Fu) | 0x43004300u;
  d[3] = ((w >> 12) & 0x000F000Fu) | 0x43004300u;
  return __builtin_bit_cast(bf16x8_t, d);
}

// A workgroup of four waves shares the activation fragments of a group through LDS (double
// buffered: wave w loads k-step w of group i + 1 for every 16-row block while all compute group i,
// then stores it).  Wave w also forms that k-step's activation sums with MB all-ones MFMAs and
// publishes them; a group's sums X are the four waves' partials added in k-step order.  Each wave
// owns NBW weight blocks and keeps their codes, scales and zeros in a two-group register ring.
// One barrier per group.
template <int MB, int NBW, bool SWI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_gemm_q4(
    const bf16x8_t* __restrict__ XF, const u32x4_t* __restrict__ Wq, const floatx4_t* __restrict__ Ws,
    const uint32_t* __restrict__ Wz, float* __restrict__ out, int M, int N, int K, int kslice,
    uint16_t* __restrict__ h) {
  constexpr int D = 2;
  __shared__ bf16x8_t xl[2][4 * MB][64];
  __shared__ float xsl[2][4][MB][16];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nb0 = (blockIdx.x * 4 + wave) * NBW;
  const int nbt = N >> 4, gbt = K >> 7;
  const int kg0 = (int)blockIdx.y * (kslice >> 7);
  const int ng = min(gbt, kg0 + (kslice >> 7)) - kg0;
  if (ng <= 0) {  // an empty K split contributes zeros
    if constexpr (!SWI) {
      for (int j = 0; j < NBW && nb0 + j < nbt; ++j)
        for (int m = lane & 15; m < M; m += 16)
          *reinterpret_cast<float4*>(out + ((size_t)blockIdx.y * M + m) * N + (nb0 + j) * 16 + 4 * (lane >> 4)) =
              make_float4(0.f, 0.f, 0.f, 0.f);
    }
    return;
  }
  bf16x8_t ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = __builtin_bit_cast(__bf16, (uint16_t)0x3F80);
  floatx4_t acc[NBW][MB];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  {
    // wave-uniform bases of each block's first group (blocks past N: clamped, never stored)
    size_t item0[NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) item0[j] = (size_t)min(nb0 + j, nbt - 1) * gbt + kg0;
    const int wl = lane, sl = lane >> 4;
    // k-step `wave` of a group, every 16-row block: fragments wave * MB .. + MB - 1 of the group's 4 MB
    const bf16x8_t* xp = XF + (size_t)kg0 * 4 * MB * 64 + (size_t)wave * MB * 64;
    u32x4_t cr[D][NBW];
    floatx4_t sr[D][NBW];
    uint32_t zr[D][NBW];
    auto load_w = [&](int d, int gg) {
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const size_t it = item0[j] + (size_t)gg;
        cr[d][j] = __builtin_nontemporal_load(Wq + it * 64 + wl);
        sr[d][j] = Ws[it * 4 + sl];  // scales of rows 4 (lane / 16) .. + 3
        zr[d][j] = Wz[it * 4 + sl];
      }
    };
    bf16x8_t xst[MB];
    auto load_x = [&](int gg) {
#pragma unroll
      for (int f = 0; f < MB; ++f) xst[f] = xp[((size_t)gg * 4 * MB + f) * 64 + lane];
    };
    auto store_x = [&](int buf) {
#pragma unroll
      for (int f = 0; f < MB; ++f) {
        xl[buf][wave * MB + f][lane] = xst[f];
        const floatx4_t p = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, xst[f], floatx4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
        if (lane < 16) xsl[buf][wave][f][lane] = p[0];
      }
    };
    load_x(0);
    store_x(0);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      load_w(d, min(d, ng - 1));
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    for (int i = 0; i < ng; i += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int g = i + d;                  // group computed now, from LDS buffer g & 1 and ring slot d
        load_x(min(g + 1, ng - 1));           // next group's fragments (clamped past the end, never used)
        if (g < ng) {
          const int buf = g & 1;
          float xs[MB];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            const int m16 = lane & 15;
            xs[mb] = ((xsl[buf][0][mb][m16] + xsl[buf][1][mb][m16]) + xsl[buf][2][mb][m16]) + xsl[buf][3][mb][m16];
          }
#pragma unroll
          for (int j = 0; j < NBW; ++j) {
            floatx4_t pp[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) pp[mb] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const bf16x8_t a = q4_operand(cr[d][j][t]);
#pragma unroll
              for (int mb = 0; mb < MB; ++mb)
                pp[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, xl[buf][t * MB + mb][lane], pp[mb], 0, 0, 0);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float sc = sr[d][j][r];
              const float off = __uint_as_float(0x43000000u | (((zr[d][j] >> (8 * r)) & 0xFFu) << 16));  // 128 + z
#pragma unroll
              for (int mb = 0; mb < MB; ++mb) acc[j][mb][r] = fmaf(sc, fmaf(-off, xs[mb], pp[mb][r]), acc[j][mb][r]);
            }
          }
        }
        load_w(d, min(g + D, ng - 1));
        store_x((g + 1) & 1);  // buffer (g + 1) & 1 was last read for group g - 1, before the last barrier
        __syncthreads();
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (nb0 + j >= nbt) continue;
    const int n = (nb0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = mb * 16 + (lane & 15);
      if (m >= M) continue;
      if constexpr (SWI) {
        const float g0 = acc[j][mb][0], u0 = acc[j][mb][1], g1 = acc[j][mb][2], u1 = acc[j][mb][3];
        const float h0 = g0 / (1.0f + expf(-g0)) * u0, h1 = g1 / (1.0f + expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(h + xoff(h, m, n >> 1, N >> 1, MB)) = pack_bf16x2(h0, h1);
      } else {
        float* o = out + (size_t)blockIdx.y * M * N;
        *reinterpret_cast<float4*>(o + (size_t)m * N + n) =
            make_float4(acc[j][mb][0], acc[j][mb][1], acc[j][mb][2], acc[j][mb][3]);
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ X, int ldx, const float* __restrict__ W,
                                                  float* __restrict__ out, int M, int N, int K) {
  __shared__ float xs[16][33];
  __shared__ float ws[16][33];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int n0 = blockIdx.x * 16, m0 = blockIdx.y * 16;
  float acc = 0.f;
  for (int k0 = 0; k0 < K; k0 += 32) {
    for (int i = threadIdx.x; i < 512; i += 256) {
      const int r = i >> 5, c = i & 31;
      const int k = k0 + c;
      xs[r][c] = (m0 + r < M && k < K) ? X[(size_t)(m0 + r) * ldx + k] : 0.f;
      ws[r][c] = (n0 + r < N && k < K) ? W[(size_t)(n0 + r) * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 32; ++c) acc += xs[ty][c] * ws[tx][c];
    __syncthreads();
  }
  const int m = m0 + ty, n = n0 + tx;
  if (m < M && n < N) out[(size_t)m * N + n] = acc;
}

int kslice_for(int K, int splits) {
  const int per = (K + splits - 1) / splits;
  return (per + 31) / 32 * 32;
}

// Compute units of the current device (looked up once per device).
int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Tile kernel grid: (padded N tiles) x (M tiles) workgroups in XCD-aware order, K splits in y.
int tile_m_tiles(int M) { return ((M + 15) / 16 + kTileMB - 1) / kTileMB; }
int tile_n_tiles(int N) { return (N / 16 + kTileNB * kTileWaves - 1) / (kTileNB * kTileWaves); }
int tile_groups(int M, int N) { return (tile_n_tiles(N) + 7) / 8 * 8 * tile_m_tiles(M); }

// Tall decode batches (129..256 rows, one activation tile) take k_gemm_wlds on a balanced grid of
// workgroups with at most kWldsBlocks weight blocks each, about one per CU per K split.
constexpr int kTallMinRows = 129, kTallMaxRows = 256;
constexpr int kTallWgBlocks = kWldsBlocks;
bool tall_batch(int M) { return M >= kTallMinRows && M <= kTallMaxRows; }
int tall_groups(int N, int splits) {
  const int nbt = N / 16;
  const int need = (nbt + kTallWgBlocks - 1) / kTallWgBlocks;
  return std::min(nbt, std::max(need, device_cus() / splits));
}

// Decode-sized batches (at most kTileDecodeRows rows) run one wave per SIMD whatever the register budget, so
// they take the deeper activation staging (14B at 256 rows: QKV -6%, O -8%, gate/up -3.5%); prefill keeps
// two waves per SIMD with three stages (7B prefill gate/up -3% against two).
constexpr int kTileDecodeRows = 256;
template <bool SWI>
void launch_tile_kernel(hipStream_t s, int splits, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N,
                        int K, uint16_t* h) {
  const int kslice = kslice_for(K, splits);
  const dim3 block(64 * kTileWaves);
  if (tall_batch(M)) {
    const dim3 grid(tall_groups(N, splits), splits);
    hipLaunchKernelGGL((k_gemm_wlds<SWI, 3, 3>), grid, block, 0, s, x, w, out, M, N, K, kslice, h);
  } else if (M <= kTileDecodeRows) {
    const dim3 grid(tile_groups(M, N), splits);
    hipLaunchKernelGGL((k_gemm_tile<kTileNB, kTileMB, SWI, 6, 1>), grid, block, 0, s, x, w, out, M, N, K, kslice, h);
  } else {
    const dim3 grid(tile_groups(M, N), splits);
    hipLaunchKernelGGL((k_gemm_tile<kTileNB, kTileMB, SWI, 3, 2>), grid, block, 0, s, x, w, out, M, N, K, kslice, h);
  }
}

hipError_t launch_tile(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                       int splits) {
  launch_tile_kernel<false>(s, splits, x, w, out, M, N, K, nullptr);
  return hipGetLastError();
}

// Ring kernel shape of the split projections (QKV, O, down at M <= 64).  Workgroups of 4 or 8 weight
// blocks, K split just far enough that the grid fills 80% of the CUs with at most one workgroup per CU: a
// CU's streaming rate bounds these kernels, so a second workgroup on some CUs sets the time, while every
// further split adds a partial for the consumer to sum.  Four-block workgroups are taken when their grid fills at least 80% of the CUs with K
// slices of at most 4096 (their activation reads per weight byte are twice those of eight blocks, which
// costs more than it saves on long K slices); their waves split the K slice four ways while each keeps at
// least 6 k-steps, else two.  Eight-block workgroups run two waves (one when the grid already holds two
// workgroups per CU).  A sweep over blocks per wave (2, 4, 8), waves per workgroup (1, 2, 4) and 1-16
// splits at M = 64 (GEMM time plus reading the partials) puts the optimum at this rule for the 7B and
// 72B QKV, O and down shapes (7B O 10.3 -> 9.3 us with 4 instead of 7 partials, QKV 11.4 -> 10.5 us with
// 3 instead of 7, 72B O 28.1 -> 26.1 us with 2 instead of 4; the two down projections keep 8 blocks), and
// the whole 7B rollout confirms it against the neighbouring shapes of each projection.
// Gate/up with SwiGLU (one split) and the LM head take the balanced grids below.
constexpr int kRingMaxRows = 64;
constexpr int kRingTargetWaves = 512;
int ring_groups(int N, int nbw) { return (N / 16 + nbw - 1) / nbw; }
bool ring_four_blocks(int N, int K, int splits) {
  const int g = ring_groups(N, 4) * splits, cus = device_cus();
  return g <= cus && 5 * g >= 4 * cus && kslice_for(K, splits) <= 4096;
}
int ring_splits(int N, int K, int max_splits) {
  const int cus = device_cus();
  const int smax = std::max(1, std::min(max_splits, K / 256));
  // the fewest splits that bring a grid of g workgroups to 80% of the CUs, never past one per CU
  auto pick = [&](int g) {
    int s = (4 * cus + 5 * g - 1) / (5 * g);
    if (s * g > cus) s = cus / g;
    s = std::max(1, std::min(smax, s));
    const int ks = kslice_for(K, s);
    return (K + ks - 1) / ks;
  };
  const int s4 = pick(ring_groups(N, 4));
  if (ring_four_blocks(N, K, s4)) return s4;
  return pick(ring_groups(N, 8));
}
// waves per workgroup of a split projection's ring kernel with nbw blocks
int ring_split_waves(int N, int K, int nbw, int splits) {
  if (nbw == 4) return kslice_for(K, splits) / 32 / 4 >= 6 ? 4 : 2;
  return ring_groups(N, nbw) * splits < 2 * device_cus() ? 2 : 1;
}
int ring_waves_per_group(int N, int nbw, int splits) {
  return ring_groups(N, nbw) * splits < kRingTargetWaves ? 2 : 1;
}

template <int NBW, bool SWI, int KW>
void launch_ring_kw(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                    int splits, uint16_t* h) {
  const int kslice = kslice_for(K, splits);
  const dim3 grid(ring_groups(N, NBW), splits), block(64 * KW);
  switch ((M + 15) / 16) {
    case 1: hipLaunchKernelGGL((k_gemm_ring<1, NBW, 2, SWI, KW>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    case 2: hipLaunchKernelGGL((k_gemm_ring<2, NBW, 2, SWI, KW>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    case 3: hipLaunchKernelGGL((k_gemm_ring<3, NBW, 2, SWI, KW>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    default: hipLaunchKernelGGL((k_gemm_ring<4, NBW, 2, SWI, KW>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
  }
}

// Gate/up with SwiGLU at decode batches, balanced: one workgroup of two waves per CU (the two waves split
// K and add their sums through LDS), the weight blocks shared out evenly, floor(nbt / CUs) or one more per
// workgroup.  The one-wave-per-four-blocks grid (7B: 592 waves) leaves 80 CUs with three waves and 176
// with two, and a CU's streaming rate, not HBM, bounds these kernels: the CUs with three waves set the
// time (7B gate/up 52.8 -> 50.0 us in isolation).  Taken when every CU gets between 4 and kBalNBW blocks.
// The same balance for single-split projections of many blocks (the LM head): four one-wave workgroups per
// CU, each with floor(nbt / grid) or one more of the blocks (7B: 9 or 10 instead of 1188 eight-block
// workgroups, 4.6 per CU; LM head 199.7 -> 180.4 us in isolation).
// Gate/up with more than kBalNBW blocks per CU (72B: 3,696 blocks, 14.4 per CU) takes two one-wave
// workgroups per CU with up to kBal2NBW blocks each, every wave streaming its blocks over the whole K:
// the one-wave-per-four-blocks grid put four workgroups on 156 CUs and three on 100 (72B rollout 2,176 ->
// 2,284 tokens/s; two two-wave workgroups per CU 2,264, four one-wave workgroups per CU 2,146).
constexpr int kBalNBW = 10;
constexpr int kBal2NBW = 8;
constexpr int kBalWavesPerCU = 4;
bool use_balanced_swiglu(int M, int N) {
  const int nbt = N / 16, cus = device_cus();
  return M <= kRingMaxRows && nbt >= 4 * cus && nbt <= kBalNBW * cus;
}
bool use_balanced_swiglu_wide(int M, int N) {
  const int nbt = N / 16, cus = device_cus();
  return M <= kRingMaxRows && nbt > kBalNBW * cus && nbt <= 2 * kBal2NBW * cus;
}
bool use_balanced_single(int M, int N, int splits) {
  const int nbt = N / 16, g = kBalWavesPerCU * device_cus();
  return M <= kRingMaxRows && splits == 1 && nbt >= 4 * g && nbt <= kBalNBW * g;
}

template <bool SWI, int KW, int NBW = kBalNBW>
hipError_t launch_ring_balanced(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                                int groups, uint16_t* h) {
  const int kslice = kslice_for(K, 1);
  const dim3 grid(groups, 1), block(64 * KW);
  switch ((M + 15) / 16) {
    case 1: hipLaunchKernelGGL((k_gemm_ring<1, NBW, 2, SWI, KW, true>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    case 2: hipLaunchKernelGGL((k_gemm_ring<2, NBW, 2, SWI, KW, true>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    case 3: hipLaunchKernelGGL((k_gemm_ring<3, NBW, 2, SWI, KW, true>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
    default: hipLaunchKernelGGL((k_gemm_ring<4, NBW, 2, SWI, KW, true>), grid, block, 0, s, x, w, out, M, N, K, kslice, h); break;
  }
  return hipGetLastError();
}

template <int NBW, bool SWI>
hipError_t launch_ring(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                       int splits, uint16_t* h) {
  if (ring_waves_per_group(N, NBW, splits) == 2)
    launch_ring_kw<NBW, SWI, 2>(s, x, w, out, M, N, K, splits, h);
  else
    launch_ring_kw<NBW, SWI, 1>(s, x, w, out, M, N, K, splits, h);
  return hipGetLastError();
}

// A split projection (no SwiGLU) on the ring kernel, shaped by ring_four_blocks / ring_split_waves.  Any
// shape gives the same partials; the split count is the caller's.
hipError_t launch_ring_split(hipStream_t s, const bf16x8_t* x, const bf16x8_t* w, float* out, int M, int N, int K,
                             int splits) {
  if (ring_four_blocks(N, K, splits)) {
    if (ring_split_waves(N, K, 4, splits) == 4)
      launch_ring_kw<4, false, 4>(s, x, w, out, M, N, K, splits, nullptr);
    else
      launch_ring_kw<4, false, 2>(s, x, w, out, M, N, K, splits, nullptr);
  } else if (ring_split_waves(N, K, 8, splits) == 2) {
    launch_ring_kw<8, false, 2>(s, x, w, out, M, N, K, splits, nullptr);
  } else {
    launch_ring_kw<8, false, 1>(s, x, w, out, M, N, K, splits, nullptr);
  }
  return hipGetLastError();
}

// int4 ring: K slices in whole 128-wide groups
int kslice_q4(int K, int splits) {
  const int per = (K + splits - 1) / splits;
  return (per + 127) / 128 * 128;
}

template <int MB, int NBW, bool SWI>
void launch_q4_mb(hipStream_t s, const bf16x8_t* x, const void* w, float* out, int M, int N, int K, int splits,
                  uint16_t* h) {
  const int kslice = kslice_q4(K, splits);
  const dim3 grid((N / 16 + 4 * NBW - 1) / (4 * NBW), splits);
  const char* base = (const char*)w;
  const u32x4_t* wq = (const u32x4_t*)base;
  const floatx4_t* ws = (const floatx4_t*)(base + q4_code_bytes(N, K));
  const uint32_t* wz = (const uint32_t*)(base + q4_code_bytes(N, K) + (size_t)N * (K / 128) * 4);
  hipLaunchKernelGGL((k_gemm_q4<MB, NBW, SWI>), grid, dim3(256), 0, s, x, wq, ws, wz, out, M, N, K, kslice, h);
}

// Weight blocks per wave: 4 for up to two 16-row activation blocks, 2 above (registers: both fit two
// waves per SIMD).
constexpr int q4_blocks(int M) { return M <= 32 ? 4 : 2; }

template <bool SWI>
hipError_t launch_q4(hipStream_t s, const bf16x8_t* x, const void* w, float* out, int M, int N, int K, int splits,
                     uint16_t* h) {
  switch ((M + 15) / 16) {
    case 1: launch_q4_mb<1, q4_blocks(16), SWI>(s, x, w, out, M, N, K, splits, h); break;
    case 2: launch_q4_mb<2, q4_blocks(32), SWI>(s, x, w, out, M, N, K, splits, h); break;
    case 3: launch_q4_mb<3, q4_blocks(48), SWI>(s, x, w, out, M, N, K, splits, h); break;
    default: launch_q4_mb<4, q4_blocks(64), SWI>(s, x, w, out, M, N, K, splits, h); break;
  }
  return hipGetLastError();
}

}  // namespace

int gemm_splits_q4(int M, int N, int K, int max_splits) {
  if (M > kRingMaxRows || max_splits <= 1) return 1;
  const int groups = (N / 16 + 4 * q4_blocks(M) - 1) / (4 * q4_blocks(M));  // workgroups per K split
  // as for the bf16 split projections: the fewest splits that fill 80% of the CUs, at most one workgroup
  // per CU (72B: QKV 3, O and down 4 instead of 7-8 splits at two workgroups per CU; 72B int4 rollout +1%)
  const int cus = device_cus();
  int s = (4 * cus + 5 * groups - 1) / (5 * groups);
  if (s * groups > cus) s = cus / groups;
  s = std::min(s, std::max(1, K / 256));
  s = std::max(1, std::min(s, max_splits));
  const int ks = kslice_q4(K, s);
  return (K + ks - 1) / ks;
}

hipError_t launch_gemm_q4(hipStream_t s, const void* X, const void* W, float* out, int M, int N, int K, int splits) {
  if (M <= 0) return hipSuccess;
  if (M > kRingMaxRows || N % 16 || K % 128 || splits < 1) return hipErrorInvalidValue;
  return launch_q4<false>(s, (const bf16x8_t*)X, W, out, M, N, K, splits, nullptr);
}

hipError_t launch_gemm_swiglu_q4(hipStream_t s, const void* X, const void* W, int M, int N, int K, void* h) {
  if (M <= 0) return hipSuccess;
  if (M > kSwigluMaxRows || M > kRingMaxRows || N % 16 || K % 128) return hipErrorInvalidValue;
  return launch_q4<true>(s, (const bf16x8_t*)X, W, nullptr, M, N, K, 1, (uint16_t*)h);
}

int gemm_splits(int dtype, int M, int N, int K, int max_splits) {
  if (dtype != ROLLOUT_DTYPE_BF16 || max_splits <= 1) return 1;
  if (M <= kRingMaxRows) return ring_splits(N, K, max_splits);
  const int nwg = tile_m_tiles(M) * tile_n_tiles(N);
  int s;
  if (tall_batch(M)) {
    // one activation tile: K splits until the 128-row weight tiles of all splits fill the 256 CUs once
    // (a partial costs M x N x 4 bytes, so no more than that)
    const int tiles = (N / 16 + kTallWgBlocks - 1) / kTallWgBlocks;
    s = std::max(1, std::min(std::min(max_splits, std::max(1, K / 256)), 256 / tiles));
  } else if (M <= 256) {
    // decode-sized batches: workgroup x of a split runs on XCD x % 8, which holds N tiles nt % 8 == j for
    // every M tile.  Split K until the busiest XCD holds one workgroup per CU (32); with long K slices
    // (> 64 k-steps) two per CU.  Fewer splits leave CUs idle, more add partial-sum traffic and a second
    // round of workgroups on the busiest XCD.
    const int per_xcd = tile_m_tiles(M) * ((tile_n_tiles(N) + 7) / 8);
    const int smax = std::max(1, std::min(max_splits, K / 256));
    s = std::max(1, std::min(smax, 32 / per_xcd));
    if (K / 32 / s > 64) s = std::max(s, std::min(smax, 64 / per_xcd));
  } else {
    // MFMA-bound batches: enough K splits for ~1.5 workgroups per CU, K slices of at least 512
    s = (384 + nwg - 1) / nwg;
    s = std::min(s, std::max(1, K / 512));
    s = std::max(1, std::min(s, max_splits));
  }
  const int ks = kslice_for(K, s);
  return (K + ks - 1) / ks;
}

hipError_t launch_gemm(hipStream_t s, int dtype, const void* X, int ldx, const void* W, float* out, int M, int N,
                       int K, int splits) {
  if (M <= 0) return hipSuccess;
  if (dtype != ROLLOUT_DTYPE_BF16) {
    dim3 grid((N + 15) / 16, (M + 15) / 16);
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, s, (const float*)X, ldx, (const float*)W, out, M, N, K);
    return hipGetLastError();
  }
  if (N % 16 || K % 32) return hipErrorInvalidValue;
  const bf16x8_t* x = (const bf16x8_t*)X;
  const bf16x8_t* w = (const bf16x8_t*)W;
  if (M <= kRingMaxRows) {
    if (use_balanced_single(M, N, splits))
      return launch_ring_balanced<false, 1>(s, x, w, out, M, N, K, kBalWavesPerCU * device_cus(), nullptr);
    return launch_ring_split(s, x, w, out, M, N, K, splits);
  }
  return launch_tile(s, x, w, out, M, N, K, splits);
}

hipError_t launch_gemm_swiglu(hipStream_t s, const void* X, const void* W, int M, int N, int K, void* h) {
  if (M <= 0) return hipSuccess;
  if (N % 32 || K % 32) return hipErrorInvalidValue;
  if (M > kRingMaxRows) {  // larger batches: the tile kernel with the same epilogue, one K split
    launch_tile_kernel<true>(s, 1, (const bf16x8_t*)X, (const bf16x8_t*)W, nullptr, M, N, K, (uint16_t*)h);
    return hipGetLastError();
  }
  if (use_balanced_swiglu(M, N))
    return launch_ring_balanced<true, 2>(s, (const bf16x8_t*)X, (const bf16x8_t*)W, nullptr, M, N, K, device_cus(),
                                         (uint16_t*)h);
  if (use_balanced_swiglu_wide(M, N))
    return launch_ring_balanced<true, 1, kBal2NBW>(s, (const bf16x8_t*)X, (const bf16x8_t*)W, nullptr, M, N, K,
                                                   2 * device_cus(), (uint16_t*)h);
  return launch_ring<4, true>(s, (const bf16x8_t*)X, (const bf16x8_t*)W, nullptr, M, N, K, 1, (uint16_t*)h);
}

}  // namespace rollout
