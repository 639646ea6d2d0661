// Stop-token termination and continuous batching (device side): slots refilled
// with whole groups, or with single completions.
//
// The paper's controller counts T_k, the non-padding tokens a generation batch
// yields (section 4.5, eq. 4), and its runs reward closeness to a 128-token
// completion length (section 5); both need completions that end when a stop
// token is drawn.  Per slot r the
// device keeps the completion it serves (seq[r], -1 for none), the next token
// column (col[r]) and an ended flag (done[r]).  The decode step draws into a
// slot-indexed buffer (draw[r], with the slot's staged uniform u_slot[r]);
// k_cb_commit then files each live slot's draw under its completion, ends it
// on a stop token or at max_new_tokens, and stages the next uniform.  Ended
// slots keep running with their last token until the host refills their
// group's range (or, in single-completion refill, their slot); their context
// length stops advancing, so their cache writes stay inside the blocks their
// slot owns.
#include "internal.h"

namespace rollout {
namespace {

// bitmap[v / 32] bit v % 32 set for every stop token v; ids outside [0, V) flag the error word
__global__ void k_stop_bitmap(uint32_t* __restrict__ bitmap, int words, const int32_t* __restrict__ ids, int n,
                              int V, int32_t* __restrict__ err) {
  // one workgroup: clear, then set (the barrier orders the two phases)
  for (int i = threadIdx.x; i < words; i += blockDim.x) bitmap[i] = 0u;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int v = ids[i];
    if (v < 0 || v >= V) {
      atomicOr(err, 1);
      continue;
    }
    atomicOr(&bitmap[v >> 5], 1u << (v & 31));
  }
}

// rows [0, S): no completion, ended, token 0 and uniform 0 (a valid input for the step kernels)
__global__ void k_cb_reset(int S, int32_t* __restrict__ seq, int32_t* __restrict__ col, int32_t* __restrict__ done,
                           int32_t* __restrict__ draw, float* __restrict__ u_slot) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= S) return;
  seq[r] = -1;
  col[r] = 0;
  done[r] = 1;
  draw[r] = 0;
  u_slot[r] = 0.f;
}

// slots r0 .. r0 + G - 1 start completions seq0 .. seq0 + G - 1 at context P; their output rows are padded
__global__ void k_cb_admit(int r0, int G, int seq0, int P, int N, int32_t* __restrict__ seq,
                           int32_t* __restrict__ col, int32_t* __restrict__ done, int32_t* __restrict__ ctx_len,
                           int32_t* __restrict__ tokens_out) {
  for (size_t i = threadIdx.x; i < (size_t)G * N; i += blockDim.x) tokens_out[(size_t)seq0 * N + i] = -1;
  for (int g = threadIdx.x; g < G; g += blockDim.x) {
    const int r = r0 + g;
    seq[r] = seq0 + g;
    col[r] = 0;
    done[r] = 0;
    ctx_len[r] = P;
  }
}

// file the draws of live slots in [r0, r1); advance = the slots' fed token was appended this step
__global__ void k_cb_commit(int r0, int r1, int N, const int32_t* __restrict__ draw,
                            const uint32_t* __restrict__ stop, const float* __restrict__ u,
                            int32_t* __restrict__ seq, int32_t* __restrict__ col, int32_t* __restrict__ done,
                            int32_t* __restrict__ ctx_len, float* __restrict__ u_slot,
                            int32_t* __restrict__ tokens_out, int32_t* __restrict__ lengths, int advance) {
  const int r = r0 + blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= r1) return;
  const int s = seq[r];
  if (s < 0 || done[r]) return;
  const int t = col[r];
  const int tok = draw[r];
  tokens_out[(size_t)s * N + t] = tok;
  if (advance) ctx_len[r] += 1;
  const bool is_stop = stop && ((stop[tok >> 5] >> (tok & 31)) & 1u);
  if (is_stop || t + 1 >= N) {
    done[r] = 1;
    lengths[s] = t + 1;
  } else {
    col[r] = t + 1;
    u_slot[r] = u[(size_t)s * N + t + 1];
  }
}

// single-completion refill: block-table row `row` = the prompt record's shared blocks (rec .. rec + n_shared),
// then either the record's copy of the partial last prompt block (prefill row, own == -1) or the slot's own
// blocks (own .. own + n_own); the rest -1
__global__ void k_seq_table(int32_t* __restrict__ tables, int max_blocks, int row, int rec, int n_shared,
                            int has_partial, int own, int n_own) {
  int32_t* t = tables + (size_t)row * max_blocks;
  for (int j = threadIdx.x; j < max_blocks; j += blockDim.x) {
    int v = -1;
    if (j < n_shared) v = rec + j;
    else if (own < 0) v = (has_partial && j == n_shared) ? rec + n_shared : -1;
    else if (j - n_shared < n_own) v = own + (j - n_shared);
    t[j] = v;
  }
}

// slot r starts completion s at context P with the token 0 its group's prefill drew (tokens_out[s][0]);
// the rest of the completion's output row is padded
__global__ void k_seq_admit(int r, int s, int P, int N, int32_t* __restrict__ seq, int32_t* __restrict__ col,
                            int32_t* __restrict__ done, int32_t* __restrict__ draw, int32_t* __restrict__ ctx_len,
                            int32_t* __restrict__ tokens_out) {
  for (int i = 1 + threadIdx.x; i < N; i += blockDim.x) tokens_out[(size_t)s * N + i] = -1;
  if (threadIdx.x == 0) {
    seq[r] = s;
    col[r] = 0;
    done[r] = 0;
    ctx_len[r] = P;
    draw[r] = tokens_out[(size_t)s * N];
  }
}

// rewards[i] = 1 - min(1, |L_i - target| / target); total[0] = sum of L_i (one workgroup)
__global__ __launch_bounds__(256) void k_length_rewards(const int32_t* __restrict__ lengths, int n, int target,
                                                        float* __restrict__ rewards,
                                                        long long* __restrict__ total) {
  __shared__ long long red[256];
  long long acc = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int L = lengths[i];
    acc += L;
    const double d = fabs((double)L - (double)target) / (double)target;
    rewards[i] = (float)(1.0 - (d < 1.0 ? d : 1.0));
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0 && total) total[0] = red[0];
}

}  // namespace

hipError_t launch_stop_bitmap(hipStream_t s, uint32_t* bitmap, int V, const int32_t* ids, int n, int32_t* err) {
  hipLaunchKernelGGL(k_stop_bitmap, dim3(1), dim3(1024), 0, s, bitmap, (V + 31) / 32, ids, n, V, err);
  return hipGetLastError();
}

hipError_t launch_cb_reset(hipStream_t s, int S, const CbState& cb) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_cb_reset, dim3((S + 255) / 256), dim3(256), 0, s, S, cb.seq, cb.col, cb.done, cb.draw,
                     cb.u_slot);
  return hipGetLastError();
}

hipError_t launch_cb_admit(hipStream_t s, const CbState& cb, int r0, int G, int seq0, int P, int N,
                           int32_t* ctx_len, int32_t* tokens_out) {
  hipLaunchKernelGGL(k_cb_admit, dim3(1), dim3(256), 0, s, r0, G, seq0, P, N, cb.seq, cb.col, cb.done, ctx_len,
                     tokens_out);
  return hipGetLastError();
}

hipError_t launch_cb_commit(hipStream_t s, const CbState& cb, int r0, int r1, int N, const uint32_t* stop,
                            const float* u, int32_t* ctx_len, int32_t* tokens_out, int32_t* lengths, bool advance) {
  if (r1 <= r0) return hipSuccess;
  hipLaunchKernelGGL(k_cb_commit, dim3((r1 - r0 + 255) / 256), dim3(256), 0, s, r0, r1, N, cb.draw, stop, u, cb.seq,
                     cb.col, cb.done, ctx_len, cb.u_slot, tokens_out, lengths, advance ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_seq_table(hipStream_t s, int32_t* tables, int max_blocks, int row, int rec, int n_shared,
                            bool has_partial, int own, int n_own) {
  hipLaunchKernelGGL(k_seq_table, dim3(1), dim3(256), 0, s, tables, max_blocks, row, rec, n_shared, has_partial ? 1 : 0,
                     own, n_own);
  return hipGetLastError();
}

hipError_t launch_seq_admit(hipStream_t s, const CbState& cb, int r, int seq_id, int P, int N, int32_t* ctx_len,
                            int32_t* tokens_out) {
  hipLaunchKernelGGL(k_seq_admit, dim3(1), dim3(256), 0, s, r, seq_id, P, N, cb.seq, cb.col, cb.done, cb.draw, ctx_len,
                     tokens_out);
  return hipGetLastError();
}

hipError_t launch_length_rewards(hipStream_t s, const int32_t* lengths, int n, int target, float* rewards,
                                 long long* total) {
  hipLaunchKernelGGL(k_length_rewards, dim3(1), dim3(256), 0, s, lengths, n, target, rewards, total);
  return hipGetLastError();
}

}  // namespace rollout
