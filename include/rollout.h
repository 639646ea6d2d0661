/*
 * rollout.h -- C ABI of the MI355X GRPO rollout library (librollout.so).
 *
 * The library runs the rollout phase of a GRPO training step (paper section 3,
 * "Background"): for each of B prompts it generates a group of G sampled
 * completions with a dense decoder-only transformer, and it computes each
 * completion's advantage relative to its own group.  Generation concurrency
 * (sequences in flight), group size, completion length, temperature and top-p
 * are per-call arguments, never cached at initialisation: they are the knobs a
 * power controller moves between calls (sections 4.1, 4.3 and 6.4, Table 4).
 *
 * Conventions for every entry point:
 *  - C linkage, no exceptions cross the boundary, plain pointers and sizes.
 *  - "d_" pointers are device (HBM) pointers owned by the caller; "h_"/plain
 *    struct pointers are host pointers owned by the caller.  The library never
 *    frees caller memory.  rollout_ctx is opaque host state owned by the
 *    library between rollout_init and rollout_destroy.
 *  - Device work is enqueued on the stream given to rollout_init (or passed
 *    directly) and the call returns; outputs are valid after that stream is
 *    synchronised or after rollout_sync.
 *  - Arguments are validated before anything is enqueued; on error nothing is
 *    enqueued and a message is available from rollout_last_error.
 *  - Sequence order is group-major: completion g of prompt p is sequence
 *    s = p * G + g, so every group is contiguous (section 4.3 keeps the
 *    generation batch a multiple of G).
 *  - Token ids are int32; logits, uniforms, rewards and advantages are fp32.
 */
#ifndef ROLLOUT_H
#define ROLLOUT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rollout_status;
#define ROLLOUT_OK 0
#define ROLLOUT_EINVAL (-1)      /* bad argument; nothing enqueued */
#define ROLLOUT_ENOMEM (-2)      /* arena or HBM budget too small for the request */
#define ROLLOUT_EDEVICE (-3)     /* HIP runtime error (message in rollout_last_error) */
#define ROLLOUT_ESTATE (-4)      /* call order violated (decode before prefill, context full) */
#define ROLLOUT_EUNSUPPORTED (-5) /* shape the kernels do not implement */

#define ROLLOUT_DTYPE_FP32 0     /* fp32 weights, cache and activations */
#define ROLLOUT_DTYPE_BF16 1     /* bf16 weights/cache/GEMM operands, fp32 residual and logits */
#define ROLLOUT_DTYPE_INT4 2     /* as BF16, but the layer projections (q, k, v, o, gate, up, down) are
                                    weight-only int4: groups of 128 inputs of one output row, each with an
                                    fp32 scale s = (hi - lo) / 15 and a zero point z = rint(-lo / s) in
                                    [0, 15], codes q = clamp(rint(w / s) + z, 0, 15) (the AWQ storage format
                                    of the 72B generation proxy, sections 5 and 6.6, which fix no format).
                                    The model multiplies with the group-quantised weight's plain value
                                    (q - z) * s, never rounded to bf16: each group's scale multiplies its
                                    integer dot product in fp32.  Embedding and LM head stay bf16.  Needs
                                    d_model, n_heads*head_dim and d_ff to be multiples of 128. */

typedef struct rollout_ctx rollout_ctx;

/*
 * Model and capacity description; immutable after rollout_init.
 * The model is a dense decoder (section 5 runs the Qwen2.5 family): RMSNorm,
 * grouped-query attention with rotate-half RoPE, SwiGLU MLP, untied LM head,
 * no biases.  Weights are synthesised on the device from weight_seed with the
 * SplitMix64-based counter hash (Irwin-Hall(4) values of standard deviation
 * weight_std; norm gains 1).
 * Supported shapes: head_dim in {32, 64, 128}; n_heads a multiple of
 * n_kv_heads with n_heads / n_kv_heads <= 16; d_model, n_heads*head_dim and
 * d_ff multiples of 32; vocab a multiple of 16; kv_block_size in {8, 16, 32}.
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rms_eps, rope_theta;
  int32_t dtype;               /* ROLLOUT_DTYPE_* */
  uint64_t weight_seed;
  double weight_std;           /* standard deviation of the synthesised weights */
  int32_t kv_block_size;       /* tokens per paged-KV block */
  int32_t max_prompt_len;      /* longest prompt any call may pass */
  int32_t max_new_tokens;      /* longest completion any call may request */
  int32_t max_seqs_in_flight;  /* requested concurrency ceiling; the plan may lower it */
  uint64_t hbm_budget_bytes;   /* 0 = free device memory reported by the runtime */
} rollout_model_config;

/* Result of planning: how many sequences fit and how big the arena must be. */
typedef struct {
  int32_t seqs_in_flight_max;  /* multiple of group_size; 0 never returned with OK */
  int32_t kv_blocks;           /* paged-KV blocks in the pool */
  uint64_t arena_bytes;        /* device bytes the caller must provide to rollout_init */
  uint64_t weight_bytes;       /* of which model weights */
  uint64_t kv_block_bytes;     /* bytes of one block across all layers, K and V */
  uint64_t kv_bytes;           /* bytes of the whole pool */
  uint64_t work_bytes;         /* activations, logits and split-K workspace */
} rollout_plan_t;

/*
 * Size the arena (section 4.3: the generation batch must be a multiple of G).
 * Host-only unless cfg->hbm_budget_bytes == 0, in which case the free memory
 * of the current HIP device is queried.  seqs_in_flight_max is the largest
 * multiple of group_size, at most cfg->max_seqs_in_flight, whose weights,
 * KV blocks (prompt blocks shared inside a group), activations, logits and
 * workspace fit in the budget.
 * Errors: EINVAL (bad config or group_size < 1), EUNSUPPORTED (shape),
 * ENOMEM (not even one group fits), EDEVICE (memory query failed).
 */
rollout_status rollout_plan(const rollout_model_config* cfg, int32_t group_size, rollout_plan_t* out);

/*
 * Set up the rollout engine of section 3's rollout phase: the model of section 5 (a dense decoder of the
 * Qwen2.5 family, here with synthetic weights) resident in HBM, ready to generate groups of completions.
 * Bind a context to a caller-owned device arena of arena_bytes (>= the plan's
 * arena_bytes for group size 1 at cfg->max_seqs_in_flight, or the value
 * returned by rollout_plan for the group size that will be used), enqueue
 * weight synthesis on hip_stream (a hipStream_t; NULL = default stream) and
 * return the context in *out.  The arena must stay allocated until
 * rollout_destroy.  Errors: EINVAL, EUNSUPPORTED, ENOMEM (arena too small),
 * EDEVICE.
 */
rollout_status rollout_init(const rollout_model_config* cfg, void* d_arena, uint64_t arena_bytes,
                            void* hip_stream, rollout_ctx** out);

/*
 * Section 3's rollout phase, first forward: a batch of B prompts, each the prompt of a group of G
 * candidate completions.
 * Start a wave: n_prompts prompts of prompt_len tokens (d_prompts, int32,
 * row-major [n_prompts, prompt_len]), each expanded to group_size sequences.
 * Each prompt is run through the model once; its KV blocks are shared by the
 * group's sequences (a partially filled last block is copied per sequence).
 * Writes the last-position logits of every sequence, fp32 row-major
 * [n_prompts * group_size, vocab], to d_logits (rows of a group are equal).
 * Any previous wave is discarded.  Errors: EINVAL (sizes, prompt_len >
 * max_prompt_len), ENOMEM (more sequences than the plan admits), EDEVICE.
 * Token ids outside [0, vocab) set the device error flag (see rollout_sync).
 */
rollout_status rollout_prefill(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts,
                               int32_t prompt_len, int32_t group_size, float* d_logits);

/*
 * One autoregressive step of section 3's rollout phase (every candidate of every group extends by one
 * token; completion length is the knob of Table 4's third row, section 6.4).
 * One decode step of the current wave: append token d_tokens[s] (int32
 * [n_seqs]) to every sequence s at its next position and write the logits of
 * that position, fp32 [n_seqs, vocab], to d_logits.  n_seqs is the wave's
 * sequence count.  Errors: ESTATE (no wave, or the context would exceed
 * max_prompt_len + max_new_tokens), EDEVICE.
 */
rollout_status rollout_decode_step(rollout_ctx* ctx, const int32_t* d_tokens, float* d_logits);

/*
 * The draw that makes a group's G candidates differ (section 3: G sampled answers to the same prompt).
 * The paper names no sampler settings; temperature and top-p are per-call knobs with the definition below.
 * Draw one token per row of d_logits (fp32 [n_seqs, vocab]) with one uniform
 * per row (d_uniforms, fp32 [n_seqs], values in [0, 1)) into d_tokens_out
 * (int32 [n_seqs]).  temperature 0 is greedy (lowest id among equal maxima).
 * Otherwise e_i = exp(z_i / T - max) in fp32; with top_p < 1 the kept set is
 * the shortest prefix, in (e descending, id ascending) order, whose mass
 * reaches top_p of the total; the token is the first kept id, in ascending
 * id order, whose running mass exceeds u times the kept mass.
 * Errors: EINVAL (n_seqs < 1, temperature < 0, top_p outside (0, 1]), EDEVICE.
 */
rollout_status rollout_sample(rollout_ctx* ctx, const float* d_logits, int32_t n_seqs, float temperature,
                              float top_p, const float* d_uniforms, int32_t* d_tokens_out);

/*
 * Group-relative advantages (section 3: each candidate's reward against its
 * own group; GRPO's normalisation by the group's standard deviation).
 * d_rewards fp32 [n_groups * group_size] in group-major order; d_adv receives
 * A = (r - mean) / (std + eps) with std using divisor group_size - std_ddof;
 * groups whose rewards are all equal (or group_size == 1) get A = 0 and are
 * counted into *d_zero_var_groups (int32, device; overwritten; may be NULL),
 * the zero-variance-group statistic of section 4.2.  Enqueued on hip_stream.
 * Errors: EINVAL (n_groups < 1, group_size < 1, std_ddof not 0 or 1, eps < 0,
 * NULL rewards or advantages), EDEVICE.
 */
rollout_status grpo_advantages(const float* d_rewards, int32_t n_groups, int32_t group_size, float eps,
                               int32_t std_ddof, float* d_adv, int32_t* d_zero_var_groups, void* hip_stream);

/*
 * The whole rollout for n_prompts prompts (d_prompts int32 [n_prompts,
 * prompt_len]): waves of whole groups, at most seqs_in_flight sequences each
 * (snapped down to a multiple of group_size, section 4.3), each wave prefilled
 * once then decoded max_new_tokens - 1 times, drawing token t of sequence s
 * with d_uniforms[s * max_new_tokens + t] (fp32 [n_prompts * group_size,
 * max_new_tokens]) into d_tokens_out[s * max_new_tokens + t] (int32, same
 * shape).  Exactly max_new_tokens tokens per completion (no end-of-sequence).
 * Errors: EINVAL, ENOMEM (one group does not fit), EDEVICE.
 */
rollout_status rollout_generate(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts,
                                int32_t prompt_len, int32_t group_size, int32_t seqs_in_flight,
                                int32_t max_new_tokens, float temperature, float top_p,
                                const float* d_uniforms, int32_t* d_tokens_out);

/*
 * Completions that end at a stop token, served by continuous batching.  The
 * paper's controller counts T_k, the non-padding tokens a batch produced
 * (section 4.5, eq. 4), and its runs reward closeness to a length target
 * (section 5): both presuppose completions that end when the model draws a
 * stop token.
 *
 * Draws are those of rollout_generate (token t of completion s = p * G + g
 * with d_uniforms[s * max_new_tokens + t]); completion s ends after drawing a
 * token of the stop set (d_stop_ids, n_stop device int32 ids in [0, vocab);
 * n_stop = 0: no stop set) or after max_new_tokens tokens.  Outputs (device,
 * caller-owned): d_tokens_out int32 [n_prompts * G, max_new_tokens], -1 after
 * the end; d_lengths_out int32 [n_prompts * G], tokens including the stop
 * token; d_admit_step_out int32 [n_prompts * G] or NULL, the decode step at
 * which each completion was admitted; *h_decode_steps_out (host, or NULL) the
 * decode steps run.
 *
 * Scheduling: every refill_interval decode steps the host reads the slots'
 * ended flags and refills, in slot order, in completion order.
 *  - whole_groups = 1: min(seqs_in_flight snapped to whole groups (section
 *    4.3), n_prompts * G) slots in ranges of G; a range whose G completions
 *    have all ended takes the next prompt's group (prefilled there, token 0
 *    drawn from its logits).
 *  - whole_groups = 0: min(seqs_in_flight, context rows - 1, n_prompts * G)
 *    slots; a slot whose completion has ended takes the next completion.  A
 *    group's prompt is prefilled once, when its first completion is admitted,
 *    into a prompt record of KV blocks shared by its members (at most slots + 1
 *    records are alive); every member's token 0 is drawn then, so group_size
 *    must not exceed the context's sequence rows (else ENOMEM).  Needs
 *    (slots + 1) * ceil(prompt / block) + slots * (blocks from the last full
 *    prompt block to the end) KV blocks; fewer slots are used if the pool is
 *    smaller.
 * The call returns when every completion has been admitted and has ended.
 * Ended completions keep running in their slot until it is refilled (their
 * rows are the padding that T_k excludes).  Errors: EINVAL (bad argument, or
 * a stop id outside [0, vocab), reported by rollout_sync), ENOMEM, EDEVICE.
 */
rollout_status rollout_generate_eos(rollout_ctx* ctx, const int32_t* d_prompts, int32_t n_prompts,
                                    int32_t prompt_len, int32_t group_size, int32_t seqs_in_flight,
                                    int32_t max_new_tokens, float temperature, float top_p,
                                    const float* d_uniforms, const int32_t* d_stop_ids, int32_t n_stop,
                                    int32_t refill_interval, int32_t whole_groups, int32_t* d_tokens_out,
                                    int32_t* d_lengths_out, int32_t* d_admit_step_out,
                                    int32_t* h_decode_steps_out);

/*
 * Length-target reward of section 5 (its formula is not given; reading:
 * r = 1 - min(1, |L - target| / target), 1 at the target, 0 at distance
 * >= target) for n completion lengths d_lengths (device int32), into
 * d_rewards (device fp32 [n]); *d_total_tokens (device int64, or NULL)
 * receives the sum of the lengths, the batch's non-padding token count T_k
 * (section 4.5).  Enqueued on hip_stream.  Errors: EINVAL, EDEVICE.
 */
rollout_status rollout_length_rewards(const int32_t* d_lengths, int32_t n, int32_t target, float* d_rewards,
                                      int64_t* d_total_tokens, void* hip_stream);

/* Wait for the context's stream and report the device error flag (EINVAL if a
 * token id outside [0, vocab) was seen since the last call; the flag is then
 * cleared).  Errors: EINVAL, EDEVICE. */
rollout_status rollout_sync(rollout_ctx* ctx);

/* Release the context's host state (never the caller's arena). NULL is a no-op. */
void rollout_destroy(rollout_ctx* ctx);

/* Last error message of ctx, or of the calling thread's last context-free
 * call when ctx is NULL.  Never NULL; valid until the next call. */
const char* rollout_last_error(const rollout_ctx* ctx);

/* ------------------------------------------------------------------------ */
/* Allocation-free draw                                                      */
/* ------------------------------------------------------------------------ */

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the draw of
 * rollout_sample without a context.  Same definition and arguments as
 * rollout_sample, plus the row width vocab and hip_stream (a hipStream_t of
 * the current device; NULL = its default stream); enqueued on that stream.
 * Nothing is allocated: the sampler kernels' scratch is one fixed device array
 * of ROLLOUT_SAMPLE_NOALLOC_SCRATCH_BYTES, held on every GPU the call runs on
 * until the process ends, and rows are drawn in batches that fit it.  Every
 * call on a GPU shares that GPU's array, so calls that overlap on one GPU
 * (several streams or threads) race on it and must be serialised by the
 * caller.  Errors (message from rollout_last_error(NULL)): EINVAL (NULL
 * buffer, n_seqs < 1, vocab < 2, temperature < 0, top_p outside (0, 1], a
 * stream of another device), ENOMEM (one row needs more scratch than the
 * array holds: vocab above 16,724,608), EDEVICE.
 */
#define ROLLOUT_SAMPLE_NOALLOC_SCRATCH_BYTES (64ull << 20)
rollout_status rollout_sample_noalloc(const float* d_logits, int32_t n_seqs, int32_t vocab, float temperature,
                                      float top_p, const float* d_uniforms, int32_t* d_tokens_out,
                                      void* hip_stream);

/* ------------------------------------------------------------------------ */
/* Inspection and measurement                                                */
/* ------------------------------------------------------------------------ */

/* Weight tensor ids of the synthesis hash: embedding 0; layer l:
 * 1 + 9 l + {1 Wq, 2 Wk, 3 Wv, 4 Wo, 6 Wgate, 7 Wup, 8 Wdown}; LM head
 * 2 + 9 n_layers.  Copies the logical [out, in] matrix, as fp32 (bf16 values
 * widened exactly), into d_out (caller-owned, rows*cols floats), whatever the
 * physical layout the kernels keep it in.  Errors: EINVAL (not a matrix id). */
rollout_status rollout_export_weight(rollout_ctx* ctx, int32_t tensor_id, float* d_out);

/* Per-kernel-class timing of one instrumented decode step of the current
 * wave, with HIP events around every launch on the context's stream.  The
 * step is run for real (it appends d_tokens like rollout_decode_step).
 * Classes: 0 projection GEMMs (QKV, O, gate/up, down, LM head), 1 decode
 * attention (+ its combine), 2 everything else.  ms[c] = summed duration,
 * launches[c] = launch count, bytes[c] = algorithmic HBM bytes (weights read
 * once, cache read once per sequence, activations), flops[c] = useful flops. */
typedef struct {
  double ms[3];
  int32_t launches[3];
  double bytes[3];
  double flops[3];
} rollout_step_profile;
rollout_status rollout_profile_decode_step(rollout_ctx* ctx, const int32_t* d_tokens, float* d_logits,
                                           rollout_step_profile* out);

/* Average duration of the projection GEMMs of one decode step of the current
 * wave, in the launch mode the rollout uses: the step's projection launches
 * (per layer QKV, O, gate/up with SwiGLU, down; then the LM head, into
 * d_logits, fp32 [n_seqs, vocab]) are captured as one HIP graph and replayed
 * reps times between two HIP events on the context's stream.  Only the
 * split-K workspace, the SwiGLU output and d_logits are written (the wave's
 * KV cache, residual stream and positions are untouched).  out: launches per
 * step, average microseconds per launch, algorithmic bytes (weights once,
 * activations and outputs once) and flops per launch on average.
 * Errors: EINVAL (reps < 1, NULL; int4 weights with more than 64 rows in the
 * wave, whose projections dequantise first), ESTATE (no wave), EDEVICE. */
typedef struct {
  int32_t launches;
  double avg_us;
  double bytes_per_launch;
  double flops_per_launch;
} rollout_projection_profile;
rollout_status rollout_profile_projections(rollout_ctx* ctx, int32_t reps, float* d_logits,
                                           rollout_projection_profile* out);

#ifdef __cplusplus
}
#endif
#endif /* ROLLOUT_H */
