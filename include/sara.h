/*
 * sara.h - C ABI of libsara: the rollout-generation hot path of SARA
 * (Sequential Adaptive Rollout Allocation) on one MI355X (gfx950).
 *
 * One allocation step (Algorithm 1, section 3.3) is driven by the host as
 *
 *     sara_begin_step(...)                      prompt pool in, prefill, first draws
 *     repeat: sara_decode_step -> sara_posterior_decide -> sara_refill
 *             (or sara_run, which replays that triple from a HIP graph)
 *     until the step is done (sara_query / sara_run report it)
 *     sara_finish_step(...)                     GRPO advantages of committed groups
 *
 * All calls enqueue work on the context's stream and return at once unless
 * stated otherwise.  Pointers prefixed d_ are device (HIP) memory, h_ host
 * memory.  Sizes are element counts.  The context is not thread safe: use one
 * context per host thread and stream.
 *
 * Errors: every int-returning call returns SARA_OK or a negative code and
 * sets a thread-local message readable with sara_last_error().  Argument
 * errors are detected synchronously (SARA_EINVAL) and enqueue nothing.
 * Budget or prompt-pool exhaustion is not an error: the step ends with fewer
 * than B committed groups.
 */
#ifndef SARA_H
#define SARA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sara_ctx sara_ctx;

enum {
  SARA_OK = 0,
  SARA_EINVAL = -1,   /* invalid argument or unsupported configuration         */
  SARA_ENOMEM = -2,   /* device allocation failed                              */
  SARA_EHIP = -3,     /* a HIP runtime call failed                             */
  SARA_ESTATE = -4,   /* call out of order (e.g. decode before begin_step)     */
  SARA_EDEVICE = -5   /* a device-side check failed (see sara_step_stats.error) */
};
enum { SARA_F32 = 0, SARA_BF16 = 1 };
/* SARA_MODE_SARA_THOMPSON: SARA with the posterior-sampling priority of the
 * index-policy proposition (Thompson sampling as the alternative index to
 * p_eff): when a prompt's rollouts are queued (at its draw, or at a CONTINUE
 * decision after n outcomes with s successes) it draws g ~ Beta(a, b), its
 * current posterior (a = alpha0 + s, b = beta0 + n - s), as the a-th
 * smallest of a + b - 1 uniforms (w + 1/2) 2^-32, w the words of
 * Philox4x32-10 under the sampler's key at counters (uid, n, c, 2), and its
 * pending rollouts are ordered by P(group of k ends mixed | g) (Eq. peff at
 * the draw: 1 - g^k - (1-g)^k, 1 - (1-g)^r after s = 0, 1 - g^r after
 * s = n, r = k - n; powers by repeated fp64 multiplication) instead of
 * p_eff.  Decisions are unchanged.  A prompt whose posterior parameters are
 * not integers, or with a + b - 1 > 4096, keeps the p_eff index. */
enum { SARA_MODE_SARA = 0, SARA_MODE_FIXED_K = 1, SARA_MODE_SARA_THOMPSON = 2 };
/* decision codes in the decision log */
enum { SARA_COMMIT = 1, SARA_ABANDON = 2, SARA_CONTINUE = 3 };
/* per-prompt status */
enum { SARA_UNDRAWN = 0, SARA_ACTIVE = 1, SARA_COMMITTED = 2, SARA_ABANDONED = 3 };
/* bits of the device error word (sara_step_stats.error) */
enum { SARA_DEVERR_WARM_ID = 1 };   /* a warm-start prompt id outside [0, n_store) */

/* Decoder shape.  Pre-norm GQA decoder: RMSNorm, rotate-half RoPE, SwiGLU,
 * untied LM head, no biases.  head_dim in {64, 128}; n_heads a multiple of
 * n_kv_heads with at most 8 query heads per KV head; d_model, d_ffn and
 * n_heads*head_dim multiples of 64; vocab a multiple of 16.  dtype SARA_BF16 stores weights, KV cache
 * and GEMM inputs in bf16 (fp32 accumulation); SARA_F32 computes in fp32.
 * eos_id = -1 disables the EOS token. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rope_theta, rms_eps;
  int32_t dtype;
  int32_t eos_id;
} sara_model_desc;

/* Allocation problem of one step (Algorithm 1 inputs; implementation-details
 * appendix for commit_min, the prior and the budget cap):
 *   mode        SARA_MODE_SARA, SARA_MODE_FIXED_K or SARA_MODE_SARA_THOMPSON
 *   B           effective groups wanted (ignored in SARA_MODE_FIXED_K)
 *   k           group size;  n0 probe rollouts per fresh prompt (1..k)
 *   commit_min  commit floor (2..k); tau_low abandon threshold in [0, 1]
 *   alpha0/beta0  Beta prior (> 0);  budget_N  rollout budget of the step
 *   pool_U      prompts in the step's pool;  n_slots concurrent rollout slots
 *   kv_block    KV page size in tokens (must be 16)
 *   max_prompt  longest prompt;  max_new  generated-token cap per rollout
 *   temperature sampling temperature (> 0);  top_p in (0, 1]: 1 samples the
 *               full softmax, < 1 the top-p nucleus (smallest set of most
 *               likely ids whose probability mass reaches top_p, with every
 *               id tied at the cut; mass counted in integer weights
 *               floor(exp(z - z_max) * 2^44) of z = fp32(logit / T)).  The
 *               nucleus path writes fp32 logits [n_slots][vocab] (library
 *               memory for bf16 models) and runs separate sampler kernels
 *   forced_eos_u32  per-token probability x / 2^32 of a forced EOS (0 = off)
 *   prio_quant_bits  quantisation of the p_eff priority key (1..21)
 *   seed        key material of the counter-based sampler and reward hash
 * Limits: min(budget_N, pool_U * k) <= 4096 queued rollouts; pool_U < 2^26;
 * n_slots <= 4096. */
typedef struct {
  int32_t B, k, n0, commit_min;
  double tau_low, alpha0, beta0;
  int64_t budget_N;
  int32_t pool_U, n_slots, kv_block, max_prompt, max_new, mode;
  float temperature, top_p;
  uint32_t forced_eos_u32;
  int32_t prio_quant_bits;
  uint64_t seed;
} sara_alloc_desc;

typedef struct {
  int32_t done;          /* 1 once no prompt is active                      */
  int32_t error;         /* device error word, 0 = none                      */
  int32_t decode_steps;  /* decode steps executed in this allocation step    */
  int32_t drawn;         /* prompts drawn from the pool                      */
  int32_t committed;     /* |C|: effective groups collected                  */
  int32_t abandoned;
  int32_t active;        /* |A|                                             */
  int32_t queued;        /* rollouts waiting for a slot                      */
  int32_t running;       /* occupied slots                                   */
  int32_t pad_;
  int64_t budget_left;   /* N - rollouts issued (k reserved per active prompt) */
  int64_t rollouts;      /* rollouts issued                                  */
  int64_t tokens;        /* tokens generated                                 */
  int64_t n_decisions, n_draws, n_assigns, n_finishes;  /* log lengths       */
} sara_step_stats;

/* Create a context on the current HIP device for one allocation problem:
 * the inputs of Algorithm 1 (its Require line: pool, target B, group size k,
 * probe n0, threshold tau_low, prior (alpha0, beta0), budget cap) plus the
 * defaults of the implementation-details appendix ("Defaults and history
 * warm-start": commit_min, the 6Bk safety cap) and the decoder that
 * generates the rollouts.
 * d_weights: n_weights device pointers in this order, each row-major
 * [out][in] in the model dtype (bf16 as raw 16-bit patterns):
 *   embed[V][d]; per layer l: attn_norm[d], wq[Hq*hd][d], wk[Hkv*hd][d],
 *   wv[Hkv*hd][d], wo[d][Hq*hd], ffn_norm[d], wg[ffn][d], wu[ffn][d],
 *   wd[d][ffn]; then final_norm[d], lm_head[V][d].
 * n_weights must be 3 + 9 * n_layers.  The weights are copied (repacked)
 * into library-owned memory; the caller may free its copies once the stream
 * has passed this call.  stream: a hipStream_t, or NULL for the null stream.
 * All KV, slot, controller and workspace memory is allocated here. */
int sara_init(const sara_model_desc* model, const sara_alloc_desc* alloc,
              const void* const* d_weights, int32_t n_weights, void* stream,
              sara_ctx** out);

/* Start an allocation step over a pool of pool_U prompts (Algorithm 1, first
 * state: the collected set empty, B fresh prompts probed with n0 rollouts
 * each; the pool is the prompt pool D of its Require line).
 * d_tokens: concatenated prompt token ids (device, int32);
 * h_offsets: pool_U + 1 host offsets into d_tokens (prompt u is
 *   [h_offsets[u], h_offsets[u+1]), length 1..max_prompt);
 * d_p: per-prompt success probability of the synthetic verifier (device, fp64);
 * d_forced_len: NULL or [pool_U * k] forced rollout lengths in 1..max_new
 *   (the token at that index becomes EOS and the rollout ends);
 * step_index: enters the sampler key and the reward hash.
 * The inputs are copied; the caller may reuse them once the stream has
 * passed this call.  Enqueues: state reset, prefill of every prompt of the
 * pool into its shared paged KV blocks, the first draws and slot
 * assignments. */
int sara_begin_step(sara_ctx* ctx, const int32_t* d_tokens, const int32_t* h_offsets,
                    const double* d_p, const int32_t* d_forced_len, int32_t step_index);

/* One decode step over every occupied slot, one token for each running
 * rollout: the batched generation call of Algorithm 1 ("one batched call"),
 * and of the implementation-details appendix ("Round-synchronous batched
 * scheduling": one generation call over all active prompts), taken here one
 * token at a time so that decisions can follow every token.  Embedding, n_layers decoder
 * layers over the paged KV cache, LM head, Gumbel-max sampling keyed by
 * (seed, step_index, rollout id uid*k + j, generated index), forced EOS,
 * reward hash, termination.
 * d_forced_tok: NULL or [pool_U * k][max_new] teacher-forcing table (device);
 * the forced token is appended and rewarded, the sampled one is recorded.
 * d_logits: NULL or [n_slots][vocab] fp32 (device); receives the logits of
 * each occupied slot's row.  model_free != 0 skips the decoder: the forced
 * table (required) supplies every token. */
int sara_decode_step(sara_ctx* ctx, const int32_t* d_forced_tok, float* d_logits,
                     int32_t model_free);

/* Section 3.2-3.3 (Beta posterior, Proposition 1, Eq. decide; the loop body
 * of Algorithm 1).  Apply the finished rollouts of the last decode step to
 * their prompts' (n, s) and decide every quiescent active prompt with Eq. decide:
 * Beta(alpha0 + s, beta0 + n - s), p_eff by Proposition 1 (fp64 lgamma),
 * commit / abandon (refund k - n) / continue (queue more rollouts). */
int sara_posterior_decide(sara_ctx* ctx);

/* The reallocation of Algorithm 1 (draw fresh prompts, probe n0, toward the
 * remaining need; advance continuing prompts prioritised by p_eff, section
 * 3.3).  Draw fresh prompts while |A| < B - |C|, budget_left >= k and the pool is
 * not exhausted; order the pending rollouts by (quantised p_eff desc, uid,
 * j) and assign them to free slots in ascending slot order. */
int sara_refill(sara_ctx* ctx);

/* The while loop of Algorithm 1 on the device (implementation-details
 * appendix, "Round-synchronous batched scheduling": rounds of one batched
 * generation call followed by the decisions and the reallocation; here the
 * decisions follow every decode step and no round barrier reaches the
 * host).  Drives the step to completion: replays [decode, decide, refill]
 * from a HIP graph of graph_iters iterations, polling the done flag
 * asynchronously.
 * Synchronises before returning.  d_forced_tok as in sara_decode_step.
 * *iters_out receives the number of loop iterations enqueued. */
int sara_run(sara_ctx* ctx, const int32_t* d_forced_tok, int32_t graph_iters,
             int64_t max_iters, int64_t* iters_out);

/* Synchronise the stream and report the step's counters: the loop state of
 * Algorithm 1 (|C|, |A|, budget left) and its cost in rollouts and tokens
 * (experimental setup appendix, "Metrics").  Returns SARA_EDEVICE when the
 * device error word is set. */
int sara_query(sara_ctx* ctx, sara_step_stats* out);

/* Last line of Algorithm 1: the GRPO update (Eq. grpo, section 2) receives
 * the effective groups of C.  Build the CSR of committed groups (ascending
 * uid, rollouts in j order) and compute their advantages with
 * grpo_group_advantages.  Enqueued. */
int sara_finish_step(sara_ctx* ctx, float eps);

/* History warm start (implementation details, "defaults and history
 * warm-start": each prompt carries its posterior across steps with an
 * exponential decay lambda).  For a finite prompt set revisited across
 * allocation steps, set prompt p keeps pseudo-counts (a_p, b_p) >= 0.
 *
 * sara_set_warm_start: from the next sara_begin_step on, pool prompt u is
 * set prompt d_ids[u] and starts from the prior Beta(alpha0 + a_{ids[u]},
 * beta0 + b_{ids[u]}) in place of Beta(alpha0, beta0): its p_eff, its
 * decisions (Eq. decide on the posterior Beta(alpha0 + a + s,
 * beta0 + b + n - s)) and the priority of its probes use that prior.
 *   d_ids  [pool_U] int32, distinct values in [0, n_store)
 *   d_a, d_b [n_store] fp64 pseudo-counts
 * All three stay owned by the caller and must stay valid while warm start is
 * on: every sara_begin_step reads d_ids, d_a and d_b (update the ids between
 * steps to move the pool over the set), sara_warm_start_update writes d_a
 * and d_b.  d_ids == NULL turns warm start off (back to Beta(alpha0, beta0)).
 * Errors: SARA_EINVAL for a null context, or non-null d_ids with null d_a /
 * d_b or n_store < 1.  An id outside [0, n_store) is found on the device:
 * that prompt falls back to Beta(alpha0, beta0) and the step's device error
 * word gets SARA_DEVERR_WARM_ID (sara_query then returns SARA_EDEVICE).
 * Duplicate ids are not detected; their count updates race. */
int sara_set_warm_start(sara_ctx* ctx, const int32_t* d_ids, double* d_a, double* d_b, int32_t n_store);

/* After a step's decode loop has ended (the step is done): for every set
 * prompt p, a_p <- lambda (a_p + s_p) and b_p <- lambda (b_p + n_p - s_p),
 * where n_p and s_p are the rollouts and successes the step gave the pool
 * prompt with id p (0 and 0 if the step did not draw it).  lambda in [0, 1]:
 * 0 forgets (every step starts cold), 1 keeps every outcome.  Enqueued.
 * Errors: SARA_EINVAL for a null context or lambda outside [0, 1];
 * SARA_ESTATE when no warm start is set or no step has begun. */
int sara_warm_start_update(sara_ctx* ctx, double lambda);

/* Asynchronous poll of the loop condition of Algorithm 1: enqueues on the
 * context's stream a small kernel that writes the device error word to
 * h_pinned[1] and then, after a system-scope fence, the done flag (1 once no
 * prompt is active) to h_pinned[0], and returns at once.  h_pinned: 2 int32
 * of pinned host memory (hipHostMalloc, or a pinned torch tensor) owned by
 * the caller.  Set h_pinned[0] = -1 before the call and spin on it (volatile
 * read) until it changes, or synchronise the stream: h_pinned[1] is valid
 * once h_pinned[0] has changed, which lets the host overlap its own work with
 * the decode loop.  Errors: SARA_EINVAL for a null argument or memory that
 * is not pinned host memory; SARA_ESTATE before sara_begin_step. */
int sara_poll(sara_ctx* ctx, int32_t* h_pinned);

/* Copy results to host (synchronises).  Any pointer may be NULL.
 *   h_tokens  [pool_U*k][max_new] int32 appended tokens (-1 past the end)
 *   h_sampled [pool_U*k][max_new] int32 sampler choices
 *   h_len     [pool_U*k] int32 rollout lengths (0 = never issued)
 *   h_reward  [pool_U*k] int32 rewards
 *   h_status, h_n, h_s [pool_U] int32; h_peff [pool_U] fp64 (last p_eff) */
int sara_read_rollouts(sara_ctx* ctx, int32_t* h_tokens, int32_t* h_sampled, int32_t* h_len,
                       int32_t* h_reward, int32_t* h_status, int32_t* h_n, int32_t* h_s,
                       double* h_peff);

/* Copy logs to host (synchronises).  Row formats (int64 each):
 *   decisions: (t, uid, code, n, s, p_eff bits as int64)   [n_decisions][6]
 *   draws:     (t_start, uid)                               [n_draws][2]
 *   assigns:   (t_start, slot, uid, j)                      [n_assigns][4]
 *   finishes:  (t, slot, uid, j, length, reward)            [n_finishes][6]
 * cap_* are row capacities of the buffers; rows beyond a capacity are dropped. */
int sara_read_logs(sara_ctx* ctx, int64_t* h_dec, int64_t cap_dec, int64_t* h_draw,
                   int64_t cap_draw, int64_t* h_asg, int64_t cap_asg, int64_t* h_fin,
                   int64_t cap_fin);

/* GRPO data of the last sara_finish_step (synchronises).
 * h_offsets [committed + 1], h_rewards / h_adv [offsets[committed]]. */
int sara_read_advantages(sara_ctx* ctx, int32_t* h_offsets, float* h_rewards, float* h_adv,
                         int32_t cap);

/* Closed-form predictor of Proposition 1 (Eq. peff) for count prompts, each
 * under its own prior (section 3.2; per-prompt priors are what the history
 * warm start of the implementation-details appendix produces):
 *   d_out[i] = P(group of size k is mixed | d_n[i] observed, d_s[i]
 *              successes) under the prior Beta(d_alpha[i], d_beta[i])
 * in fp64 via lgamma (the posterior is Beta(alpha + s, beta + n - s)).
 * All five arrays are device memory of count elements, owned by the caller.
 * Entries with a non-positive or non-finite prior parameter, or outside
 * 0 <= s <= n <= k, give NaN.  Argument errors (count < 0, k < 1, a null
 * array with count > 0) return SARA_EINVAL and enqueue nothing.  Pure;
 * enqueued on stream. */
int sara_peff_batch(const double* d_alpha, const double* d_beta, const int32_t* d_n,
                    const int32_t* d_s, int32_t k, int32_t count, double* d_out, void* stream);

/* Group-relative advantages of Eq. grpo: for group g with rewards
 * d_r[d_group_off[g] .. d_group_off[g+1]), A_i = (r_i - mean) / (std + eps),
 * std unbiased (m - 1); groups of size < 2 get 0.  d_group_off has
 * n_groups + 1 entries (device).  Enqueued on stream. */
int grpo_group_advantages(const float* d_r, const int32_t* d_group_off, int32_t n_groups,
                          float eps, float* d_adv, void* stream);

/* Sampler alone, for parity on given logits: rows r < n_rows, logits
 * d_logits[r][vocab] fp32, rollout ids d_rid[r], generated indices d_pos[r]
 * -> d_tok[r] (Gumbel-max at temperature over the top-p nucleus, the whole
 * vocabulary when top_p = 1; forced EOS if eos_id >= 0 and forced_eos_u32 >
 * 0).  top_p in (0, 1], else SARA_EINVAL.  Synchronises the stream. */
int sara_sample_logits(const float* d_logits, int32_t n_rows, int32_t vocab,
                       const int32_t* d_rid, const int32_t* d_pos, uint64_t seed,
                       int32_t step_index, float temperature, float top_p, int32_t eos_id,
                       uint32_t forced_eos_u32, int32_t* d_tok, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * sampler of sara_sample_logits with the same arguments and results, whose
 * buffers (row count, per-row chunk winners, top-p histograms and state)
 * live in one static device array per GPU of SARA_NOALLOC_SCRATCH_BYTES
 * bytes, held from the first call on a device until the process ends.  It
 * calls no allocating routine and does not synchronise: the work is
 * enqueued on stream (which must belong to the current device) and d_tok is
 * valid once the stream has passed it.
 * Limits: n_rows <= SARA_NOALLOC_MAX_ROWS, and n_rows <=
 * SARA_NOALLOC_MAX_TOPP_ROWS when top_p < 1; larger inputs, like the
 * argument errors of sara_sample_logits, return SARA_EINVAL and enqueue
 * nothing.  Every call on one GPU shares that GPU's array: calls whose work
 * overlaps on the device (other streams, other threads) race and give
 * undefined tokens; calls ordered on one stream are safe. */
#define SARA_NOALLOC_MAX_ROWS 4096
#define SARA_NOALLOC_MAX_TOPP_ROWS 64
#define SARA_NOALLOC_SCRATCH_BYTES 17307136
int sara_sample_logits_noalloc(const float* d_logits, int32_t n_rows, int32_t vocab,
                               const int32_t* d_rid, const int32_t* d_pos, uint64_t seed,
                               int32_t step_index, float temperature, float top_p, int32_t eos_id,
                               uint32_t forced_eos_u32, int32_t* d_tok, void* stream);

/* Self-check of the fused LM-head sampler (bf16 models).  That sampler
 * scores every vocabulary id with an fp32 estimate of the Gumbel noise and
 * re-scores exactly (fp64 noise rounded to fp32, the definition of the noise
 * above) only the ids whose estimate lies within a fixed margin of the best;
 * its output equals the exact Gumbel-max provided the estimate is within
 * 2e-5 of the exact noise for every input.  This call evaluates both for all
 * 2^24 noise inputs on the device and writes the largest absolute distance
 * to *h_out (host).  Synchronous on stream; returns SARA_EHIP on HIP
 * failure. */
int sara_gumbel_fast_max_error(double* h_out, void* stream);

/* Per-kernel timing of eager decode steps.  While enabled, every
 * sara_decode_step call (not the graph replays of sara_run) records a HIP
 * event pair around each kernel it launches on the context's stream, waits
 * for them before returning, and adds to that kernel's class the elapsed
 * time and the algorithmic HBM bytes and flops of the launch (weights,
 * activations and the K/V pages the kernel must touch; workspace traffic
 * of split-K partials is not algorithmic and is not counted). */
typedef struct {
  char name[40];
  int64_t launches;
  double ms;      /* summed event-timed kernel time */
  double bytes;   /* algorithmic bytes of those launches */
  double flops;   /* algorithmic flops of those launches */
} sara_kernel_profile;

int sara_set_profiling(sara_ctx* ctx, int32_t enable);   /* totals are kept */
int sara_reset_profile(sara_ctx* ctx);                   /* zero the totals */
/* Copy up to cap classes (in a fixed order) and their totals; *n_out receives
 * the number of classes. */
int sara_read_profile(sara_ctx* ctx, sara_kernel_profile* out, int32_t cap, int32_t* n_out);

void sara_destroy(sara_ctx* ctx);
const char* sara_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SARA_H */
