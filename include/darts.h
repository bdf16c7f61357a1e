/*
 * darts.h -- C ABI of the MI355X (gfx950) rollout hot path of DARTS
 * (Distribution-Aware Active Rollout Trajectory Shaping).
 *
 * What the library computes (paper Sec. 4.1, Sec. 4.3.1, Alg. 2):
 *   For a batch of N prompts it decodes M'_i = m redundant trajectories per
 *   prompt (intra-prompt redundant rollout), scores every generated token
 *   (log-probability of the taken token and entropy of the next-token
 *   distribution), and per prompt selects the training group of M = k
 *   trajectories: shortest-only selection with proactive early stopping when
 *   m >= m_up (aborting the remaining candidates and reclaiming their KV
 *   pages), or dual-end selection (top-K shortest + top-L longest valid) when
 *   m < m_up.  The notation follows the paper's Tab. 1: q_i prompt, M group
 *   size, M'_i redundant rollout size, N prompts per batch.
 *
 * Conventions for every call
 *   - Return value: 0 (DARTS_OK) or a positive darts_status.  No C++
 *     exception ever crosses this boundary.
 *   - "d_" pointers are device pointers (HIP global memory on the context's
 *     device), "h_" pointers are host pointers.  All are caller-owned unless
 *     stated otherwise; the library never frees them.
 *   - Work is enqueued on the HIP stream given at init (run->stream, NULL is
 *     the legacy default stream).  Calls that return host values synchronise
 *     that stream first.
 *   - Calls on one context must not run concurrently.  Different contexts are
 *     independent.
 *   - After DARTS_EHIP the context is poisoned: every call except
 *     darts_destroy returns DARTS_EHIP again; darts_last_error has the text.
 *
 * Trajectory ids: trajectory j of prompt i has global id g = i*m + j, where
 * m is the context's largest group size; with a redundancy plan (Alg. 1,
 * darts_set_plan) prompt i has candidates j < M'_i <= m only.
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11), key = 64-bit seed,
 * so every trajectory's tokens depend only on (seed, g, step), never on batch
 * composition, row order or physical page ids.
 */
#ifndef DARTS_H
#define DARTS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DARTS_OK = 0,
  DARTS_EINVAL = 1,   /* bad argument or inconsistent shapes */
  DARTS_ENOMEM = 2,   /* device allocation failed or KV page pool exhausted */
  DARTS_ESTATE = 3,   /* call out of order (e.g. decode before prefill) */
  DARTS_EHIP = 4      /* HIP runtime error; context poisoned */
} darts_status;

typedef enum { DARTS_F32 = 0, DARTS_BF16 = 1 } darts_dtype;

/* Flags for darts_run_cfg.flags */
#define DARTS_FLAG_NO_ABORT      0x1u  /* counterfactual: no proactive early stop; every
                                          trajectory runs to its own end before its group
                                          is selected (kept sets are unchanged) */
#define DARTS_FLAG_PERMUTE_PAGES 0x2u  /* initial free list in a seeded random order
                                          (physical page ids must not change any output) */
#define DARTS_FLAG_TIMING        0x4u  /* record HIP events around decode-attention and
                                          GEMM launches on the context's stream, in the
                                          prefill and in every 8th decode step (steps
                                          8, 16, ...); darts_get_stats reports them */
#define DARTS_FLAG_SHARED_PREFIX 0x8u  /* bf16 models: decode attention reads a prompt's
                                          shared pages once per group of its live members
                                          (a prefix kernel) instead of once per row */

#define DARTS_FLAG_STEP_TIMES    0x10u /* record device time of every sampling step (first
                                          launch of the step to the end of its selection
                                          kernel); darts_get_step_times reports them */

#define DARTS_FLAG_STREAM        0x20u /* keep every trajectory's token and log-prob history on
                                          the device ([n_prompts*m][cap] each) for
                                          darts_stream_chunks */

/* Decoder shape.  Weights are generated on the device from weight_seed
 * (Philox uniform, variance 1/fan_in, rounded to bf16 for DARTS_BF16).
 * Dense SwiGLU when n_experts == 0, else top_k-of-n_experts MoE.            */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;    /* n_q_heads % n_kv_heads == 0 (GQA) */
  int32_t head_dim;      /* 32, 64 or 128 */
  int32_t ffn_dim;       /* dense FFN hidden size (ignored for MoE) */
  int32_t vocab;         /* multiple of 4; the end-of-sequence id is vocab-1 */
  int32_t n_experts;     /* 0 for dense; MoE needs BF16, d_model % 256 == 0,
                            d_model <= 5120 */
  int32_t top_k;         /* experts per token (renormalised softmax weights) */
  int32_t expert_ffn;    /* expert SwiGLU hidden size, multiple of 256 */
  float rope_theta;
  float rms_eps;
  int32_t dtype;         /* darts_dtype: F32 (all fp32) or BF16 (bf16 operands,
                            fp32 accumulation and residual stream) */
  uint64_t weight_seed;
  const void* const* weights;  /* NULL: every tensor is generated from weight_seed.
     Otherwise darts_weight_count() device pointers, caller-owned, one per tensor
     in this order, each a row-major [rows][cols] array in the model's dtype (fp32,
     or bf16 bits for DARTS_BF16):
       embed [V][d], lm_head [V][d], then for every layer
         wq [hq*hd][d], wk [hkv*hd][d], wv [hkv*hd][d], wo [d][hq*hd], and
         dense:  w_gate [F][d], w_up [F][d], w_down [d][F]
         MoE:    router [E][d], expert_gate [E][Fe][d], expert_up [E][Fe][d],
                 expert_down [E][d][Fe]
     (the same tensors and layout the generated weights follow; ffn out = w_down
     (silu(w_gate x) * (w_up x))).  darts_init copies them into the context's own
     layout (fused QKV rows, gate/up rows interleaved for the SwiGLU epilogue) and
     keeps no reference: the caller may free them once darts_init returns. */
} darts_model_cfg;

/* Number of tensors in darts_model_cfg.weights for this model: 2 + n_layers *
 * (7 dense, 8 MoE).  0 for a null model.                                    */
int32_t darts_weight_count(const darts_model_cfg* model);

/* One rollout batch.  m and k are passed to darts_init separately.          */
typedef struct {
  int32_t n_prompts;     /* N */
  int32_t prompt_len;    /* Lp, multiple of page_size */
  int32_t cap;           /* system length limit: max generated tokens, < 2^20 */
  int32_t L;             /* dual-end long side size, 1 <= L < k when used (paper: 1) */
  int32_t m_up;          /* shortest-only threshold M_up; 0 means 2k (paper default) */
  int32_t page_size;     /* must be 16 */
  uint64_t kv_pool_bytes;/* KV pool budget in bytes; 0 sizes it for the worst case
                            (every trajectory reaching cap) */
  uint64_t sample_seed;
  float temperature;     /* > 0 */
  uint32_t flags;        /* DARTS_FLAG_* */
  uint64_t page_perm_seed; /* used with DARTS_FLAG_PERMUTE_PAGES */
  void* stream;          /* hipStream_t */
  int32_t traj_base;     /* global id of this batch's trajectory 0, >= 0: the sampler's
                            counters use traj_base + g.  A data-parallel rank that runs
                            prompts [a, b) of a batch sets a*m, so its trajectories draw
                            the random numbers they would draw in a one-GPU run of the
                            whole batch (Sec. 4.2.1: the batch's cost is the maximum
                            over the data-parallel groups).  Every id the library reports
                            stays local (0 .. n_prompts*m-1). */
} darts_run_cfg;

/* Per-step outputs, one row per trajectory decoded in the step (live-list
 * order, ascending trajectory id).  Every pointer is a caller-owned device
 * buffer of capacity n_prompts*m; `sampled` may be NULL.  n_rows is written
 * on the host by the call.                                                  */
typedef struct {
  int32_t* traj_id;      /* global trajectory id g of the row */
  int32_t* token;        /* taken token: end-of-sequence at the forced length,
                            else the teacher-forced token if given, else the sample */
  int32_t* sampled;      /* Gumbel-max sample before any forcing (may be NULL) */
  float* logprob;        /* log p(taken token) under softmax(logits / T) */
  float* entropy;        /* entropy of softmax(logits / T) */
  uint8_t* finished;     /* 0 live, 1 end-of-sequence (valid), 2 truncated at cap */
  int32_t n_rows;
} darts_step_out;

typedef struct {
  int64_t steps;             /* sampling steps done (prefill counts as step 1) */
  int64_t tokens_decoded;    /* all generated tokens, including later-aborted ones */
  int64_t n_pages;           /* KV pool size in pages */
  int64_t pages_used;        /* pages in use now */
  int64_t pages_hwm;         /* high-water mark of pages in use */
  int32_t n_live;
  int32_t n_done;            /* prompts whose kept set is complete */
  /* With DARTS_FLAG_TIMING, estimates for the whole run from the timed
   * launches: each launch of a timed decode step counts 8 times (the steps
   * between timed ones), a prefill launch once.  Ratios (bytes / ms,
   * FLOP / ms) are those of the timed launches.                            */
  double attn_ms;            /* decode-attention time */
  double attn_bytes;         /* algorithmic bytes of those launches: each distinct key and
                                value once per kv head (a prompt's shared pages once per
                                live group), q and out, page ids */
  int64_t attn_launches;
  double gemm_ms;            /* GEMM time (decode and prefill) */
  double gemm_flop;          /* 2*M*N*K summed over those launches */
  int64_t gemm_launches;
  double gemm_cls_ms[6];     /* per GEMM class: QKV, O, gate-up, down, LM head, MoE block
                                (router + routing + grouped experts + combine) */
  double gemm_cls_flop[6];
  double attn_traj_bytes;    /* the same launches' bytes if every row read its whole
                                context itself (equal to attn_bytes unless
                                DARTS_FLAG_SHARED_PREFIX) */
  /* Mixture-of-experts models with DARTS_FLAG_TIMING: the grouped expert
   * GEMMs inside the MoE block ([0] gate/up with the SwiGLU epilogue, [1]
   * down), estimated for the whole run as above.  Bytes are algorithmic:
   * the weights of every expert that received rows, once, plus the routed
   * rows' inputs and outputs.                                              */
  double moe_expert_ms[2];
  double moe_expert_bytes[2];
  int64_t moe_expert_launches[2];
} darts_stats;

typedef struct darts_ctx darts_ctx;

/* ---------------------------------------------------------------- stateful */

/* Allocate a context: weights generated from the seed or copied from the
 * caller's (model->weights), paged KV pool (page = 16 tokens,
 * one pool per layer, prompt pages shared by the prompt's m trajectories),
 * page tables, per-trajectory state and scratch, all owned by the context.
 * m = M'_i (uniform), k = M (paper Tab. 1).  Errors: DARTS_EINVAL if k < 1,
 * k > m, m > 64, L < 1 or L >= k, prompt_len % 16 != 0, cap out of range,
 * unsupported head_dim, or GEMM dimensions that are not multiples of 64/128
 * for BF16, a null entry in model->weights or one that does not point into
 * a device allocation of at least its size; DARTS_ENOMEM if device memory
 * is short.  *out is written only on success.                              */
int darts_init(const darts_model_cfg* model, int32_t m, int32_t k,
               const darts_run_cfg* run, darts_ctx** out);

/* Set the redundancy plan of the next batch (paper Sec. 4.2.2, Alg. 1 output
 * M' = {M'_i}): prompt i gets h_plan[i] candidates, k <= h_plan[i] <= m, and
 * its group is selected shortest-only with early stop when h_plan[i] >=
 * m_up, dual-end otherwise (Alg. 2).  Valid only before darts_prefill
 * (after darts_init or darts_reset, which both restore the uniform plan
 * h_plan[i] = m).  Errors: DARTS_EINVAL for a size out of [k, m],
 * DARTS_ESTATE after the prefill.  Synchronises the stream.                */
int darts_set_plan(darts_ctx* ctx, const int32_t* h_plan);

/* Prefill every prompt and sample generated token 0 of every trajectory
 * (paper Alg. 2: rollout of the candidate pool T_i).
 *   d_prompts      [n_prompts * prompt_len] int32 token ids in [0, vocab)
 *   d_forced_len   [n_prompts * m] int32 >= 1: trajectory g emits the
 *                  end-of-sequence id as its d-th generated token when
 *                  d <= cap; d > cap means it is truncated at cap
 *   d_force_tokens NULL or [n_prompts * m] int32 teacher-forced token 0 per
 *                  trajectory (-1: no force)
 * Writes `out` (n_rows = the number of candidates of the plan, n_prompts*m
 * for the uniform one).  DARTS_ESTATE if called twice.                      */
int darts_prefill(darts_ctx* ctx, const int32_t* d_prompts, const int32_t* d_forced_len,
                  const int32_t* d_force_tokens, darts_step_out* out);

/* One decode step over the live trajectories: consume each one's last token,
 * append its key/value to the paged pool (taking a fresh page when a page
 * fills), run the decoder, and sample + score the next token.
 *   d_force_tokens NULL or [n_prompts * m] int32 indexed by trajectory id
 *                  (-1: no force): the token to take at this step.
 * DARTS_ENOMEM when the pool lacks the pages this step needs (checked before
 * any write; state unchanged).  DARTS_ESTATE before prefill or when no
 * trajectory is live.                                                      */
int darts_decode_step(darts_ctx* ctx, const int32_t* d_force_tokens, darts_step_out* out);

/* Apply the selection of Alg. 2 to every prompt whose group can complete
 * after the latest step: shortest-only with early stop (m >= m_up) keeps the
 * first k valid finished trajectories in shortest-first order and aborts the
 * live rest; dual-end (m < m_up) waits for all members, then keeps the K
 * shortest followed by the L longest valid of the rest.  Frees the private
 * pages of every trajectory that finished or was aborted, and a prompt's
 * shared pages when its last member is done; compacts the live list.
 *   d_kept      [n_prompts * k] int32, row i = prompt i's kept ids (short
 *               side first); -1 in rows of prompts not complete yet
 *   d_done_step [n_prompts] int32: the step at which prompt i completed
 *               (the prefill is step 1), -1 while incomplete
 *   h_n_live, h_n_done: host outputs (may be NULL).
 * Idempotent when nothing changed.                                          */
int darts_select_and_prune(darts_ctx* ctx, int32_t* d_kept, int32_t* d_done_step,
                           int32_t* h_n_live, int32_t* h_n_done);

int darts_get_stats(const darts_ctx* ctx, darts_stats* out);

/* Per decode step wall time on the device (DARTS_FLAG_STEP_TIMES): step i
 * decoded h_rows[i] trajectories in h_ms[i] milliseconds, from its first
 * launch to the end of the selection kernel that followed it; up to cap
 * entries are written, *h_n = the number of decode steps recorded since the
 * prefill.  *h_prefill_ms (may be NULL): the prefill step.  These are the
 * (batch size, per-token latency) samples of the cost model (Sec. 4.2.1,
 * App. A).  DARTS_ESTATE without the flag.                                 */
int darts_get_step_times(const darts_ctx* ctx, int32_t* h_rows, float* h_ms, int32_t cap,
                         int32_t* h_n, float* h_prefill_ms);

/* Token-level streaming, producer side (Sec. 4.3.2, App. E).  Tokens generated
 * since a trajectory's last dispatch are pending; when the pending total over
 * all trajectories is >= threshold, or flush != 0 and anything is pending or
 * some ended trajectory has not been marked final, every trajectory with
 * pending tokens or an unsent final mark gets one descriptor, ascending id:
 *   d_desc[4i .. 4i+3] = {trajectory id, first token index, token count,
 *                         final status (1 eos, 2 truncated, 3 aborted; 0: more
 *                         tokens will come)}
 * and its tokens and log-probs are copied, in descriptor order, to
 * d_tokens / d_logprobs (out_cap entries each).  Otherwise nothing is
 * written and *h_n_desc = 0.  Kept sets come from darts_select_and_prune.
 * d_desc holds n_prompts*m*4 int32.  Call after darts_select_and_prune; flush
 * once every kept set is complete to deliver the rest.  Errors: DARTS_ESTATE
 * without DARTS_FLAG_STREAM or before the prefill; DARTS_ENOMEM if the
 * pending tokens exceed out_cap (nothing dispatched, state unchanged).       */
int darts_stream_chunks(darts_ctx* ctx, int64_t threshold, int32_t flush, int32_t* d_desc,
                        int32_t* d_tokens, float* d_logprobs, int64_t out_cap, int32_t* h_n_desc,
                        int64_t* h_n_tokens);

/* Start a new batch on the same context: weights, pool and buffers are
 * kept; the free list, page tables, per-trajectory and per-prompt state and
 * the statistics are reset.  Synchronises the stream.  The next call must be
 * darts_prefill.                                                           */
int darts_reset(darts_ctx* ctx);

/* Final per-trajectory scores (device buffers of n_prompts*m, each may be
 * NULL): generated length, float32 sum of log-probs in step order, mean
 * = sum / length, status (0 live, 1 eos, 2 truncated, 3 aborted, 4 not a
 * candidate of the plan: length 0).                                        */
int darts_get_traj_scores(darts_ctx* ctx, int32_t* d_len, float* d_sum_lp, float* d_mean_lp,
                          uint8_t* d_status);

/* Copy the last step's float32 logits [n_rows * vocab] (rows in the order of
 * the last darts_step_out) into d_dst.  For verification.                  */
int darts_debug_logits(darts_ctx* ctx, float* d_dst, int32_t* h_n_rows);

/* Set every byte of the context's key and value pools to `byte` (0..255;
 * 0xff makes every element a NaN), as memory left by earlier work might
 * hold.  For verification that no result depends on pool contents the
 * rollout has not written itself.  Synchronises the stream.  Errors:
 * DARTS_ESTATE unless called after darts_init or darts_reset and before
 * darts_prefill; DARTS_EINVAL for a byte outside 0..255.                   */
int darts_debug_fill_kv(darts_ctx* ctx, int32_t byte);

/* Verification of mixture-of-experts routing (MoE models only).  Until the
 * next call, every prefill and decode step reads and writes, for each of its
 * rows and each layer l, entries [key][l][0..top_k) of these device buffers
 * (each [n_keys][n_layers][top_k], caller-owned, any may be NULL), where key
 * is the prompt position i*prompt_len + t for prefill rows and the
 * trajectory id for decode rows:
 *   d_force_ids  int32 expert ids to combine instead of the router's own
 *                top-k, weighted by their own softmax probabilities
 *                renormalised over the k (the routing analogue of teacher
 *                forcing); a row whose entry 0 is negative, or that holds an
 *                id outside [0, n_experts), keeps its own routing
 *   d_own_ids    int32 out: the router's own top-k ids, rank order
 *   d_used_p     float out: softmax probability of each combined expert
 * All NULL turns verification off.  Errors: DARTS_EINVAL for a dense model
 * or n_keys < max(n_prompts*prompt_len, n_prompts*m).                      */
int darts_debug_moe_routing(darts_ctx* ctx, const int32_t* d_force_ids, int32_t* d_own_ids,
                            float* d_used_p, int64_t n_keys);

int darts_destroy(darts_ctx* ctx);
const char* darts_strerror(int status);
const char* darts_last_error(const darts_ctx* ctx);

/* ------------------------------------------------------- batch planning   */
/* Host-only calls (no device work, no context): they decide the redundancy
 * plan of the next batch from the previous rollouts.  All arithmetic is
 * float64; results are bitwise reproducible.                               */

/* Population standard deviation of each prompt's candidate lengths, the
 * per-prompt long-tail signal of Sec. 4.2.2: h_std[i] over h_len[i*m + j],
 * j < h_plan[i] (h_plan NULL: j < m).  h_len as from darts_get_traj_scores
 * (aborted candidates count with the length they reached).                 */
int darts_prompt_length_std(const int32_t* h_len, const int32_t* h_plan, int32_t n_prompts,
                            int32_t m, double* h_std);

/* Exponential moving average of a per-prompt statistic (the smoothed
 * historical variance of Sec. 4.2.2 / App. C): for every i with h_obs[i]
 * not NaN, h_est[i] = h_obs[i] if !h_seen[i] else alpha*h_obs[i] +
 * (1-alpha)*h_est[i], and h_seen[i] = 1.  0 < alpha <= 1.                   */
int darts_ema_update(double* h_est, uint8_t* h_seen, const double* h_obs, int32_t n, double alpha);

/* Adaptive total budget (App. B): the utility rho*ln(M) - lambda*(k_cost*M
 * + c) peaks at M* = rho / (lambda*k_cost); *h_m_total = clip(floor(M*),
 * M*n_prompts, 2*M*n_prompts).  rho = sigma_L / mean_L of recent response
 * lengths, k_cost = rollout seconds per extra candidate (cost model of
 * Sec. 4.2.1).  lambda <= 0 or k_cost <= 0 gives the upper bound.           */
int darts_redundancy_budget(double rho, double lambda, double k_cost, int32_t n_prompts, int32_t M,
                            int64_t* h_m_total);

/* Variance-based allocation (Alg. 1): w_i = min-max normalised h_sigma[i]
 * (all equal: 1; prompts with h_seen[i] == 0 first take the mean of the
 * seen ones; h_seen NULL: all seen); every prompt starts at m_low and the
 * remaining m_total - n*m_low candidates go one at a time to the prompt
 * with the largest w_i*(1/M'_i - 1/(M'_i+1)) still below m_up (ties: lowest
 * index).  A surplus beyond n*m_up stays unallocated.  Writes h_plan[n].    */
int darts_allocate_redundancy(const double* h_sigma, const uint8_t* h_seen, int32_t n_prompts,
                              int32_t m_low, int32_t m_up, int64_t m_total, int32_t* h_plan);

/* Rollout cost model, Eq. 4 (Sec. 4.2.1): with the n lengths sorted
 * (l_[0] = 0), *h_T = sum_m (l_[m] - l_[m-1]) * PTL(n - m + 1), where
 * PTL(b) = c0 + c1*b + c2*max(0, b-b1) + c3*max(0, b-b2) and
 * h_ptl = {b1, b2, c0, c1, c2, c3}.  Lengths are the numbers of decode steps
 * each trajectory takes part in; the result is in PTL's unit.  For data
 * parallel ranks the batch cost is the maximum over ranks.                  */
int darts_rollout_cost(const int32_t* h_len, int32_t n, const double* h_ptl, double* h_T);

/* Eq. 4 under data parallelism (Sec. 4.2.1): trajectory i runs on rank
 * h_rank[i] in [0, n_ranks); each rank's batch costs Eq. 4 over its own
 * lengths and *h_T is the maximum over ranks (an empty rank costs 0).
 * DARTS_EINVAL for a rank out of range.                                     */
int darts_rollout_cost_dp(const int32_t* h_len, const int32_t* h_rank, int32_t n, int32_t n_ranks,
                          const double* h_ptl, double* h_T);

/* Three-stage piecewise-linear PTL fit (App. A): least squares of
 * h_lat[i] ~ PTL(h_bsz[i]) over every breakpoint pair b1 = xs[i] < b2 = xs[j],
 * 1 <= i < j <= D-2, of the D distinct batch sizes xs (ascending), the
 * smallest residual winning (ties: the first pair).  D < 4: one line
 * (b1 = b2 = largest size, c2 = c3 = 0); D = 1: the mean.  Writes
 * h_ptl[6] = {b1, b2, c0, c1, c2, c3}.  DARTS_EINVAL for non-finite
 * latencies.                                                               */
int darts_fit_ptl(const int32_t* h_bsz, const double* h_lat, int32_t n, double* h_ptl);

/* ----------------------------------------------------- stateless kernels  */
/* These run one kernel of the path on caller-provided device buffers, for
 * kernel sweeps and parity checks "given the same inputs".  A call whose
 * work size (rows, M, trajectories, groups, bytes, elements) is zero checks
 * its scalar arguments, does nothing and returns DARTS_OK; its device
 * pointers may then be NULL.                                               */

/* Fill d_dst[0..n) with element idx = bf16(((w>>8)|1)*2^-23 - 1),
 * w = Philox(key=seed, counter=(idx>>2, tensor, 0, 3)) word idx&3, stored as
 * bf16 or (dtype DARTS_F32) as the same value in float32.                  */
int darts_fill_uniform(void* d_dst, uint64_t n, int32_t tensor, uint64_t seed, int32_t dtype,
                       void* stream);

/* Read d_src[0..bytes) once with 16-byte non-temporal loads (2048 blocks x
 * 256 threads, grid-stride) and write 8192 wavefront sums to d_sink
 * (caller-owned, 8192 floats).  A streaming-read reference: the HBM read
 * rate this device sustains (non-temporal loads stream faster than plain
 * ones), against which the bandwidth-bound kernels are also reported.
 * bytes must be a multiple of 16 and d_src 16-byte aligned.                */
int darts_stream_read(const void* d_src, int64_t bytes, float* d_sink, void* stream);

/* Fill the paged K and V pools of the attention sweep with the values above
 * (tensor 1 for K, 2 for V) at logical index ((page*Hkv + h)*16 + slot)*hd + d,
 * written in the library's physical pool layouts (n_pages pages, dtype as
 * for darts_fill_uniform).  Each pool holds n_pages*Hkv*16*hd elements;
 * head_dim must be a positive multiple of 32 (else DARTS_EINVAL).          */
int darts_fill_kv_pool(void* d_k_pool, void* d_v_pool, int64_t n_pages, int32_t n_kv_heads,
                       int32_t head_dim, uint64_t seed, int32_t dtype, void* stream);

/* Bytes of workspace darts_attn_decode needs for these sizes.              */
size_t darts_attn_workspace_bytes(int32_t n_rows, int32_t n_q_heads, int32_t n_kv_heads,
                                  int32_t head_dim, int32_t max_ctx);

/* Paged GQA decode attention (the scaled dot-product attention of the
 * decoder): for each row r and q head h,
 *   out[r][h] = sum_j softmax_j(q[r][h] . k_j / sqrt(hd)) v_j,  j < ctx_len[r],
 * key j of row r lives in page page_table[r*pt_stride + j/16], slot j%16, kv
 * head h / (n_q_heads/n_kv_heads).
 *   d_q, d_out    [n_rows][n_q_heads][head_dim] (bf16, or f32 with DARTS_F32)
 *   d_k_pool/v    pools of n_pages pages in the library layout (as filled by
 *                 darts_fill_kv_pool); page ids are clamped into [0, n_pages)
 *   d_page_table  [n_rows][pt_stride] int32, pt_stride >= ceil(max_ctx/16)
 *   d_ctx_len     [n_rows] int32 in [1, max_ctx] (larger values are clamped,
 *                 rows with ctx <= 0 are left unwritten), or NULL: every row
 *                 has max_ctx keys.  This equal-context form is the one a
 *                 decode step takes (in bf16 the work is mapped without a
 *                 device-built list, and from 64 rows each wavefront keeps
 *                 two page pairs in flight).
 *   d_workspace   darts_attn_workspace_bytes(...) bytes, 256-byte aligned
 * In bf16 the value slots of a row's last page at or past ctx_len[r] take
 * part in the P.V product with weight 0, so they must hold finite values
 * (the context's own decode appends clear them when they open a page).
 */
int darts_attn_decode(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                      int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                      const int32_t* d_ctx_len, int32_t n_rows, int32_t n_q_heads,
                      int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx, int32_t dtype,
                      void* d_out, void* d_workspace, size_t workspace_bytes, void* stream);

/* Allocation-free decode attention, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation, kernels and results as
 * darts_attn_decode (bit for bit), with the workspace taken from an array of
 * DARTS_ATTN_NOALLOC_SCRATCH_BYTES that the library's code object holds on
 * each GPU for the life of the process.  The call allocates nothing, neither
 * device nor host memory.  Arguments as for darts_attn_decode without the
 * workspace.  Errors: DARTS_EINVAL as there, and also when
 * darts_attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim,
 * max_ctx) exceeds DARTS_ATTN_NOALLOC_SCRATCH_BYTES (nothing is launched);
 * DARTS_EHIP if the array's device address cannot be looked up.  Every call
 * on one GPU uses that GPU's one array: calls that overlap in time on the
 * same GPU (other streams, other threads) race and must be serialised by
 * the caller.                                                              */
#define DARTS_ATTN_NOALLOC_SCRATCH_BYTES (64u << 20)
int darts_attn_decode_noalloc(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                              int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                              const int32_t* d_ctx_len, int32_t n_rows, int32_t n_q_heads,
                              int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx, int32_t dtype,
                              void* d_out, void* stream);

/* Bytes of workspace darts_attn_decode_shared needs for these sizes.       */
size_t darts_attn_shared_workspace_bytes(int32_t n_rows, int32_t n_q_heads, int32_t n_kv_heads,
                                         int32_t head_dim, int32_t ctx_len, int32_t prefix_pages);

/* The same decode attention for rows that share a prompt prefix, as the m
 * trajectories of one prompt do in the rollout (their prompt's KV pages are
 * shared, Alg. 2 samples them from one prompt): the shared pages are read
 * once per group of rows instead of once per row.  bf16 only.
 *   d_row_traj    [n_rows] int32: row r uses page-table row d_row_traj[r]
 *                 (clamped into [0, pt_rows)); rows r with equal
 *                 d_row_traj[r] / m that are consecutive form a group
 *   d_page_table  [pt_rows][pt_stride] int32, pt_stride >= ceil(ctx_len/16);
 *                 the members of a group must have equal first prefix_pages
 *                 entries (the prefix is read through the group's first row)
 *   ctx_len       every row's context, > 16 * prefix_pages
 *   d_q, d_out, pools, page ids: as for darts_attn_decode
 *   d_workspace   darts_attn_shared_workspace_bytes(...) bytes, 256-byte aligned
 * Returns DARTS_EINVAL for inconsistent sizes or dtype != DARTS_BF16.       */
int darts_attn_decode_shared(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                             int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                             int32_t pt_rows, const int32_t* d_row_traj, int32_t m,
                             int32_t prefix_pages, int32_t ctx_len, int32_t n_rows, int32_t n_q_heads,
                             int32_t n_kv_heads, int32_t head_dim, int32_t dtype, void* d_out,
                             void* d_workspace, size_t workspace_bytes, void* stream);

/* Fused sampler: for each row, Gumbel-max token with counter (traj, step),
 * log-prob of the taken token (d_force[r] if d_force != NULL and >= 0, else
 * the sample) and entropy of softmax(logits / T).
 *   d_logits [n_rows][vocab] (bf16 or f32), d_traj/d_step [n_rows] int32.
 * A row with no finite perturbed score (every logit -inf or NaN) samples
 * token 0 and gets NaN log-prob and entropy; no memory outside the row is
 * read.  (The rollout's sampler behaves the same way.)                      */
int darts_sample(const void* d_logits, int32_t n_rows, int32_t vocab, int32_t dtype,
                 uint64_t seed, const int32_t* d_traj, const int32_t* d_step, float temperature,
                 const int32_t* d_force, int32_t* d_token, float* d_logprob, float* d_entropy,
                 void* stream);

/* Stateless selection over groups of m consecutive trajectories (Alg. 2),
 * with the page reclaim of the aborted and finished candidates (Alg. 2's
 * abort; Sec. 4.3.1, proactive early stopping frees the pruned candidates).
 *   d_status   [n_traj] uint8 in/out: 0 live, 1 eos, 2 truncated, 3 aborted
 *              (aborted is written for pruned live members: the abort mask)
 *   d_len      [n_traj] int32 generated lengths (< 2^20)
 *   d_mean_lp  [n_traj] float32 mean log-probs (tie-break only)
 *   d_kept     [n_groups * k] int32 out (rows of incomplete groups untouched)
 *   d_complete [n_groups] uint8 out: 1 if the group completed now
 *   m_up: shortest-only when m >= m_up; early_stop: 0 or 1.
 * Page reclaim (d_page_off NULL: none, and the next four pointers are
 * ignored): trajectory g owns the KV page ids d_pages[d_page_off[g] ..
 * d_page_off[g+1]) (d_page_off: [n_traj + 1] int32, non-decreasing, from 0).
 * Every group that completes in this call frees the pages of all its
 * members, which are all done once it completes: they are written to
 * d_free_out (capacity d_page_off[n_traj] ids) in group order, member order
 * and list order, and their number to the device int32 *d_n_free.  d_work:
 * n_traj / m + 1 int32 of scratch.  The call keeps no state: a caller passes
 * each group's pages until the call that completes the group, then drops
 * them (or gives that group an empty list).                                */
int darts_select_groups(uint8_t* d_status, const int32_t* d_len, const float* d_mean_lp,
                        int32_t n_traj, int32_t m, int32_t k, int32_t L, int32_t m_up,
                        int32_t early_stop, int32_t* d_kept, uint8_t* d_complete,
                        const int32_t* d_page_off, const int32_t* d_pages, int32_t* d_free_out,
                        int32_t* d_n_free, int32_t* d_work, void* stream);

/* Group-normalised advantages of the kept training groups (Sec. 3.1, Eq. 2):
 * for group i with kept ids d_kept[i*k + j] (as written by
 * darts_select_and_prune), d_adv[i*k + j] = (r_j - mu_i) / (sigma_i + eps)
 * with r_j = d_reward[kept id], mu_i and sigma_i the mean and population
 * standard deviation of the group's k rewards, in float32.  A group holding
 * an id outside [0, n_traj) (not complete) gets NaN.  k <= 64.             */
int darts_group_advantages(const int32_t* d_kept, int32_t n_groups, int32_t k, const float* d_reward,
                           int32_t n_traj, float eps, float* d_adv, void* stream);

/* The decoder's dense projection (a plain GEMM with the decoder's fused
 * epilogues): C = A[M,K] . W[N,K]^T with fp32 accumulation.
 *   d_a  [M][K], d_w [N][K]: bf16 (DARTS_BF16) or f32 (DARTS_F32), row-major
 *   epilogue 0: d_c [M][N] f32 = result
 *            1: d_c [M][N] in the operand dtype = result (rounded)
 *            2: d_c [M][N] f32 += result (residual add)
 *            3: SwiGLU: W rows are interleaved in groups of 16 (16 gate rows,
 *               then the 16 up rows of the same features); d_c [M][N/2] in
 *               the operand dtype = silu(gate) * up
 *   bf16 requires N % 128 == 0 and K % 256 == 0.  d_workspace must hold
 *   darts_gemm_workspace_bytes(M, N, K) bytes (split-K partial sums).      */
size_t darts_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K);
int darts_gemm(const void* d_a, const void* d_w, void* d_c, int32_t M, int32_t N, int32_t K,
               int32_t dtype, int32_t epilogue, void* d_workspace, size_t workspace_bytes,
               void* stream);

/* Gumbel noise map used by darts_sample: d_g[i] = -ln(-ln(d_u[i])) with the
 * library's float32 logarithm (a fixed sequence of correctly rounded float32
 * operations: atanh series on the reduced mantissa).  d_u in (0, 1).  For
 * bit-exact verification of the sampler's noise.                           */
int darts_debug_gumbel(const float* d_u, float* d_g, int64_t n, void* stream);

/* The sampler's fast Gumbel map (two hardware log2 evaluations), which only
 * pre-selects candidates: d_g[i] = -ln(-ln(d_u[i])) approximately, d_u in
 * [2^-24, 1 - 2^-24].  darts_sampler_gumbel_bound() is the distance from the
 * exact map (darts_debug_gumbel) that the sampler's filter assumes; the
 * token is the exact-noise argmax provided the fast map stays within it on
 * every u = (2k+1) 2^-24, which callers can check exhaustively with these
 * two entries.  The filter's soundness argument: a thread's best fast score
 * more than twice that distance (plus float32 rounding of the sums) above
 * its second best is its exact winner; nearer cases are rescanned exactly.
 * Same stream and error semantics as darts_debug_gumbel.                   */
int darts_debug_gumbel_fast(const float* d_u, float* d_g, int64_t n, void* stream);
float darts_sampler_gumbel_bound(void);

#ifdef __cplusplus
}
#endif
#endif /* DARTS_H */
