/*
 * rft.h - C ABI of the MI355X (gfx950) GRPO/PPO trainer-step core.
 *
 * The library computes the data-parallel core of one reinforcement
 * fine-tuning trainer step as described in the Trinity-RFT report
 * (arXiv 2505.17826): per-token policy log-probabilities and entropy over the
 * whole vocabulary, GRPO group-normalised advantages, the clipped PPO
 * surrogate with a KL term toward a reference policy, and the backward pass
 * of that loss to the hidden states and the lm_head weight.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Memory.  Every pointer argument is a DEVICE pointer unless its comment
 *    says (host).  The caller allocates and owns every buffer; the library
 *    never allocates or frees device memory inside a call.  Scratch memory
 *    is passed in as a workspace (`ws`, `ws_bytes`) sized by
 *    rft_workspace_bytes().  Device buffers must be 16-byte aligned.
 *  - Streams.  `stream` is a hipStream_t (NULL = the default stream).  Every
 *    call only enqueues work on that stream and returns without a device
 *    synchronisation.  A return value other than RFT_OK means nothing was
 *    enqueued (except RFT_E_HIP, which reports a launch failure).
 *  - Environment.  RFT_GEMM_STORE_TILE=256 or 384 fixes the workgroup tile
 *    of the fp32-store GEMMs on tile-blocked operands (d_hidden, d_weight);
 *    unset, each call picks the one that takes fewer rounds of tiles on the
 *    device's compute units.  The results are the same bit for bit.
 *  - Errors.  Calls return an rft_status; rft_last_error() gives a
 *    thread-local text describing the last failure.  No call aborts or lets
 *    an exception cross the ABI.  Problems that only the device can see
 *    (token ids out of range) are reported in rft_ppo_stats.n_bad_ids and by
 *    a NaN log-probability for that row; ids are never clamped.
 *  - Token layout (rft_tokens).  T rows (tokens) form n_seq rollouts;
 *    rollout i owns rows [seq_start[i], seq_start[i+1]) with seq_start[0] = 0,
 *    non-decreasing, seq_start[n_seq] = T (a padded [n_seq, L] batch has
 *    seq_start[i] = i*L).  mask[t] != 0 marks a response token that enters
 *    the objective (action mask; multi-turn rollouts mask the environment's
 *    tokens, Sec. 2.2 and Sec. 3.1.2).  Masked rows are never read from the
 *    hidden states or logits and give 0 in every per-row output.  The
 *    contents of seq_start are not validated; an invalid layout gives
 *    unspecified values but every access stays in bounds.
 *  - Expert rollouts (MIX, Sec. 4 example of a new algorithm: online GRPO
 *    mixed with SFT on expert trajectories).  rft_tokens.is_expert may be
 *    NULL (every rollout is an on-policy rollout) or point to n_seq flags;
 *    with flags the loss is (1 - mix_mu) * GRPO loss over the other rollouts
 *    (their own normalisers) + mix_mu * SFT loss over the expert rollouts
 *    (mean of -logp over their valid tokens).
 *  - Matrices are row-major.  hidden is [T, d], weight is [V, d] (the
 *    nn.Linear layout; logits z_t = weight . hidden_t), logits are [T, V].
 *    bf16 data requires d % 8 == 0 and V <= 4194048 (2^22 - 256).
 */
#ifndef RFT_H_
#define RFT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RFT_ABI_VERSION 7

typedef enum {
  RFT_OK = 0,
  RFT_E_NULL = 1,        /* a required pointer is NULL                         */
  RFT_E_SHAPE = 2,       /* a size is negative, inconsistent or unsupported   */
  RFT_E_DTYPE = 3,       /* unknown dtype                                      */
  RFT_E_PARAM = 4,       /* a scalar parameter is out of range                 */
  RFT_E_WORKSPACE = 5,   /* workspace NULL or smaller than required            */
  RFT_E_UNSUPPORTED = 6, /* valid request the library does not implement       */
  RFT_E_HIP = 7          /* the HIP runtime reported an error                  */
} rft_status;

typedef enum { RFT_F32 = 0, RFT_BF16 = 1 } rft_dtype;

/* Loss aggregation over the masked tokens. */
typedef enum {
  RFT_AGG_SEQ_MEAN_TOKEN_MEAN = 0, /* mean over rollouts of per-rollout token means:
                                      weight 1/(S * n_i), S = rollouts with n_i > 0 */
  RFT_AGG_TOKEN_MEAN = 1           /* mean over all valid tokens: weight 1/N          */
} rft_agg;

/* Advantage estimators over explicit groups (rft_group_advantages_ids). */
typedef enum {
  RFT_ADV_GRPO = 0,          /* (r - mean) / (sample std + eps); equal rewards give 0 */
  RFT_ADV_MEAN_CENTER = 1,   /* r - mean                                              */
  RFT_ADV_LEAVE_ONE_OUT = 2  /* r - mean of the other rollouts of the group           */
} rft_adv_mode;

/* Operations, for rft_workspace_bytes(). */
typedef enum {
  RFT_OP_TOKEN_LOGPROBS = 0,
  RFT_OP_TOKEN_LOGPROBS_FROM_LOGITS = 1,
  RFT_OP_PPO_FWD = 2,
  RFT_OP_PPO_BWD = 3,
  RFT_OP_PPO_BWD_LOGITS = 4,
  RFT_OP_PPO_FUSED_LOGITS = 5,
  RFT_OP_PPO_STEP = 6,
  RFT_OP_SFT_FWD = 7,
  RFT_OP_DPO_FWD = 8
} rft_op;

/* (host struct holding device pointers) */
typedef struct {
  int64_t T;                 /* rows                                             */
  int64_t n_seq;             /* rollouts                                         */
  const int32_t* seq_start;  /* [n_seq + 1] row offsets                          */
  const uint8_t* mask;       /* [T] 1 = token in the objective                   */
  const int32_t* token_ids;  /* [T] sampled ids; valid rows should be in [0, V)  */
  const uint8_t* is_expert;  /* [n_seq] 1 = expert rollout (MIX), or NULL        */
} rft_tokens;

/* (host struct) PPO-clip / KL parameters. */
typedef struct {
  float eps_low;          /* ratio lower bound 1 - eps_low, 0 <= eps_low <= 1       */
  float eps_high;         /* ratio upper bound 1 + eps_high, eps_high >= 0 (inf ok) */
  float kl_coef;          /* beta >= 0; 0 disables the KL term (ref_logp may be NULL) */
  int32_t agg;            /* rft_agg                                                */
  double denom_override;  /* 0: use the call's own S (or N); > 0: use this value,
                             e.g. the global count across micro-batches             */
  float mix_mu;           /* weight of the SFT loss on expert rollouts, 0 <= mu <= 1;
                             used only when tokens.is_expert != NULL               */
  float entropy_coef;     /* entropy bonus c_H >= 0: the loss gains
                             -c_H * sum_t w_t H_t over the on-policy tokens (the
                             aggregation weights of the PPO-clip term)             */
} rft_ppo_params;

/* (device struct) loss value and metrics written by the loss calls.  With
 * expert rollouts (MIX), pg_loss, kl_loss, kl_mean, ratio_mean and clipfrac
 * cover the on-policy tokens (N - n_expert of them) and
 * loss = (1 - mix_mu) * (pg_loss + kl_loss - entropy_coef * entropy_loss)
 *        + mix_mu * sft_loss
 * (without expert flags: pg_loss + kl_loss - entropy_coef * entropy_loss). */
typedef struct {
  double loss;          /* pg_loss + kl_loss (MIX: see above)        */
  double pg_loss;       /* sum_t w_t * clipped surrogate              */
  double kl_loss;       /* sum_t w_t * beta * kl_t                    */
  double kl_mean;       /* mean over on-policy tokens of kl_t (0 without ref_logp) */
  double entropy_mean;  /* mean over valid tokens of entropy (0 if no entropy given) */
  double ratio_mean;    /* mean over on-policy tokens of exp(logp - old) */
  double clipfrac;      /* n_clipped / on-policy tokens               */
  int64_t n_valid;      /* N                                          */
  int64_t n_seq_valid;  /* S                                          */
  int64_t n_clipped;
  int64_t n_bad_ids;
  double sft_loss;      /* mean of -logp over expert tokens (0 without) */
  int64_t n_expert;     /* valid tokens of expert rollouts            */
  double entropy_loss;  /* sum_t w_t H_t over on-policy tokens (0 if no entropy given) */
} rft_ppo_stats;

/* (device struct) DPO loss value and metrics written by rft_dpo_loss_fwd.
 * Means are over the counted pairs (both rollouts have a valid token). */
typedef struct {
  double loss;             /* mean of -(1-ls) log sigmoid(u) - ls log sigmoid(-u) */
  double chosen_reward;    /* mean beta (pi_c - rho_c)                           */
  double rejected_reward;  /* mean beta (pi_r - rho_r)                           */
  double reward_acc;       /* fraction of pairs with u > 0                       */
  double margin_mean;      /* mean u                                             */
  int64_t n_pairs;         /* counted pairs P                                    */
  int64_t n_valid;         /* valid tokens N                                     */
  int64_t n_bad_ids;
} rft_dpo_stats;

/* Version of this ABI (RFT_ABI_VERSION). */
int rft_abi_version(void);

/* Static text for a status code. */
const char* rft_status_str(int status);

/* (host) Thread-local description of the last failure in this thread. */
const char* rft_last_error(void);

/* Workspace bytes the operation `op` needs for this layout and sizes (d and V
 * as in the call; dtype of hidden/weight).  For RFT_OP_PPO_BWD and
 * RFT_OP_PPO_STEP the value is the recommended size; any size >=
 * rft_workspace_min_bytes() works, a larger workspace processes more rows per
 * chunk.  For RFT_OP_TOKEN_LOGPROBS the value may include tile-blocked operand
 * copies (see rft_token_logprobs); the minimum is the size without them.  Returns 0 for invalid
 * arguments. */
size_t rft_workspace_bytes(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype);
size_t rft_workspace_min_bytes(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype);

/* Workspace bytes with which RFT_OP_PPO_BWD or RFT_OP_PPO_STEP processes row
 * chunks of chunk_rows rows (rounded up to the chunk alignment, 256 for bf16 and
 * 64 for fp32, and capped at the largest chunk the layout can use).  A caller
 * that knows its count of valid rows can size the workspace so that one chunk
 * holds them all (the step then runs each GEMM once instead of once per chunk).
 * Returns 0 for other operations or invalid arguments. */
size_t rft_workspace_bytes_rows(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype,
                                int64_t chunk_rows);

/* Rows per chunk that RFT_OP_PPO_BWD or RFT_OP_PPO_STEP processes with a
 * workspace of ws_bytes for this layout and sizes (the calls loop over
 * ceil(T / chunk) chunks); 0 if the workspace is too small, the operation has
 * no row chunks or an argument is invalid.  A chunk never exceeds 2^21 rows
 * (its transposed tiles stay within one 2 GiB buffer descriptor). */
int64_t rft_chunk_rows(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype,
                       size_t ws_bytes);

/* GRPO group-relative advantages (Sec. 3.2, Listing 4: advantage_fn "grpo",
 * repeat_times 8; Sec. 3.3.1: 8 rollouts per task).
 * rewards[n_groups * group_size] (f32); rollouts g*G .. g*G+G-1 form group g.
 * adv_i = (r_i - mean_g) / (std_g + eps), std the sample standard deviation
 * (divisor G - 1) when unbiased != 0, else the population one (divisor G); a
 * group whose rewards are all equal (or G == 1) gets 0.
 * adv[n_groups * group_size] (f32) may not alias rewards.
 * Errors: RFT_E_NULL, RFT_E_SHAPE (n_groups < 0, group_size < 1),
 * RFT_E_PARAM (eps < 0 or not finite). */
rft_status rft_group_advantages(const float* rewards, int64_t n_groups, int32_t group_size,
                                float eps, int32_t unbiased, float* adv, void* stream);

/* Advantages over explicit, variable-size groups (Sec. 2.2: rollouts that
 * failed, were skipped or wait for a lagged reward leave their group smaller;
 * Sec. 3.2, Listing 4: advantage_fn grpo).  group_id[i] in [0, n_groups) puts
 * rollout i in that group; an id outside that range leaves the rollout out
 * (advantage 0).  G = the number of rollouts of the group; groups with G < 2
 * give 0.  mode: RFT_ADV_GRPO (as rft_group_advantages: std + eps, the std
 * unbiased as there),
 * RFT_ADV_MEAN_CENTER, RFT_ADV_LEAVE_ONE_OUT (r_i - (sum_g - r_i) / (G - 1)).
 * The rollouts are bucketed by group id (counts, a scan and a scatter in the
 * workspace) and each group's members are sorted by index, so the work grows
 * linearly with n (a group of more than 16384 rollouts scans the ids instead);
 * the fp64 sums over a group's members run in a fixed order, so results are
 * the same run to run.
 * rewards, adv [n] f32, group_id [n] int32; adv may not alias rewards.
 * ws: rft_group_advantages_ids_workspace_bytes(n, n_groups) bytes (about
 * 4 n + 12 n_groups), 16-byte aligned; may be NULL when n == 0.
 * Errors: RFT_E_NULL, RFT_E_SHAPE (n or n_groups < 0 or > 2^31 - 1),
 * RFT_E_PARAM (mode unknown, eps < 0 or not finite), RFT_E_WORKSPACE. */
size_t rft_group_advantages_ids_workspace_bytes(int64_t n, int64_t n_groups);
rft_status rft_group_advantages_ids(const float* rewards, const int32_t* group_id, int64_t n,
                                    int64_t n_groups, int32_t mode, float eps, int32_t unbiased,
                                    float* adv, void* ws, size_t ws_bytes, void* stream);

/* Per-token log-probability of the sampled id, entropy and log-sum-exp of the
 * policy head z_t = weight . hidden_t over the whole vocabulary (Sec. 3.1.1:
 * log-probs of the response tokens; Sec. 3.4.2: actor entropy).
 * hidden [T, d] and weight [V, d] in `dtype` (bf16: MFMA tiles with fp32
 * accumulation; f32: fp32 arithmetic).  The logits are formed tile by tile
 * and folded into an online log-sum-exp; the T x V logits are never stored.
 * Workspace: rft_workspace_bytes(RFT_OP_TOKEN_LOGPROBS, ...) is the
 * recommended size; for bf16 with d % 64 == 0 it includes tile-blocked copies
 * of the valid hidden rows and of weight (about Vpad d 2 bytes more, Vpad = V
 * rounded up to 256), with which the GEMM runs on larger tiles.  Any size >=
 * rft_workspace_min_bytes() works and gives the same results bit for bit.
 * Outputs (f32, [T]): logp (NaN for a valid row whose id is out of range),
 * entropy (may be NULL), lse.  Masked rows are 0.  hidden and the outputs may
 * be NULL when T == 0.
 * Errors: RFT_E_NULL, RFT_E_SHAPE (d < 1, V < 1, T < 0, bf16 with d % 8),
 * RFT_E_DTYPE, RFT_E_WORKSPACE. */
rft_status rft_token_logprobs(const rft_tokens* tok, const void* hidden, const void* weight,
                              int dtype, int64_t d, int64_t V, float* logp, float* entropy,
                              float* lse, void* ws, size_t ws_bytes, void* stream);

/* The same statistics from given fp32 logits [T, V] (Sec. 3.1.1: log-probs of
 * the response tokens under the policy, which PPO and GRPO need; Sec. 3.4.2:
 * the actor's entropy).  This is the statistics half of the loss-only path,
 * for callers whose logits already exist.  gathered (may be NULL)
 * receives logits[t, id_t] (bit-exact copy; NaN for an out-of-range id).
 * Logits of -inf mark vocabulary entries the caller excludes: they get p = 0
 * and add 0 to the entropy, so the results are those of the vocabulary without
 * them (a row needs one finite logit).  The same holds in the loss-only and
 * d_logits calls, whose d_logits are exactly 0 in those columns. */
rft_status rft_token_logprobs_from_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                          float* logp, float* entropy, float* lse,
                                          float* gathered, void* ws, size_t ws_bytes,
                                          void* stream);

/* Clipped PPO surrogate with a k3 KL term toward the reference policy over the
 * masked tokens (Sec. 3.3.2: ratio clipped to 1 +/- 0.2 by default, KL
 * penalty or loss; Sec. 3.2, Listing 4: the policy loss takes the log-probs,
 * the old log-probs, the action mask and the advantages and returns the loss
 * with its metrics).  Per valid token t of rollout i:
 *   rho = exp(logp - old), A = adv[i],
 *   pg = max(-A rho, -A clamp(rho, 1-eps_low, 1+eps_high)),
 *   kl = exp(ref - logp) - (ref - logp) - 1,
 *   loss = sum_t w_t (pg + beta kl)  with w_t from params.agg,
 *   grad_logp[t] = w_t (-A rho [not clipped] + beta (1 - exp(ref - logp))).
 * "Clipped" means A > 0 and rho > 1+eps_high, or A < 0 and rho < 1-eps_low
 * (strict: on a bound the gradient is -A rho).  The test is taken in fp32 on
 * logp - old against fp32(log(1 +/- eps)); it agrees with the exact test
 * except for a token within fp32 rounding (about 1e-7 relative) of a bound.
 * Inputs f32 [T] (adv is [n_seq]); ref_logp may be NULL when kl_coef == 0
 * (no KL: kl_mean is 0); when given, kl_mean reports the KL to it whatever
 * kl_coef, as a metric;
 * entropy may be NULL (entropy_mean 0) unless entropy_coef > 0.  Outputs:
 * grad_logp [T] (0 on masked rows), *stats (device), and, if not NULL,
 * grad_entropy [T]: e_t = d loss / d H_t times -1, i.e. the coefficient of
 * the entropy bonus term in the backward (entropy_coef * w_t on on-policy
 * tokens, scaled by 1 - mix_mu under MIX; 0 elsewhere).  A valid row with an out-of-range id counts
 * in n_bad_ids and adds nothing to the loss, metrics or gradient.  With N = 0
 * the loss and every metric are 0.  Reductions run in fp64 in a fixed order.
 * Errors: RFT_E_NULL, RFT_E_SHAPE, RFT_E_PARAM, RFT_E_WORKSPACE. */
rft_status rft_ppo_clip_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp,
                                 const float* old_logp, const float* ref_logp, const float* adv,
                                 const float* entropy, const rft_ppo_params* params,
                                 float* grad_logp, float* grad_entropy, rft_ppo_stats* stats,
                                 void* ws, size_t ws_bytes, void* stream);

/* Backward of the PPO-clip/KL loss of Sec. 3.3.2 (whose call shape is that of
 * Sec. 3.2, Listing 4: log-probs, old log-probs, action mask, advantages in;
 * loss out) through the policy head z_t = weight . hidden_t, i.e. the
 * trainer's gradient of that loss with respect to the hidden states and the
 * lm_head weight.  The same call back-propagates any loss whose gradient with
 * respect to the log-probs is given (the SFT and DPO losses below).
 * With c_t = grad_logp[t],
 *   dZ_tj = c_t ([j == id_t] - p_tj) + e_t p_tj (z_tj - (lse_t - H_t)),
 *   p_tj = exp(z_tj - lse_t), c_t = grad_logp[t], e_t = grad_entropy[t]
 *   (the entropy bonus term; grad_entropy and entropy may both be NULL,
 *   then e_t = 0),
 *   d_hidden = dZ . weight   ([T, d] f32, masked rows 0, always overwritten),
 *   d_weight = dZ^T . hidden ([V, d] f32, overwritten, or added to when
 *              accumulate_dw != 0).
 * z is recomputed from hidden and weight (it is never stored by the forward);
 * dZ is formed in chunks of rows in the workspace (bf16 for bf16 inputs, kept
 * in both layouts with the chunk's hidden rows transposed, so that both GEMMs
 * read K-contiguous operands: about 4 Vpad + 2 d bytes per chunk row).
 * lse and grad_logp [T] are normally the outputs of rft_token_logprobs and
 * rft_ppo_clip_loss_fwd.
 * Errors: as rft_token_logprobs. */
rft_status rft_ppo_clip_loss_bwd(const rft_tokens* tok, const void* hidden, const void* weight,
                                 int dtype, int64_t d, int64_t V, const float* lse,
                                 const float* grad_logp, const float* grad_entropy,
                                 const float* entropy, float* d_hidden, float* d_weight,
                                 int32_t accumulate_dw, void* ws, size_t ws_bytes, void* stream);

/* Backward of the same loss (Sec. 3.3.2; Sec. 3.2, Listing 4) to given fp32
 * logits, the loss-only path's gradient:
 * d_logits[t, j] = c_t ([j == id_t] - p_tj) + e_t p_tj (z_tj - (lse_t - H_t))
 * with z = logits, as rft_ppo_clip_loss_bwd (grad_entropy and entropy may both
 * be NULL); 0 on masked rows (every row of d_logits [T, V] f32 is written). */
rft_status rft_ppo_clip_loss_bwd_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                        const float* lse, const float* grad_logp,
                                        const float* grad_entropy, const float* entropy,
                                        float* d_logits, void* ws, size_t ws_bytes, void* stream);

/* The loss-only path in one pass per row (Sec. 3.1.1 log-probs and Sec. 3.4.2
 * entropy of the response tokens, the PPO-clip/KL loss of Sec. 3.3.2 with the
 * metrics Sec. 3.2, Listing 4 returns, and its gradient to the logits):
 * log-softmax statistics of the given
 * logits, the PPO-clip/KL loss and metrics, and d_logits, reading each valid
 * logits row once from HBM (the row stays on chip between the statistics and
 * the gradient) and writing d_logits once.  Outputs as rft_token_logprobs_from_logits,
 * rft_ppo_clip_loss_fwd and rft_ppo_clip_loss_bwd_logits (entropy may be
 * NULL; lse and grad_logp may be NULL).  The entropy bonus uses the entropy
 * the call computes, whether or not it is returned. */
rft_status rft_ppo_clip_fused_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                     const float* old_logp, const float* ref_logp,
                                     const float* adv, const rft_ppo_params* params, float* logp,
                                     float* entropy, float* lse, float* grad_logp,
                                     float* d_logits, rft_ppo_stats* stats, void* ws,
                                     size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * call as rft_ppo_clip_fused_logits with the same arguments, results and
 * errors, but no workspace argument.  Its scratch (token bookkeeping and one
 * loss partial per row) lives in a device array inside the library, of
 * rft_noalloc_scratch_bytes() bytes (16 MiB) per GPU, held until the process
 * ends; the call itself allocates and frees nothing.  Limit: the scratch the
 * layout needs must fit, which holds for T <= 131072 rows with n_seq <= T
 * (about 101 bytes per row plus 4 per rollout); a larger layout returns
 * RFT_E_WORKSPACE before anything is enqueued.  Every call on one GPU shares
 * that GPU's array: calls that overlap on one GPU (other streams, other host
 * threads) race and give wrong results, so serialise them.  The array keeps
 * the last call's contents; nothing in it needs to start at zero. */
size_t rft_noalloc_scratch_bytes(void);
rft_status rft_ppo_clip_fused_logits_noalloc(const rft_tokens* tok, const float* logits, int64_t V,
                                             const float* old_logp, const float* ref_logp,
                                             const float* adv, const rft_ppo_params* params,
                                             float* logp, float* entropy, float* lse,
                                             float* grad_logp, float* d_logits,
                                             rft_ppo_stats* stats, void* stream);

/* The whole trainer-side step of the policy head in one call (Sec. 3.3.2 and
 * Listing 4: the trainer's update with the PPO-clip surrogate and k3 KL to the
 * reference model; Sec. 3.1.1: log-probs of the masked response tokens;
 * Sec. 3.2: GRPO advantages given per rollout): the outputs of
 * rft_token_logprobs (logp, entropy, lse), of rft_ppo_clip_loss_fwd
 * (grad_logp, *stats) and of rft_ppo_clip_loss_bwd (d_hidden, d_weight), for
 * the same inputs and with the same conventions (masked rows 0, bad ids,
 * accumulate_dw).  adv is [n_seq] (e.g. from rft_group_advantages).
 * The rows are processed in chunks sized by the workspace.  For bf16 inputs
 * the chunk's forward GEMM keeps, next to the log-sum-exp partials, each
 * logit minus its row's maximum over a 256-column tile in fp16 in the
 * workspace, and the backward forms dZ from it instead of recomputing the
 * logits (6 N d V flops instead of 8 N d V); dZ is kept in both layouts
 * (rows x vocabulary for d_hidden, transposed for d_weight), so the
 * workspace per chunk row is about 4 Vpad + 2 d bytes (the recommended size
 * holds chunks of up to 131072 rows: ~85 GB at V = 152064, d = 3584; a
 * smaller workspace gives smaller chunks, and rft_workspace_bytes_rows sizes
 * one that holds a known count of valid rows in one chunk); logp, entropy, lse, grad_logp
 * and the stats equal those of the separate calls bit for bit, d_hidden and
 * d_weight agree to the rounding of dZ.  For fp32 inputs the call runs the
 * three separate calls in order.  logits are never stored beyond one chunk.
 * entropy may be NULL only when params->entropy_coef == 0.
 * Errors: as rft_token_logprobs and rft_ppo_clip_loss_fwd. */
rft_status rft_ppo_clip_step(const rft_tokens* tok, const void* hidden, const void* weight,
                             int dtype, int64_t d, int64_t V, const float* old_logp,
                             const float* ref_logp, const float* adv,
                             const rft_ppo_params* params, float* logp, float* entropy,
                             float* lse, float* grad_logp, float* d_hidden, float* d_weight,
                             int32_t accumulate_dw, rft_ppo_stats* stats, void* ws,
                             size_t ws_bytes, void* stream);

/* SFT loss of the train-only mode (Sec. 2.1.1: SFT as a special case of
 * training from stored experiences): loss = sum_t w_t (-logp_t) over the
 * valid tokens, w_t from `agg` and `denom_override` as in rft_ppo_params
 * (RFT_AGG_TOKEN_MEAN gives the mean negative log-likelihood, the SFT term of
 * the MIX loss); grad_logp[t] = -w_t (0 on masked rows and for out-of-range
 * ids, which count in n_bad_ids).  tokens.is_expert is ignored.  Writes
 * loss = sft_loss, n_valid, n_seq_valid and n_bad_ids of *stats (the PPO
 * fields are 0).  The gradient feeds rft_ppo_clip_loss_bwd or
 * rft_ppo_clip_loss_bwd_logits.
 * Errors: RFT_E_NULL, RFT_E_SHAPE, RFT_E_PARAM (agg unknown, denom_override
 * negative or not finite), RFT_E_WORKSPACE. */
rft_status rft_sft_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp, int32_t agg,
                            double denom_override, float* grad_logp, rft_ppo_stats* stats,
                            void* ws, size_t ws_bytes, void* stream);

/* DPO loss of the train-only mode (Sec. 2.1.1, DPO on preference pairs;
 * Sec. 2.3.1, the preference-pair data model).  Rollouts 2k and 2k+1 are the
 * chosen and the rejected response of pair k (n_seq must be even).  With
 * pi_s, rho_s the sums of logp and ref_logp over rollout s's valid tokens
 * whose id is in range (fp64, fixed order):
 *   u_k = beta ((pi_2k - rho_2k) - (pi_2k+1 - rho_2k+1)),
 *   loss = (1/P) sum_k [-(1 - ls) log sigmoid(u_k) - ls log sigmoid(-u_k)]
 * over the P pairs whose two rollouts both have a valid token (ls = label
 * smoothing, 0 for plain DPO).  grad_logp[t] = d loss / d pi_s of the row's
 * rollout (0 on masked rows, rows with an out-of-range id and rows of pairs
 * that do not count); it feeds the backward calls as for the other losses.
 * seq_logp [n_seq] (may be NULL) receives pi_s.  Inputs f32 [T].
 * Errors: RFT_E_NULL, RFT_E_SHAPE (odd n_seq), RFT_E_PARAM (beta <= 0 or not
 * finite, ls outside [0, 0.5]), RFT_E_WORKSPACE. */
rft_status rft_dpo_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp,
                            const float* ref_logp, float beta, float label_smoothing,
                            float* grad_logp, float* seq_logp, rft_dpo_stats* stats, void* ws,
                            size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* RFT_H_ */
