/*
 * rlk — policy-gradient hot path of black-box agentic RL on MI355X (gfx950).
 *
 * The computation (ClawGym II, Sec. 2.3 and 3.2):
 *   z_t = W h_t over the whole vocabulary (LM-head projection),
 *   log pi(y_t|s_t) = z_{t,y_t} - logsumexp(z_t), entropy H_t of softmax(z_t),
 *   group-relative advantage A_i = (R_i - mu_q)/(sigma_q + eps) over the rollouts of a
 *   task (or task-harness pair) with the population std (Sec. 2.3.2, Sec. 3.2.3, Sec. 3.3),
 *   the masked clipped surrogate min(rho A, clip(rho, 1-eps_lo, 1+eps_hi) A) with
 *   rho = exp(logp - old_logp) and binary mask M_t (Sec. 2.3.1, masked GRPO objective of
 *   Sec. 2.3.2), and its gradients dL/dhidden and dL/dW.
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer unless stated otherwise; row-major layout.
 *   - hidden [N, d], W [V, d] and dhidden [N, d] use the batch dtype (fp32 or bf16).
 *     Their base pointers and rows must be 16-byte aligned: d must be a multiple of 8
 *     (a misaligned pointer is rejected with RLK_EINVAL).
 *   - targets[t] is the token sampled at position t, already aligned with hidden[t] (no
 *     shift inside); on policy rows it must lie in [0, V); on other rows it is ignored.
 *   - mask[t] = 1 marks a policy-generated token (trained); 0 marks harness/tool tokens.
 *     NULL means every token is a policy token.
 *   - cu_seqlens [R+1] (device int32) packs rollouts back to back: rollout r owns
 *     positions [cu[r], cu[r+1]); cu[0] = 0, cu[R] = N, non-decreasing.
 *   - group_ids [R] are opaque int32 keys; rollouts sharing a key form one group.
 *     A negative key excludes the rollout from advantage estimation and from the loss
 *     (sandbox failures, Sec. 3.4).
 *   - Ownership: the caller owns every buffer including the workspace; the library never
 *     allocates or frees device memory on any call below.
 *   - Streams: all work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *     Calls return without synchronising; outputs are valid once the stream reaches the
 *     point of the call.  Concurrent calls must use distinct workspaces.
 *   - Errors: invalid arguments are reported synchronously before anything is launched
 *     (RLK_EINVAL, RLK_ESHAPE, RLK_EDTYPE, RLK_EWORKSPACE); a failed launch returns
 *     RLK_EHIP.  Errors in device-resident data (out-of-range target on a policy row,
 *     malformed cu_seqlens) cannot be seen by the host without a sync; kernels stay in
 *     bounds, set bits in a status word held in the workspace, and rlk_check_status()
 *     reports them.  Setting the environment variable RLK_DEBUG_SYNC=1 makes every call
 *     synchronise and check that word.  rlk_last_error() describes the last failure of
 *     the calling thread.
 */
#ifndef RLK_H
#define RLK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RLK_VERSION 7

typedef int32_t rlk_status_t;
enum {
  RLK_OK = 0,
  RLK_EINVAL = 1,     /* null pointer or out-of-range scalar argument */
  RLK_ESHAPE = 2,     /* inconsistent or unsupported sizes */
  RLK_EDTYPE = 3,     /* unknown dtype */
  RLK_EWORKSPACE = 4, /* workspace missing, misaligned or too small */
  RLK_EHIP = 5,       /* a HIP runtime call or kernel launch failed */
  RLK_EDATA = 6       /* device data error found by rlk_check_status */
};

enum { RLK_DTYPE_F32 = 0, RLK_DTYPE_BF16 = 1 };

/* Token aggregation of the objective.
 * SEQ_MEAN_TOKEN_MEAN (default, the masked GRPO objective of Sec. 2.3.2 with the
 *   tree rule of Sec. 3.2.3): per-rollout masked token mean, 1/G_q over the rollouts of
 *   a group, then the mean over the Q groups of the batch.
 * TOKEN_MEAN (the hat-E_t form of Sec. 2.3.1): one masked token mean over the batch. */
enum { RLK_AGG_SEQ_MEAN_TOKEN_MEAN = 0, RLK_AGG_TOKEN_MEAN = 1 };

/* Bits of the device status word (rlk_check_status). */
enum {
  RLK_DERR_TARGET = 1,       /* a policy row's target lies outside [0, V) */
  RLK_DERR_CU_SEQLENS = 2,   /* cu[0] != 0, cu decreasing, or cu[R] != N */
  RLK_DERR_POLICY_BOUND = 4  /* more trained tokens than rlk_batch_t.max_policy_tokens; the
                                outputs of that call are not valid */
};

/* Size limits: the GEMMs address 256-row operand panels with 32-bit buffer offsets, so a
 * panel (256 rows of d, V or chunk_rows elements) must stay below 2 GiB. */
#define RLK_MAX_DIM 2097152
#define RLK_MAX_CHUNK_ROWS 1048576

typedef struct {
  int64_t N;                  /* packed tokens (rows of hidden) */
  int32_t R;                  /* rollouts */
  int32_t d;                  /* hidden size, multiple of 8, at most RLK_MAX_DIM */
  int32_t V;                  /* vocabulary size, 1 .. RLK_MAX_DIM */
  int32_t dtype;              /* RLK_DTYPE_F32 or RLK_DTYPE_BF16 */
  const int32_t* cu_seqlens;  /* device [R+1] */
  float temperature;          /* sampling temperature tau of the policy: logits z = W h / tau;
                                 0 means 1 (the default); otherwise finite and > 0 */
  int32_t max_policy_tokens;  /* optional host-known upper bound on the trained tokens (mask = 1 in
                                 non-excluded rollouts): 0 = unknown, the chunk loop then covers all
                                 N rows and skips empty chunks on the device; > 0 sizes the chunk
                                 loop for at most that many tokens (fewer launches, chunk rows
                                 chosen for whole waves of GEMM tiles).  A batch holding more sets
                                 RLK_DERR_POLICY_BOUND.  Must be >= 0. */
} rlk_batch_t;

typedef struct {
  float eps_low;        /* clip range [1 - eps_low, 1 + eps_high]; symmetric when equal */
  float eps_high;
  float adv_eps;        /* epsilon added to sigma_q; the paper leaves it unstated: 1e-6 */
  float entropy_coef;   /* coefficient of an entropy bonus in the objective (0 = off) */
  int32_t agg;          /* RLK_AGG_* */
  int32_t accumulate_dW;/* 0: dW is overwritten; 1: the gradient is added to dW */
  double norm_override; /* > 0: replaces Q (SEQ) or the policy-token count (TOKEN) so that
                           micro-batched calls add up to the one-call gradient */
  int64_t chunk_rows;   /* policy tokens per backward chunk, multiple of 256, at most
                           RLK_MAX_CHUNK_ROWS; 0 = auto: the largest multiple of 256, at most
                           65,536, whose chunk buffers fit 40 GiB (4 GiB for rlk_logprob_fwd),
                           then, with max_policy_tokens, the fewest chunks covering the bound */
  /* Token-level truncated importance sampling (Sec. 3.2.4): with rollout_logp (device [N] f32,
   * the inference engine's log-prob of each sampled token) the loss of token t is scaled by
   * w_t = min(exp(old_logp[t] - rollout_logp[t]), tis_cap), held constant in the gradient.
   * NULL = off (w_t = 1); tis_cap must then be 0, else finite and > 0. */
  const float* rollout_logp;
  /* KL term of the GRPO objective (Sec. 2.3.2): objective -= kl_coef * D_KL(pi_theta || pi_ref)
   * per token, estimated at the sampled token as r - log r - 1 with r = pi_ref / pi_theta from
   * ref_logp (device [N] f32, the reference policy's log-prob of each sampled token).
   * kl_coef = 0: off (ref_logp unused); kl_coef > 0 needs ref_logp. */
  const float* ref_logp;
  float tis_cap;
  float kl_coef;
  /* PPO (Sec. 2.3.1): device [N] f32 per-token advantages (e.g. from rlk_gae) used in place of
   * the group advantages; NULL = group advantages (GRPO).  Rewards and group ids still define
   * exclusion and the SEQ aggregation. */
  const float* token_adv;
  /* Optional host-known count of the trained tokens whose rollout advantage is not 0 (the tokens
   * that go through the backward when the loss has no entropy term, KL term or per-token
   * advantages; see rlk_pg_loss_fwd_bwd), with max_policy_tokens > 0: the chunk loop then puts a
   * chunk boundary at that count rounded up to a multiple of 256, so the backward runs on
   * well-filled chunks.  0 = unknown.  It only plans the chunks: any value gives the same results,
   * and the workspace size depends on it (query rlk_workspace_size with the same params).
   * Must be >= 0. */
  int64_t grad_tokens;
} rlk_pg_params_t;

typedef struct {
  float loss;             /* = *loss */
  float pg_loss;          /* loss without the entropy term */
  float entropy_mean;     /* token mean of H over policy tokens */
  float clip_frac;        /* fraction of policy tokens whose surrogate is clipped */
  float ratio_mean;       /* token mean of rho */
  int32_t n_groups;       /* Q */
  int32_t n_valid_rollouts;
  int64_t n_policy_tokens;/* N_eff */
  float kl_mean;          /* token mean of the sampled-token KL estimate (0 when off) */
  float tis_mean;         /* token mean of the importance weight w_t (1 when off) */
  int32_t n_chunks;       /* chunk iterations of the call */
  int32_t n_dz_chunks;    /* chunks whose logit gradient dz was formed explicitly (see
                           * rlk_pg_loss_fwd_bwd); the others applied dz = diag(s) q in the GEMMs */
  int64_t n_grad_tokens;  /* policy tokens that went through the backward GEMMs: N_eff, less the
                           * tokens of rollouts whose advantage is exactly 0 when the loss has no
                           * other term (see rlk_pg_loss_fwd_bwd) */
} rlk_pg_stats_t;

/* Workspace bytes needed by rlk_logprob_fwd (p == NULL) or by rlk_pg_loss_fwd_bwd (p
 * != NULL) for this batch.  Host pointers; cu_seqlens is not read.  The workspace must
 * be 256-byte aligned.  Returns RLK_ESHAPE for unsupported sizes. */
rlk_status_t rlk_workspace_size(const rlk_batch_t* b, const rlk_pg_params_t* p, size_t* bytes);

/* Workspace bytes needed by rlk_group_advantage for R rollouts. */
rlk_status_t rlk_advantage_workspace_size(int32_t R, size_t* bytes);

/* pi_old / pi_theta log-prob forward (Sec. 3.2.4: the trainer's own forward pass).
 * For every row t with mask[t] = 1: logp[t] = log softmax(W h_t)[targets[t]],
 * entropy[t] = H(softmax(W h_t)) in nats, lse[t] = logsumexp(W h_t).  Rows with
 * mask 0 are written as 0.  entropy and lse may be NULL.  The logits are never stored:
 * the log-softmax is taken online over vocabulary tiles. */
rlk_status_t rlk_logprob_fwd(const rlk_batch_t* b, const void* hidden, const void* W,
                             const int32_t* targets, const uint8_t* mask, float* logp,
                             float* entropy, float* lse, void* ws, size_t ws_bytes,
                             void* stream);

/* Policy-token compaction and rollout segmentation (Sec. 2.3.1 mask; Sec. 3.2.3 per-rollout
 * token count; Sec. 3.4 exclusion).  idx [N]: ascending positions t with mask[t] = 1 inside
 * rollouts whose group id is >= 0 (group_ids NULL: no rollout is excluded), valid in its first
 * *n_eff entries; tok_rollout [N]: the rollout of each such position; n_pol [R]: number of
 * kept positions per rollout (0 for excluded rollouts); n_eff: device int32[1].  targets
 * (optional) are checked on kept rows and flag RLK_DERR_TARGET.  Uses the workspace of
 * rlk_logprob_fwd.  These are the gather lists through which every later operand is read. */
rlk_status_t rlk_compact(const rlk_batch_t* b, const uint8_t* mask, const int32_t* group_ids,
                         const int32_t* targets, int32_t* idx, int32_t* tok_rollout, int32_t* n_pol,
                         int32_t* n_eff, void* ws, size_t ws_bytes, void* stream);

/* Group-relative advantage (Sec. 2.3.2; tree GRPO, Sec. 3.2.3; task-harness groups,
 * Sec. 3.3; exclusion, Sec. 3.4).  adv[r] = (R_r - mu_q)/(sigma_q + adv_eps) with mu, sigma
 * the mean and population std of the non-excluded rewards of r's group; exactly 0 when
 * every reward of the group is bitwise equal (including groups of one) and for excluded
 * rollouts.  group_index[r] (optional) = rank of r's key among the sorted distinct
 * non-negative keys, -1 if excluded; n_groups (optional, device int32[1]) = Q.
 * Supports R <= 16384. */
rlk_status_t rlk_group_advantage(int32_t R, const float* rewards, const int32_t* group_ids,
                                 float adv_eps, float* adv, int32_t* group_index,
                                 int32_t* n_groups, void* ws, size_t ws_bytes, void* stream);

/* rlk_group_advantage without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments, computation and results; the workspace is a fixed device array inside the library of
 * the size rlk_group_advantage needs for 16384 rollouts (590,336 bytes), one copy per device, held
 * by each GPU the library runs on until the process ends.  R above 16384 returns RLK_ESHAPE before
 * anything is launched; `stream` must belong to the current device (RLK_EINVAL otherwise).  Nothing
 * is allocated: no hipMalloc, hipFree or allocating library call.  Every call on one GPU uses that
 * GPU's array, so calls that overlap on one GPU (other streams or host threads) race: the caller
 * serialises them.  No part of the array has to start at zero (the first launch resets the status
 * word, later ones write every entry they read). */
rlk_status_t rlk_group_advantage_noalloc(int32_t R, const float* rewards, const int32_t* group_ids,
                                         float adv_eps, float* adv, int32_t* group_index,
                                         int32_t* n_groups, void* stream);

/* Masked clipped policy-gradient loss, forward and backward (Sec. 2.3.1-2.3.2,
 * Sec. 3.2.3, Sec. 3.3, Sec. 3.4), with the log-prob forward inside.
 *   loss      device float[1]: L = -objective under p->agg.
 *   dhidden   [N, d] batch dtype: dL/dhidden; rows that are not trained are exactly 0.
 *   dW        [V, d] fp32: dL/dW, overwritten or accumulated (p->accumulate_dW).
 *   logp_out, entropy_out  [N] fp32 or NULL: per-token log-prob / entropy of the
 *             current policy on trained rows, 0 elsewhere.
 *   stats     device rlk_pg_stats_t or NULL.
 * old_logp [N] fp32 is read on trained rows only.  With no trainable token the loss is 0,
 * dhidden is 0 and an overwritten dW is 0.
 * The logit gradient is dz_tj = g_t ([j = y_t] - p_tj) (plus the entropy term when
 * entropy_coef != 0).  For bf16 without an entropy term the stored probabilities are taken
 * against each token's target logit, which makes dz = diag(s) q with q the stored values (target
 * entry adjusted), so the dhidden and dW GEMMs apply the row scale s and dz is never written; a
 * chunk holding a token with a target far below its largest logits (log-prob below about -40)
 * forms dz explicitly instead, with the same result.  stats->n_dz_chunks counts those chunks.
 * Without an entropy term, a KL term or per-token advantages, the surrogate gradient of a rollout
 * whose advantage is exactly 0 (every rollout of an all-equal group) is exactly 0: its tokens get
 * the forward (log-prob, entropy, loss, stats) but skip the backward GEMMs, and their dhidden rows
 * are written as 0; stats->n_grad_tokens counts the tokens that went through the backward. */
rlk_status_t rlk_pg_loss_fwd_bwd(const rlk_batch_t* b, const void* hidden, const void* W,
                                 const int32_t* targets, const uint8_t* mask,
                                 const float* old_logp, const float* rewards,
                                 const int32_t* group_ids, const rlk_pg_params_t* p,
                                 float* loss, void* dhidden, float* dW, float* logp_out,
                                 float* entropy_out, rlk_pg_stats_t* stats, void* ws,
                                 size_t ws_bytes, void* stream);

/* Masked generalised advantage estimation (Sec. 2.3.1 GAE equation; Sec. 3.2.3: the rollout's
 * terminal reward arrives at its final token, gamma = lambda = 1 giving A_t = R_i - V(s_t)).
 * Per rollout r (rows cu_seqlens[r] .. cu_seqlens[r+1] - 1 of the packed batch, one trajectory):
 * over its policy rows (mask 1) in order, delta_t = gamma V[next] - V[t] with next the following
 * policy row of the rollout, or rewards[r] - V[t] at the last one; adv[t] = sum_l (gamma
 * lam)^l delta_{t+l}; returns[t] = adv[t] + V[t].  Tool rows (mask 0) are stepped over and
 * written as 0, as are the rows of excluded rollouts (group_ids[r] < 0; group_ids may be NULL).
 * Device pointers: mask [N], values [N] f32, rewards [R] f32, adv and returns [N] f32 (returns
 * may be NULL).  cu_seqlens [R+1] device; entries are clamped to [0, N] (no error is raised).
 * Uses no workspace. */
rlk_status_t rlk_gae(int64_t N, int32_t R, const int32_t* cu_seqlens, const uint8_t* mask,
                     const float* values, const float* rewards, const int32_t* group_ids, float gamma,
                     float lam, float* adv, float* returns, void* stream);

/* Masked mean-squared value loss (Sec. 2.3.1): loss = mean over the policy rows of non-excluded
 * rollouts of (values[t] - returns[t])^2 (0 when there is none); dvalues[t] = dloss/dvalues[t]
 * = 2 (values[t] - returns[t]) / count on those rows, 0 elsewhere (dvalues may be NULL).
 * Device pointers as in rlk_gae; loss device float[1].  ws: rlk_value_workspace_size bytes,
 * 256-byte aligned, deterministic reduction (per-rollout fp64 partial sums). */
rlk_status_t rlk_value_workspace_size(int32_t R, size_t* bytes);
rlk_status_t rlk_value_loss(int64_t N, int32_t R, const int32_t* cu_seqlens, const uint8_t* mask,
                            const float* values, const float* returns, const int32_t* group_ids, float* loss,
                            float* dvalues, void* ws, size_t ws_bytes, void* stream);

/* Linear value head for the PPO critic (Sec. 2.3.1: GAE needs V(s_t); the paper leaves the
 * critic's form open, and with a critic sharing the policy's trunk it is a linear head on the
 * final hidden state): values[t] = w_v . hidden[t] + b_v on the policy rows (mask = 1, or every
 * row when mask is NULL) of non-excluded rollouts, 0 on the other rows.  hidden [N, d] and w_v [d]
 * in the batch dtype (V is not read), values device f32 [N].  Reductions in a fixed order.
 * Uses no workspace. */
rlk_status_t rlk_value_head_fwd(const rlk_batch_t* b, const void* hidden, const void* w_v, float b_v,
                                const uint8_t* mask, const int32_t* group_ids, float* values, void* stream);

/* Its backward for dvalues [N] f32 (e.g. from rlk_value_loss): on the rows rlk_value_head_fwd
 * computes, dhidden[t] = dvalues[t] w_v, added to dhidden when accumulate = 1 (other rows then
 * untouched) and written otherwise (other rows then set to 0); dhidden may be NULL (skipped).
 * dw_v [d] f32 = sum_t dvalues[t] hidden[t] and db_v [1] f32 = sum_t dvalues[t] over those rows,
 * from per-256-row partial sums added in row order (deterministic).  ws:
 * rlk_value_head_workspace_size bytes, 256-byte aligned. */
rlk_status_t rlk_value_head_workspace_size(const rlk_batch_t* b, size_t* bytes);
rlk_status_t rlk_value_head_bwd(const rlk_batch_t* b, const void* hidden, const void* w_v, const uint8_t* mask,
                                const int32_t* group_ids, const float* dvalues, void* dhidden, int32_t accumulate,
                                float* dw_v, float* db_v, void* ws, size_t ws_bytes, void* stream);

/* Prefix-tree packing of each rollout's model calls (Sec. 3.2.1; the trainable-token rule of
 * Sec. 3.2.3).  Host code, host pointers; no GPU involved.
 * Calls of rollout r are call_off[r] .. call_off[r+1]-1, in capture order; call c has the input
 * context x_tok[x_off[c] .. x_off[c+1]) and the model response y_tok[y_off[c] .. y_off[c+1]).
 * Tree: rooted at the first call's context (the task prompt); each call attaches to the node
 * whose accumulated history is the longest prefix of its context (ties: the earliest node) and
 * adds a node holding the intervening harness tokens (not trainable) followed by its response
 * (trainable); a node identical to an existing sibling is that sibling.  A context extending no
 * node's history starts another tree of the rollout.
 * Packing: per rollout, nodes depth-first (children in first-seen order).  Positions carry the
 * token, parent (packed index of the previous token on the root path, -1 at a tree's first token)
 * and depth (index on that path), for the trunk's tree attention and position ids.  Rows, one per
 * position with a parent: src = parent (the hidden state that predicts the token), target = the
 * token, mask = 1 for response tokens; row_cu [R+1] segments the rows by rollout and is the
 * cu_seqlens of the batch the loss entry points take (hidden rows gathered at src).  leaves [R]:
 * number of leaf nodes (trajectories) per rollout.  All indices are batch-global.
 * Size query: with every output pointer NULL, fills n_pos and n_rows and returns RLK_OK; with
 * outputs given, capacities below the need return RLK_ESHAPE (n_pos, n_rows still filled). */
typedef struct {
  int32_t R;
  const int64_t* call_off;  /* [R+1] */
  const int64_t* x_off;     /* [C+1], C = call_off[R] */
  const int32_t* x_tok;
  const int64_t* y_off;     /* [C+1] */
  const int32_t* y_tok;
} rlk_calls_t;

typedef struct {
  int64_t cap_pos, cap_rows;
  int32_t* token;           /* [cap_pos] */
  int32_t* parent;          /* [cap_pos] */
  int32_t* depth;           /* [cap_pos] */
  int64_t* pos_off;         /* [R+1] */
  int32_t* row_src;         /* [cap_rows] */
  int32_t* row_target;      /* [cap_rows] */
  uint8_t* row_mask;        /* [cap_rows] */
  int32_t* row_cu;          /* [R+1] */
  int32_t* leaves;          /* [R] */
  int64_t n_pos, n_rows;    /* out */
} rlk_tree_out_t;

rlk_status_t rlk_tree_pack(const rlk_calls_t* calls, rlk_tree_out_t* out);

/* Synchronises `stream`, then reads the status word that the previous calls using `ws`
 * left there.  *flags (optional host pointer) receives RLK_DERR_* bits; returns RLK_OK or
 * RLK_EDATA.  Each entry point clears the word when it starts. */
rlk_status_t rlk_check_status(const void* ws, void* stream, int32_t* flags);

const char* rlk_status_string(rlk_status_t s);
const char* rlk_last_error(void);
int32_t rlk_version(void);

/* Kernel timing for measurement.  Between rlk_profile_begin() and rlk_profile_end() every
 * kernel launch of the entry points above is bracketed by a pair of HIP events on the
 * call's stream.  rlk_profile_begin() creates the events beforehand (a pool of 8192, reused by
 * later windows; more are created only if a window records more), so the launches inside the
 * window allocate nothing.  rlk_profile_end() waits for them and fills, per kernel kind
 * k < *n_kinds (host arrays of length max_kinds), the summed milliseconds and the launch count. */
rlk_status_t rlk_profile_begin(void);
rlk_status_t rlk_profile_end(int32_t max_kinds, double* total_ms, int32_t* launches,
                             int32_t* n_kinds);
const char* rlk_kernel_kind_name(int32_t kind);

#ifdef __cplusplus
}
#endif

#endif /* RLK_H */
