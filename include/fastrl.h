/*
 * fastrl.h -- C ABI of the MI355X (gfx950) hot path of a FastRL GRPO step.
 *
 * The method is "Learn from the Gap: Differential-Aware Advantage Pruning with
 * Adaptive Rollout Sampling for GRPO" (arXiv 2609.36932).  One step of the hot path
 * evaluates the kept rollouts only:
 *   fastrl_advantage            group-normalised advantage        (Sec. 3.2, Eq. advantage)
 *   fastrl_prune(_ex)           MDAP pruning + keep budget + compaction of kept tokens
 *                                                                 (Sec. 3.2; Alg. 1 Phase 2)
 *   fastrl_token_logprob        LM-head log-prob of the sampled tokens
 *                                                                 (Sec. 3.2, post-pruning evaluation)
 *   fastrl_policy_loss_fwd_bwd  GRPO/DAPO/GSPO clipped loss, backward to dhidden and dW
 *                                                                 (Sec. 3.1, Eq. 1, Eq. grad)
 *   fastrl_adamw_step           AdamW update of W consuming dW    (Sec. 4.1; Alg. 1 update)
 *   fastrl_ars_*                adaptive rollout sampling, host only (Sec. 3.3; Alg. 1 Phase 1)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every array argument is a DEVICE pointer owned by the caller unless its
 *   name ends in _host.  The library never allocates or frees device memory; calls
 *   that need scratch space take a caller-owned workspace (ws, ws_bytes) whose
 *   minimum size is returned by the matching *_workspace_size() query (a workspace
 *   must be 256-byte aligned).  Outputs must not alias inputs.
 * Layout.  Matrices are row-major and dense: hidden[rows][d], W[V][d], dW[V][d],
 *   dhidden[T][d].  Rows are d elements apart.
 * Streams.  Work is enqueued on `stream` (0 = the null stream) and is asynchronous;
 *   a kernel fault surfaces at the caller's next synchronisation.  No call
 *   synchronises the device except where stated (none does).
 * Errors.  Every int-returning function returns 0 (FASTRL_OK) or a negative
 *   fastrl_status.  Arguments are validated on the host first; on a host-side error
 *   nothing is enqueued and fastrl_last_error() (thread-local) holds a message.
 *   Data-dependent faults found by kernels (a token id outside [0, V), offsets that
 *   are not monotone, a group larger than the promised maximum, a non-finite reward)
 *   set bits of the optional device word `status` (bitwise OR, FASTRL_SB_*), and the
 *   offending item is skipped; the caller must zero `status` before the call.
 * Threading.  Calls are reentrant; the only global state is the thread-local error
 *   text and the optional kernel-timing recorder (fastrl_profile_*).
 * dtypes.  hidden and W share one dtype: FASTRL_F32 (float) or FASTRL_BF16
 *   (bfloat16 bits, 2 bytes); accumulation is always float32.
 */
#ifndef FASTRL_H
#define FASTRL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

typedef enum fastrl_status {
  FASTRL_OK = 0,
  FASTRL_ERR_NULL_PTR = -1,     /* a required pointer is NULL */
  FASTRL_ERR_SHAPE = -2,        /* a size is negative, zero where forbidden, or too large */
  FASTRL_ERR_VALUE = -3,        /* a scalar parameter is out of its documented range */
  FASTRL_ERR_DTYPE = -4,        /* unknown dtype enum */
  FASTRL_ERR_WORKSPACE = -5,    /* workspace NULL, misaligned or smaller than required */
  FASTRL_ERR_HIP = -6,          /* a HIP runtime call failed (message has the HIP error) */
  FASTRL_ERR_UNSUPPORTED = -7   /* valid request outside what the library implements */
} fastrl_status;

/* device status word bits (OR-ed by kernels) */
#define FASTRL_SB_BAD_OFFSETS   0x1   /* group_off / traj_tok_off / seq_off not monotone or out of range */
#define FASTRL_SB_BAD_TOKEN     0x2   /* a token id outside [0, V) */
#define FASTRL_SB_GROUP_TOO_BIG 0x4   /* a question has more rollouts than max_group */
#define FASTRL_SB_SEQ_TOO_LONG  0x8   /* a trajectory is longer than max_len */
#define FASTRL_SB_BAD_REWARD    0x10  /* a non-finite reward */
#define FASTRL_SB_BAD_INDEX     0x20  /* row_index / seq_index entry out of range */
#define FASTRL_SB_SHIFT_REDO    0x40  /* informational: some logits were re-evaluated with a
                                         per-token shift because exp(z) left float range */
#define FASTRL_SB_BAD_GRAD      0x80  /* a non-finite gradient entry reached the optimizer */
#define FASTRL_SB_FILL_SHORT    0x100 /* DP alignment: too few unselected trajectories to reach
                                         a multiple of dp_align */
#define FASTRL_SB_SYNC_TIMEOUT  0x200 /* a GEMM block's wavefronts did not meet within the bounded
                                         wait of its stage hand-over (results not reliable) */

typedef enum fastrl_dtype { FASTRL_F32 = 0, FASTRL_BF16 = 1 } fastrl_dtype;
typedef enum fastrl_algo { FASTRL_GRPO = 0, FASTRL_DAPO = 1, FASTRL_GSPO = 2 } fastrl_algo;
typedef enum fastrl_norm {
  FASTRL_NORM_SEQ_MEAN_TOKEN_MEAN = 0, /* w_t = 1 / (S * L_i): Eq. 1 with G -> kept sequences */
  FASTRL_NORM_TOKEN_MEAN = 1           /* w_t = 1 / T over all kept tokens (DAPO token level)  */
} fastrl_norm;

/* Thread-local text of the last host-side error of this thread ("" if none). */
const char* fastrl_last_error(void);
/* Library ABI version: major * 10000 + minor * 100 + patch. */
int fastrl_version(void);

/* ------------------------------------------------------------------------------------
 * fastrl_advantage -- Sec. 3.2, Eq. (advantage): A_i = (r_i - mean r) / (std r + eps) over
 * the G_q rollouts of question q, std with `std_ddof` degrees of freedom (1 = sample std).
 * Also the advantage classes of Eq. (grouping): class_id[i] numbers the distinct reward
 * values of question q (0, 1, ... in order of first occurrence; equal rewards <=> equal
 * advantages whenever std > 0).  With drop_uniform != 0 (DAPO) a question whose rewards are
 * all equal gets group_valid[q] = 0, else 1.
 *
 *   rewards     [N] float, device.      group_off [Q+1] int32, device, group_off[0] = 0,
 *   adv         [N] float out.          monotone, group_off[Q] = N; question q owns
 *   class_id    [N] int32 out.          trajectories group_off[q] .. group_off[q+1]-1.
 *   group_valid [Q] uint8 out.
 *   Q >= 0, N >= 0; std_ddof in {0, 1}; eps >= 0.  Sums are taken in float64.
 * ------------------------------------------------------------------------------------ */
int fastrl_advantage(const float* rewards, const int32_t* group_off, int32_t Q, int32_t N,
                     int32_t std_ddof, float eps, int32_t drop_uniform, float* adv,
                     int32_t* class_id, uint8_t* group_valid, int32_t* status,
                     hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * fastrl_prune -- Maximizing Differential Advantage Pruning (Sec. 3.2; Alg. 1 Phase 2),
 * an optional keep-ratio budget, and stream compaction of the kept tokens.
 *
 * MDAP, per question and per advantage class, traverses the class members in ascending
 * index and keeps o_i unless an already-kept member o_j has token n-gram Jaccard distance
 * theta_ij = 1 - |N_n(o_i) & N_n(o_j)| / |N_n(o_i) | N_n(o_j)| < tau (strict; N_n = set of
 * distinct contiguous n-grams; theta = 0 when both sets are empty).  tau = tau_num / tau_den
 * and the test is exact integer arithmetic.  mdap_count[q] = |S(q)| (the count ARS uses).
 *
 * Budget (keep_ratio > 0; not part of the paper): K_q = clamp(floor(keep_ratio*G_q + 0.5),
 * 1, G_q) trajectories are kept: classes are ordered by |G_q r_k - sum_j r_j| descending
 * (sum in index order, float64; ties by first member), and a round-robin over the ordered
 * classes takes first the MDAP-kept members, then the MDAP-pruned ones, each in ascending
 * index.  keep_ratio == 0 keeps exactly the MDAP set.  Invalid questions keep nothing.
 *
 * Compaction: kept trajectories in ascending index -> kept_traj[0..N_kept), their token
 * offsets kept_tok_off[0..N_kept] (exclusive scan of lengths) and, for every kept token t,
 * its source token index tok_src[t].  counts[0] = N_kept, counts[1] = T_kept (device;
 * the caller reads them to size the next launches -- the step's one device->host sync).
 *
 *   token_ids [T_total] int32 in [0, V);  traj_tok_off [N+1] int64 (trajectory i owns
 *   tokens traj_tok_off[i] .. traj_tok_off[i+1]-1);  rewards [N];  group_off [Q+1];
 *   class_id [N] (from fastrl_advantage);  group_valid [Q] or NULL (all valid).
 *   max_group >= every G_q (<= 256); max_len >= every trajectory length (<= 16384);
 *   V in [1, 2^21); ngram_n in {1, 2, 3}; tau_num >= 0, tau_den > 0; keep_ratio in [0, 1].
 *   Outputs: keep_mask [N] uint8 (0/1), mdap_count [Q] int32, kept_traj [N] (first N_kept
 *   valid), kept_tok_off [N+1] (first N_kept+1 valid), tok_src [T_total] (first T_kept
 *   valid), counts [2] int64.  T_total < 2^31.
 * ------------------------------------------------------------------------------------ */
size_t fastrl_prune_workspace_size(int32_t Q, int32_t N, int64_t T_total, int32_t max_group,
                                   int32_t ngram_n);
int fastrl_prune(const int32_t* token_ids, const int64_t* traj_tok_off, int64_t T_total,
                 const float* rewards, const int32_t* group_off, const int32_t* class_id,
                 const uint8_t* group_valid, int32_t Q, int32_t N, int32_t max_group,
                 int32_t max_len, int32_t V, int32_t ngram_n, int32_t tau_num,
                 int32_t tau_den, double keep_ratio, uint8_t* keep_mask,
                 int32_t* mdap_count, int32_t* kept_traj, int64_t* kept_tok_off,
                 int32_t* tok_src, int64_t* counts, int32_t* status, void* ws,
                 size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * fastrl_prune_ex -- fastrl_prune with the paper's variants of the advantage partition.
 *
 * Fields up to `ws_bytes` mean what the fastrl_prune arguments of the same name mean, and
 * the workspace is fastrl_prune_workspace_size().  Added:
 *   adv        [N] float, device, or NULL: the advantages fastrl_advantage wrote.  When
 *              given, the members of each class are traversed by |A| descending, ties by
 *              ascending index (Alg. 1 Phase 2 order); inside a class of bit-equal rewards
 *              that is the ascending index order of fastrl_prune.  The budget follows the
 *              same order: a class's kappa uses its first visited member's reward, classes
 *              tie on their lowest member index, and each round takes a class's next member
 *              in visiting order.
 *   group_eps  0: classes are class_id (bit-equal rewards, Eq. grouping).  > 0: continuous
 *              rewards (appendix on the grounding task, eps = 1e-4 there): the classes of a
 *              question are the connected components of |A_i - A_j| < group_eps over its
 *              adv values (float32 read as float64, gaps in float64), numbered 0, 1, ... by
 *              lowest member index.  class_id is then ignored and may be NULL; adv is required.
 *              Non-finite adv values are treated as 0 and set FASTRL_SB_BAD_REWARD.
 *   class_out  [N] int32, device, or NULL: the class id each trajectory was pruned under.
 *   dp_align   0 or 1: off.  d > 1 (<= 4096): Alg. 1's alignment to d data-parallel ranks,
 *              after MDAP and the budget: while the kept count is not a multiple of d, the
 *              unselected trajectory with the highest |A| is added, round-robin over the
 *              valid questions in index order (one per question per round, |A| descending,
 *              ties by index).  Needs adv.  If too few unselected trajectories are left, all
 *              of them are added and FASTRL_SB_FILL_SHORT is set.  mdap_count is the MDAP
 *              count before the fill (what ARS observes).
 * fastrl_prune_args_size() returns sizeof(fastrl_prune_args) for binding checks.
 * Errors as fastrl_prune; group_eps must be finite and >= 0 (FASTRL_ERR_VALUE).
 * ------------------------------------------------------------------------------------ */
typedef struct fastrl_prune_args {
  const int32_t* token_ids;
  const int64_t* traj_tok_off;
  int64_t T_total;
  const float* rewards;
  const int32_t* group_off;
  const int32_t* class_id;
  const uint8_t* group_valid;
  int32_t Q, N, max_group, max_len, V, ngram_n, tau_num, tau_den;
  double keep_ratio;
  uint8_t* keep_mask;
  int32_t* mdap_count;
  int32_t* kept_traj;
  int64_t* kept_tok_off;
  int32_t* tok_src;
  int64_t* counts;
  int32_t* status;
  void* ws;
  size_t ws_bytes;
  const float* adv;
  double group_eps;
  int32_t* class_out;
  int32_t dp_align;
} fastrl_prune_args;
size_t fastrl_prune_args_size(void);
int fastrl_prune_ex(const fastrl_prune_args* args, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * fastrl_token_logprob -- Sec. 3.2 (post-pruning evaluation): logits of the kept tokens
 * z[t, v] = hidden[r_t] . W[v], r_t = row_index ? row_index[t] : t, and
 *   lse[t]  = log sum_v exp(z[t, v])       (vocab-chunked online max / sum-exp)
 *   logp[t] = z[t, y_t] - lse[t],          y_t = token_ids[r_t]
 * The [T, V] logits are never stored.  hidden row r is the final hidden state whose LM-head
 * output scores token_ids[r].  d % 8 == 0, V >= 1, T >= 0; lse may be NULL.  hidden and W
 * are read in 16-byte pieces: both must be 16-byte aligned (FASTRL_ERR_VALUE otherwise).
 * ------------------------------------------------------------------------------------ */
size_t fastrl_token_logprob_workspace_size(int64_t T, int32_t d, int32_t V, int32_t dtype);
int fastrl_token_logprob(const void* hidden, const int32_t* row_index, const void* W,
                         int32_t dtype, int64_t T, int32_t d, int32_t V,
                         const int32_t* token_ids, float* logp, float* lse,
                         int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * fastrl_token_logprob_noalloc -- fastrl_token_logprob for callers that cannot allocate
 * device memory or pass a workspace (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): same arguments, results and errors (results are bit
 * for bit those of fastrl_token_logprob), without ws / ws_bytes.  It calls no allocating
 * routine; its scratch is a fixed device array of fastrl_token_logprob_noalloc_scratch_bytes()
 * (64 MiB) that every GPU the library runs on holds from its first use until the process
 * ends.  The tokens run in chunks of fastrl_token_logprob_noalloc_max_chunk(V) (14080 at
 * V = 152064); a V for which not even 256 tokens fit gives FASTRL_ERR_SHAPE (V above ~8.38M).
 * `stream` must belong to the current device (FASTRL_ERR_VALUE otherwise).  All calls on one
 * GPU share its array: calls that overlap on one GPU (other streams, other threads) race and
 * must be serialised by the caller.  The first call on a device looks the array's address
 * up (hipGetSymbolAddress) with that device current.
 * ------------------------------------------------------------------------------------ */
int fastrl_token_logprob_noalloc(const void* hidden, const int32_t* row_index, const void* W,
                                 int32_t dtype, int64_t T, int32_t d, int32_t V,
                                 const int32_t* token_ids, float* logp, float* lse,
                                 int32_t* status, hipStream_t stream);
size_t fastrl_token_logprob_noalloc_scratch_bytes(void);
int64_t fastrl_token_logprob_noalloc_max_chunk(int32_t V);

/* ------------------------------------------------------------------------------------
 * fastrl_policy_loss_fwd_bwd -- Sec. 3.1: the clipped surrogate of Eq. (1) (loss = -J),
 * its per-token coefficient g_t = dL/dlogp_t (Eq. grad; clipping indicator with inclusive
 * edges), and the LM-head backward dZ = g (onehot(y) - softmax(z)), dhidden = dZ W,
 * dW = dZ^T hidden, for T kept tokens grouped in S kept sequences.
 *
 * With x = logp, o = old_logp, f = ref_logp, rho = exp(x - o), A = advantage of the token's
 * sequence, w_t the normaliser weight (fastrl_norm) and W_i = sum of w_t over sequence i:
 *   GRPO / DAPO  l_t = -min(rho A, clip(rho, 1-eps_low, 1+eps_high) A) + beta k3_t,
 *                k3_t = exp(f - x) - (f - x) - 1,       loss = sum_t w_t l_t
 *   GSPO         s_i = exp(mean_{t in i}(x - o)),  l_i = -min(s_i A, clip(s_i, ..) A),
 *                loss = sum_i W_i l_i + beta sum_t w_t k3_t
 * (GRPO and DAPO differ only in the caller's eps_low / eps_high / norm choice.)
 *
 * Inputs (device unless _host): hidden / W / token_ids / old_logp / ref_logp as in
 *   fastrl_token_logprob, all read through row_index.  ref_logp may be NULL iff beta == 0.
 *   seq_off [S+1] int64 (seq_off[0] = 0, monotone, seq_off[S] = T): kept token t belongs to
 *   sequence i iff seq_off[i] <= t < seq_off[i+1]; seq_off_host is a host copy of the same
 *   array (used to cut the work into slabs of whole sequences).  adv: advantage per
 *   trajectory; sequence i uses adv[seq_index[i]] (seq_index NULL: adv[i]).
 * Outputs: loss [1] float (sum accumulated in float64); logp, lse [T] (each may be NULL);
 *   dhidden [T][d] in dhidden_dtype (NULL: not computed); dW [V][d] float32 (NULL: not
 *   computed), overwritten, or accumulated into when dW_accumulate != 0; stats [2] float
 *   (may be NULL): clipped tokens (token objectives) or tokens of clipped sequences (GSPO),
 *   and the count of logit rows re-evaluated with a shift; stats[0] / T is the clip
 *   fraction.  entropy [T] float (may be NULL): the policy entropy of each kept token,
 *   H_t = -sum_v p_v log p_v = lse_t - sum_v p_v z_v (the statistic the paper tracks during
 *   training, Sec. 4), accumulated in the same pass as the log-sum-exp (one more partial
 *   sum exp(z - s_t) z per vocabulary block).  entropy_sum [1] float (may be NULL): sum_t H_t
 *   in float64, fixed order (the mean entropy is entropy_sum / T).
 * Limits: d % 8 == 0; hidden, W and dW 16-byte aligned (FASTRL_ERR_VALUE); S >= 0;
 *   slab_tokens >= 0 (FASTRL_ERR_VALUE).
 * Slabs: the work runs in slabs of whole sequences.  slab_tokens is the target slab size
 *   (0 = 32768 tokens, whatever T is); each slab takes an even share of the tokens left
 *   (ceil(left / slab_tokens) slabs to go, recounted after every slab) and never holds more
 *   than max(1.25 slab_tokens, longest sequence) tokens.  Each slab stores exp(z - s_t)
 *   (s_t = 0, or the row max when exp(z) would leave float range) for its tokens in the
 *   workspace, with each token's label entry lowered by exp(lse_t - s_t) so that the two
 *   backward contractions over it yield the whole of dZ, one-hot term included (that term
 *   thus carries one rounding to the operand's type: at most 2^-8 |g_t| per token in bf16,
 *   as with a bf16 dlogits operand).  The [T, V] logits are never stored: the workspace holds
 *   slab * V_pad * sizeof(dtype) bytes (V_pad = V rounded up to 256; 10 GB for the default
 *   slab at V = 152064 in bf16), W^T (d * V_pad) when dhidden is wanted, and small per-token
 *   and per-(vocabulary block, token) arrays.
 * ------------------------------------------------------------------------------------ */
typedef struct fastrl_loss_args {
  const void* hidden;
  const int32_t* row_index;
  const void* W;
  int32_t dtype;
  int32_t d;
  int32_t V;
  int32_t S;
  int64_t T;
  const int32_t* token_ids;
  const float* old_logp;
  const float* ref_logp;
  const int64_t* seq_off;
  const int64_t* seq_off_host;
  const float* adv;
  const int32_t* seq_index;
  int32_t algo;
  int32_t norm;
  float eps_low;
  float eps_high;
  float beta;
  float* loss;
  float* logp;
  float* lse;
  void* dhidden;
  int32_t dhidden_dtype;
  int32_t dW_accumulate;
  float* dW;
  float* stats;
  int64_t slab_tokens;
  int32_t* status;
  void* ws;
  size_t ws_bytes;
  float* entropy;
  float* entropy_sum;
} fastrl_loss_args;

/* sizeof(fastrl_loss_args) as compiled into the library (lets bindings check layout). */
size_t fastrl_loss_args_size(void);
size_t fastrl_policy_loss_workspace_size(const fastrl_loss_args* args);
int fastrl_policy_loss_fwd_bwd(const fastrl_loss_args* args, hipStream_t stream);

/* fastrl_policy_loss_slab_plan -- the slabs fastrl_policy_loss_fwd_bwd runs for these
 * arguments (host only: reads S, T, seq_off_host and slab_tokens; validates like the call
 * itself, without the workspace).  Returns the slab count n >= 0 (0 when S == 0) or a
 * negative fastrl_status.  *max_slab_tokens (may be NULL) receives the largest slab's token
 * count; when seq_begin_host is not NULL and capacity > n, seq_begin_host[0..n] receives the
 * first sequence of each slab followed by S (with a smaller capacity nothing is written). */
int fastrl_policy_loss_slab_plan(const fastrl_loss_args* args, int32_t* seq_begin_host,
                                 int32_t capacity, int64_t* max_slab_tokens);

/* ------------------------------------------------------------------------------------
 * fastrl_adamw_step -- the policy update that consumes dW (Alg. 1, "update pi_theta"; the
 * paper trains with AdamW, lr 1e-6, weight decay 1e-2, Sec. 4.1).  Decoupled weight decay
 * with bias correction, per element, t = step (1-based), g = grad_scale * grad:
 *   theta <- theta (1 - lr wd);  m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2
 *   theta <- theta - (lr / (1 - beta1^t)) m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
 * float32 arithmetic on float32 master weights; theta, m, v are updated in place.
 *   theta, m, v [n] float, device, 16-byte aligned (m = v = 0 before the first step);
 *   grad [n] float, device, 16-byte aligned (e.g. dW from fastrl_policy_loss_fwd_bwd, after
 *   any data-parallel reduction); w_bf16 [n] bfloat16 or NULL, 8-byte aligned: receives
 *   round-to-nearest-even(theta) for the bf16 LM-head kernels.  n >= 0, step >= 1,
 *   lr >= 0, 0 <= beta1, beta2 < 1, eps >= 0, weight_decay >= 0, all finite.
 * A non-finite g sets FASTRL_SB_BAD_GRAD in status (the update still runs, as in the usual
 * optimizers, and propagates the value).  No workspace.
 * ------------------------------------------------------------------------------------ */
int fastrl_adamw_step(float* theta, uint16_t* w_bf16, const float* grad, float* m, float* v,
                      int64_t n, int64_t step, float lr, float beta1, float beta2, float eps,
                      float weight_decay, float grad_scale, int32_t* status,
                      hipStream_t stream);

/* ------------------------------------------------------------------------------------
 * Adaptive Rollout Sampling (Sec. 3.3; Alg. 1 Phase 1(a)/(b)).  Host-only, plain data:
 * the struct may be copied to checkpoint and restore the controller.
 *   fastrl_ars_init     G1 >= 2 initial rollouts, total_steps M >= 1, steps_per_epoch >= 1.
 *   fastrl_ars_next_n   Phase 1(a): n = max(round(min(G - (G'_ref - G'_t), G)), 2) when
 *                       G'_t < G'_ref (both set), else G.  round = half to even.
 *   fastrl_ars_observe  Phase 1(b) for one step: counts_host[q] = |S(q)| for the Q questions
 *                       (valid_host[q] == 0 skips q; NULL = all).  Appends mean and max;
 *                       at an epoch end sets alpha = step / M,
 *                       G'_t = alpha mean(B_mean) + (1 - alpha) mean(B_max), G'_ref once
 *                       (first epoch) = (mean(B_mean) + mean(B_max)) / 2, resets buffers.
 * NaN in G_ref / G_t means "not set".
 * ------------------------------------------------------------------------------------ */
typedef struct fastrl_ars_state {
  int32_t G;
  int32_t pad_;
  int64_t total_steps;
  int64_t steps_per_epoch;
  int64_t step;
  double G_ref;
  double G_t;
  double sum_mean;   /* running sum of the epoch buffer B_mean */
  double sum_max;    /* running sum of the epoch buffer B_max  */
  int64_t n_buf;     /* entries in the epoch buffers            */
} fastrl_ars_state;

int fastrl_ars_init(fastrl_ars_state* st, int32_t G1, int64_t total_steps,
                    int64_t steps_per_epoch);
int32_t fastrl_ars_next_n(const fastrl_ars_state* st);
int fastrl_ars_observe(fastrl_ars_state* st, const int32_t* counts_host,
                       const uint8_t* valid_host, int32_t Q);

/* ------------------------------------------------------------------------------------
 * Kernel timing (for benchmarks).  While enabled, every launch of the dominant kernels is
 * bracketed by HIP events on the launch stream; fastrl_profile_read synchronises those
 * events and returns the summed duration (ms), the launch count and the algorithmic
 * FLOPs of the launches of one kernel kind.  Off by default.  The recorder is one
 * process-wide list behind a lock: launches from every thread and stream are summed.
 * ------------------------------------------------------------------------------------ */
typedef enum fastrl_kernel_kind {
  FASTRL_K_LOGITS_FWD = 0,  /* logits GEMM + online log-sum-exp epilogue        */
  FASTRL_K_DHIDDEN = 1,     /* dhidden = dZ W GEMM                               */
  FASTRL_K_DW = 2,          /* dW = dZ^T hidden GEMM                             */
  FASTRL_K_BACKWARD = 3,    /* dhidden and dW GEMMs of one slab in one launch
                               (bf16 with both gradients asked for)              */
  FASTRL_K_COUNT = 4
} fastrl_kernel_kind;

int fastrl_profile_enable(int32_t on);
int fastrl_profile_reset(void);
int fastrl_profile_read(int32_t kind, double* total_ms, int64_t* launches, double* flops);

#ifdef __cplusplus
}
#endif
#endif /* FASTRL_H */
