/*
 * agrl.h -- C ABI of the fused policy-loss library for AMD MI355X (gfx950).
 *
 * The library computes, on one GPU, the trainer-side hot path of agentic RL
 * with GRPO and task advantage normalisation (AgentRL, arXiv 2510.04206):
 *
 *   agrl_task_adv_norm     per-trajectory action-token counts, GRPO group
 *                          advantages and task advantage normalisation
 *                          (Sec. 3.2; App. B.2 GRPO objective);
 *   agrl_policy_loss_fwd   logits H W^T by vocabulary tiles on the matrix
 *                          cores (never stored), log-softmax, the sampled
 *                          token's log-probability (App. B.1, token-level
 *                          factorisation of the action probability), ratio
 *                          against the behaviour policy and the clipped
 *                          surrogate, masked to action tokens and averaged
 *                          over them (App. B.2 PPO objective; App. A, the
 *                          DAPO objective's decoupled clip bounds and
 *                          token-level normalisation);
 *   agrl_policy_loss_bwd   dH and dW of that loss, recomputing the logits;
 *   agrl_sequence_mean_weights  per-token weights that turn the loss into the
 *                          sequence-level mean of App. B.2's GRPO objective.
 *
 * Conventions for every entry point:
 *   - Array arguments are DEVICE pointers owned by the caller; the library
 *     allocates no memory.  Scalars and `opt` are host values.  `stream` is a
 *     hipStream_t passed as void* (NULL = the null stream).
 *   - Calls only enqueue work on `stream` and return; they never synchronise.
 *     Argument errors are reported synchronously, before anything is
 *     launched, and leave every output untouched.
 *   - Row-major, contiguous.  H is [T, d]; W is [V, d] (the nn.Linear weight
 *     layout, logits = H W^T).  Row n of H is the hidden state that predicts
 *     token_id[n]; the caller shifts labels, the library never does.
 *   - Tokens with action_mask == 0 (environment observations, padding) are
 *     never read for H, token_id, adv_tok, old_logp, lse or logp.  Their
 *     outputs are logp = lse = 0 and dH row = +0.
 *   - Faults found on the device (an id out of range, more action tokens
 *     than max_act) set bits in a per-device error word; read it with
 *     agrl_get_device_error.  An action token whose token_id lies outside
 *     [0, V) poisons the call's outputs, so that a caller who does not read
 *     the word still sees the fault: that token's logp and lse are NaN, the
 *     loss is NaN, and in the backward its logit-gradient row is NaN, which
 *     makes its dH row and every row of dW NaN.  Other tokens' logp and lse
 *     are unaffected.  With more action tokens than max_act the loss is NaN
 *     and the other outputs are unspecified.
 *   - Results are deterministic: every reduction has a fixed order, no
 *     floating-point atomics are used.
 */
#ifndef AGRL_H
#define AGRL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AGRL_OK = 0,
  AGRL_E_NULL = -1,        /* a required pointer is NULL */
  AGRL_E_SHAPE = -2,       /* a size is negative, zero where it must not be, or too large */
  AGRL_E_DTYPE = -3,       /* dtype is not AGRL_BF16 or AGRL_F32 */
  AGRL_E_FLAGS = -4,       /* an option or a clip bound is out of range */
  AGRL_E_WORKSPACE = -5,   /* workspace NULL or smaller than agrl_policy_loss_workspace_size */
  AGRL_E_HIP = -6,         /* the HIP runtime reported an error (see agrl_last_error) */
  AGRL_E_UNSUPPORTED = -7  /* a valid but unimplemented configuration */
} agrl_status;

typedef enum { AGRL_BF16 = 0, AGRL_F32 = 1 } agrl_dtype;

/* Options.  A zero-initialised struct (or opt == NULL) selects the defaults. */
typedef struct {
  int32_t std_ddof;      /* 0: population std in both normalisation stages (default); 1: sample std */
  float std_eps;         /* added to each std before dividing; 0 selects 1e-6 */
  float temperature;     /* logits are (H W^T) / temperature; 0 selects 1 */
  int32_t dw_accumulate; /* 0: dW is overwritten (default); 1: dW += gradient */
  /* Bound on the backward's logit-gradient buffers for one vocabulary chunk:
   * G, roundup(max_act, 256) * Vc * 2 bytes, for AGRL_BF16 (dW reads G
   * transposed); G and G^T, twice that at 4 bytes per element, for AGRL_F32.
   * The backward walks the vocabulary in equal chunks of Vc columns (a
   * multiple of 256), as few as fit the bound; 0 selects 4 GiB.  The full
   * T x V logit gradient is held only when it fits the bound. */
  int64_t g_chunk_bytes;
  /* Optional instrumentation: NULL, or a host array of 8 hipEvent_t.  The
   * library records events[2k] on `stream` just before and events[2k+1] just
   * after its matrix-core launch k: 0 forward logits, 1 backward logit
   * recompute, 2 dW product, 3 dH product.  For AGRL_BF16 the dW and dH
   * products run as one launch, bracketed by events 4/5, and events 6/7 are
   * recorded back to back.  With several vocabulary chunks the last chunk's
   * launches are the ones bracketed. */
  void* const* phase_events;
  /* KL penalty against a reference policy (App. A: the PPO and GRPO
   * objectives subtract beta * D_KL).  Per action token, with l = logp and
   * r = ref_logp[t]: kl_estimator 0 (k3, default) KL = exp(r - l) - (r - l) - 1,
   * 1 (k1) KL = l - r.  The loss uses s - kl_beta * KL in place of the
   * surrogate s.  kl_beta = 0 disables it; otherwise ref_logp is a device
   * array of T fp32 values, read on action tokens. */
  float kl_beta;
  int32_t kl_estimator;
  const float* ref_logp;
  /* Per-token loss weights (device, T fp32, read on action tokens): the loss
   * becomes L = -sum_t w_t (s_t - kl_beta KL_t) in place of the token mean
   * -(1/N) sum_t (...), and n_norm is ignored.  Sequence-level aggregation
   * (App. B.2's GRPO form: a token mean per trajectory, then a mean over
   * trajectories) is w_t = 1 / (n_seq * n_traj(t)).  NULL: token mean. */
  const float* token_weight;
  /* agrl_task_adv_norm only: 1 drops every GRPO group whose rewards are all
   * equal (App. A, DAPO's dynamic sampling): its trajectories get advantage 0
   * and are left out of the task statistics.  Needs traj_group. */
  int32_t drop_uniform_groups;
  /* agrl_task_adv_norm only: NULL, or a device array of 2 * (n_group + n_task)
   * int32 (2 * n_task without traj_group) that the call uses as scratch.  With
   * it, the call records the lowest and the highest index of each group's and
   * each task's trajectories, and each group's and task's wave scans only that
   * index range instead of all n_traj trajectories: the stages then take work
   * proportional to the members' spans rather than n_group * n_traj and
   * n_task * n_traj (trajectories stored segment by segment make every span its
   * segment's size).  The results are bit-identical either way: the summation
   * order below does not depend on it.  Calls that overlap must not share it. */
  int32_t* adv_ranges;
} agrl_options;

/*
 * Advantage normalisation over a global batch of T_g tokens (Sec. 3.2).
 *
 *   traj_id[T_g]      int32, trajectory of each token, -1 for padding
 *   action_mask[T_g]  uint8, 1 for model-generated (action) tokens
 *   traj_task[n_traj] int32, task of each trajectory, in [0, n_task)
 *   traj_group[n_traj] int32, GRPO group (one sample's rollouts) of each
 *                     trajectory, in [0, n_group); NULL skips the group stage
 *   reward[n_traj]    fp32, one reward per trajectory
 * Outputs (all written):
 *   act_count[n_traj] int32, number of action tokens of each trajectory
 *   task_count[n_task] int64, number of action tokens of each task (N_i)
 *   task_mean, task_std [n_task] fp32, mean and std of the task's token-level
 *                     advantage set
 *   adv_traj[n_traj]  fp32, normalised advantage of each trajectory
 *   adv_tok[T_g]      fp32, adv_traj[traj_id[t]] on action tokens, 0 elsewhere
 *                     (NULL: not written)
 *
 * Group stage (App. B.2 GRPO advantage): A_hat = (R - mean_g R) / (std_g R + eps).
 * Task stage (Sec. 3.2): every action token of trajectory tau carries A_hat_tau;
 * mu_i and sigma_i are the mean and std of that token-level set of task i and
 * A_tilde = (A_hat - mu_i) / (sigma_i + eps).  A task without action tokens
 * gets mu = sigma = 0 and A_tilde = 0.
 *
 * Bit-exact fp32: every sum over a segment (a group or a task) deals its
 * terms to 64 partial sums by trajectory index mod 64, adds each partial in
 * ascending trajectory order, and combines the partials by an xor butterfly
 * (offsets 32, 16, 8, 4, 2, 1); products, quotients and the square root are
 * single correctly rounded operations.  Counts are exact integers.
 */
int agrl_task_adv_norm(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                       const int32_t* traj_id, const uint8_t* action_mask,
                       const int32_t* traj_task, const int32_t* traj_group,
                       const float* reward, const agrl_options* opt, int32_t* act_count,
                       int64_t* task_count, float* task_mean, float* task_std, float* adv_traj,
                       float* adv_tok, void* stream);

/*
 * Per-token loss weights of the sequence-level aggregation.  App. B.2 writes
 * GRPO's objective as a mean over the responses of a token mean within each
 * response; for a packed micro-batch of T tokens this is
 *   seq_count[j]    = action tokens of trajectory j in this micro-batch
 *                     (action_mask != 0 and traj_id == j), int32
 *   n_seq           = trajectories with seq_count[j] > 0
 *   token_weight[t] = fp32(1 / (n_seq * seq_count[traj_id[t]])) on action
 *                     tokens with traj_id >= 0 (the quotient is formed in
 *                     fp64 and rounded once), 0 on every other token.
 * Passed as agrl_options.token_weight to the policy-loss calls, the loss
 * becomes -(1/n_seq) sum_j (1/seq_count[j]) sum_{t in j} (...).  A trajectory
 * cut by the packing counts only its tokens in this micro-batch.
 *   traj_id[T]       int32 trajectory of each token, -1 for padding (device)
 *   action_mask[T]   uint8 (device)
 *   seq_count[n_traj]  int32, written (device)
 *   token_weight[T]  fp32, written (device)
 * A traj_id >= n_traj sets ERR bit 2 of the device error word and the token
 * is ignored.  T = 0 writes seq_count only.
 */
int agrl_sequence_mean_weights(int64_t T, int32_t n_traj, const int32_t* traj_id,
                               const uint8_t* action_mask, int32_t* seq_count,
                               float* token_weight, void* stream);

/*
 * Bytes of device workspace the forward and backward calls need for a packed
 * micro-batch of T tokens of which at most max_act are action tokens
 * (max_act <= 0 means T).  The same workspace serves both calls.  Returns 0
 * for invalid sizes.
 */
size_t agrl_policy_loss_workspace_size(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                       int32_t dtype, const agrl_options* opt);

/*
 * Vocabulary columns per backward chunk for these sizes and options (the same
 * arguments as agrl_policy_loss_workspace_size): a multiple of 256, at most
 * roundup(V, 256).  The backward recomputes the logits and forms G for
 * ceil(V / chunk) chunks in order; the last holds the remaining columns.
 * Returns 0 for invalid sizes.  Host-only; no device work.
 */
int64_t agrl_policy_loss_vocab_chunk(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                     int32_t dtype, const agrl_options* opt);

/*
 * Forward of the token-level clipped policy loss over a packed micro-batch.
 *
 *   T, d, V         tokens, hidden size (multiple of 64), vocabulary size
 *   max_act         upper bound on the number of action tokens (<= 0: T)
 *   dtype           AGRL_BF16 (bf16 inputs, fp32 accumulation on the matrix
 *                   cores) or AGRL_F32
 *   H[T, d], W[V, d]  hidden states and LM head, in `dtype`
 *   token_id[T]     int32 sampled token of each position (read on action tokens)
 *   action_mask[T]  uint8
 *   adv_tok[T]      fp32 advantage of each token (e.g. agrl_task_adv_norm's adv_tok)
 *   old_logp[T]     fp32 log-probability of token_id under the behaviour policy
 *   clip_eps_low, clip_eps_high  ratio clipped to [1 - low, 1 + high],
 *                   0 <= low < 1, high >= 0
 *   n_norm          loss divisor; <= 0 uses the number of action tokens
 * Outputs:
 *   loss[1]         L = -(1/N) sum over action tokens of min(rho A, clip(rho) A),
 *                   rho = exp(logp - old_logp); 0 when N == 0
 *   logp[T], lse[T] fp32 log-probability of token_id and log-sum-exp of the
 *                   logits on action tokens, 0 elsewhere
 *   n_clip[2]       int64 {#tokens with A > 0 and rho > 1 + high,
 *                          #tokens with A < 0 and rho < 1 - low}; NULL: skipped
 */
int agrl_policy_loss_fwd(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                         const void* H, const void* W, const int32_t* token_id,
                         const uint8_t* action_mask, const float* adv_tok,
                         const float* old_logp, float clip_eps_low, float clip_eps_high,
                         int64_t n_norm, const agrl_options* opt, void* workspace,
                         size_t ws_bytes, float* loss, float* logp, float* lse, int64_t* n_clip,
                         void* stream);

/*
 * Backward of the same loss, scaled by grad_loss (the upstream dL).
 *
 * Arguments as for the forward, plus lse[T] and logp[T] as returned by the
 * forward on the same inputs.  With g_n = dL/dlogp_n = -(grad_loss/N) A_n rho_n
 * (0 for tokens whose clipped branch is active) and p the softmax of the
 * logits, the logit gradient is G[n, v] = g_n (1[v = y_n] - p[n, v]) / temperature and
 *   dH[T, d] fp32 = G W       (+0 rows for masked tokens)
 *   dW[V, d] fp32 = G^T H     (overwritten, or added to with opt->dw_accumulate)
 * dH and dW must be 16-byte aligned (AGRL_E_UNSUPPORTED otherwise): their rows
 * are written 16 bytes per lane.
 * The logits are recomputed tile by tile; G is rounded to `dtype` (bf16 for
 * AGRL_BF16) before the two products, which accumulate in fp32.
 */
int agrl_policy_loss_bwd(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                         const void* H, const void* W, const int32_t* token_id,
                         const uint8_t* action_mask, const float* adv_tok,
                         const float* old_logp, float clip_eps_low, float clip_eps_high,
                         int64_t n_norm, const agrl_options* opt, const float* lse,
                         const float* logp, float grad_loss, void* workspace, size_t ws_bytes,
                         float* dH, float* dW, void* stream);

/*
 * Forward-only token log-probabilities over a packed batch: log pi(a_t | s_t)
 * of every action token, the factorised log-probability of an action
 * (App. B.1), as needed for the old-policy denominator of the PPO ratio
 * (App. B.2) when it is recomputed on the trainer rather than taken from the
 * rollout engine.  The same tiles, partials and merge as agrl_policy_loss_fwd,
 * so logp and lse are bit-identical to that call's on the same inputs.
 *
 *   T, max_act, d, V, dtype, H, W, token_id, action_mask, opt: as for
 *                   agrl_policy_loss_fwd (opt->temperature divides the logits)
 *   workspace       at least agrl_token_logprob_workspace_size bytes (the
 *                   policy-loss workspace also serves)
 * Outputs:
 *   logp[T], lse[T] fp32 on action tokens, 0 elsewhere
 * Errors as for agrl_policy_loss_fwd; T == 0 enqueues nothing.
 */
size_t agrl_token_logprob_workspace_size(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                         int32_t dtype, const agrl_options* opt);
int agrl_token_logprob(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                       const void* H, const void* W, const int32_t* token_id,
                       const uint8_t* action_mask, const agrl_options* opt, void* workspace,
                       size_t ws_bytes, float* logp, float* lse, void* stream);

/*
 * agrl_token_logprob without a workspace argument, for callers that cannot
 * allocate device memory around the call: code being captured into a HIP
 * graph, tight serving loops, harnesses that forbid allocation.  The same
 * kernels, outputs and errors as agrl_token_logprob; their workspace is a
 * fixed array of AGRL_NOALLOC_SCRATCH_BYTES of device memory that the library
 * holds on every GPU it runs on until the process ends.  The call allocates
 * nothing (no hipMalloc, no library routine that allocates); the caller still
 * passes the inputs and outputs.
 *   Arguments as for agrl_token_logprob, without workspace and ws_bytes.
 *   Sizes whose agrl_token_logprob_workspace_size exceeds the array are
 *   refused with AGRL_E_WORKSPACE before anything is launched.
 * Every call on one GPU uses that GPU's array, and an array keeps what the
 * last call left in it (nothing in it needs to start at zero: the kernels
 * write every value they read).  Calls that overlap on one GPU, from two
 * streams or two host threads, race on the array; serialise them.
 */
#define AGRL_NOALLOC_SCRATCH_BYTES (64ll << 20)
int agrl_token_logprob_noalloc(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                               const void* H, const void* W, const int32_t* token_id,
                               const uint8_t* action_mask, const agrl_options* opt, float* logp,
                               float* lse, void* stream);

/* Text for a status code (static storage). */
const char* agrl_status_string(int status);

/* Message of the last AGRL_E_* returned on this host thread ("" if none). */
const char* agrl_last_error(void);

/*
 * Synchronises `stream`, then reads and clears the current device's error
 * word into *code (0 = no fault; bits: 1 token id, 2 trajectory id, 4 task
 * id, 8 group id, 16 more action tokens than max_act).
 */
int agrl_get_device_error(void* stream, int32_t* code);

#ifdef __cplusplus
}
#endif

#endif /* AGRL_H */
