/*
 * sao.h -- C ABI of the SAO per-token training-loss pass on AMD MI355X (gfx950).
 *
 * The pass is the loss side of single-rollout asynchronous RL with direct
 * double-sided importance sampling (DIS): per-token log-probs of the LM head,
 * skip-observation GAE advantages, the DIS ratio against the rollout engine's
 * log-probs with a strict two-sided token mask, a token-level mean, and the
 * backward into the hidden states and the head weights. Next to it are the
 * objectives and estimators the paper compares DIS and the critic with (the
 * clipped PPO surrogate and its decoupled form, step-level GAE, GRPO's group
 * normalisation, a running-mean baseline) and the critic's explained variance.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.   Every array argument is a DEVICE pointer owned by the caller. The
 *           library never allocates or frees caller-visible memory. Its only
 *           mutable host state is per calling thread (the last error message and
 *           the measurement hooks sao_debug_time_kernel and
 *           sao_debug_clock_samples), plus, per device, the
 *           address of sao_clipped_loss_noalloc's static scratch. Scratch space is the caller's `ws` buffer of
 *           `ws_bytes` bytes (device memory, 256-byte aligned), at least
 *           sao_workspace_size(...) bytes; its contents on entry are ignored.
 * Streams.  All work is enqueued on `stream` (a hipStream_t; NULL = the null
 *           stream). Calls return before the device finishes and never
 *           synchronise. Calls on one stream are ordered; the caller orders
 *           calls on different streams. The library is reentrant.
 * Layouts.  Token-major, row-major. `hidden` is T rows of H elements with row
 *           stride `ld_hidden` elements; `w_head` is V rows of H elements with
 *           row stride `ld_w`. Strides must be >= H and multiples of 8, H must
 *           be a multiple of 8, and the two bases 16-byte aligned. A row stride may
 *           span at most 2^24 bytes (8,388,608 bf16 or 4,194,304 fp32 elements). Per-token
 *           arrays are dense, length T, aligned so that hidden[t] predicts
 *           target[t] and logp_rollout[t], values[t], rewards[t], mask[t]
 *           describe the same action a_t.
 * Dtypes.   SAO_BF16: hidden/w_head/dhidden are bfloat16 (bit patterns, 2 bytes),
 *           products accumulate in fp32. SAO_F32: they are float32.
 * Masks.    mask[t] = 1 marks a model-generated action token (the loss mask);
 *           0 marks prompt/observation tokens.
 * Errors.   Anything checkable on the host is returned synchronously before any
 *           work is enqueued: SAO_ERR_NULL (required pointer NULL), SAO_ERR_SHAPE
 *           (negative size, H or V < 1, bad stride/alignment, B < 1),
 *           SAO_ERR_VALUE (epsilon negative or non-finite, gamma or lambda
 *           outside [0,1], alpha negative or non-finite), SAO_ERR_DTYPE, SAO_ERR_WORKSPACE
 *           (ws too small or misaligned), SAO_ERR_DEVICE (a HIP launch failed).
 *           sao_last_error_message() gives a thread-local detail string.
 *           T == 0 is a no-op that returns SAO_OK.
 *           Data errors visible only on the device (a target outside [0,V),
 *           cu_seqlens not non-decreasing or not ending at T, a non-finite
 *           log-sum-exp, a running-mean key out of range) OR bits into the
 *           optional device word `*status`
 *           (SAO_STATUS_*) without a host synchronisation; the affected outputs
 *           are NaN rather than silently valid.
 * Accumulation.  Outputs documented as "+=" accumulate so that chunked calls sum
 *           to the whole batch; the caller zeroes them. The explained-variance
 *           moments and the running-mean history are in/out states that a call
 *           combines with or advances. All other outputs are overwritten.
 *
 * Citations name sections and equations of "Single-Rollout Asynchronous
 * Optimization for Agentic Reinforcement Learning" (arXiv 2607.07508).
 */
#ifndef SAO_H
#define SAO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

typedef enum {
  SAO_OK = 0,
  SAO_ERR_NULL = 1,
  SAO_ERR_SHAPE = 2,
  SAO_ERR_VALUE = 3,
  SAO_ERR_DTYPE = 4,
  SAO_ERR_WORKSPACE = 5,
  SAO_ERR_DEVICE = 6
} sao_status_t;

typedef enum { SAO_BF16 = 0, SAO_F32 = 1 } sao_dtype_t;

typedef enum {
  SAO_OP_LOGPROB = 0,
  SAO_OP_ADVANTAGE = 1,
  SAO_OP_LOSS = 2,
  SAO_OP_BACKWARD = 3,
  SAO_OP_VALUE = 4,
  SAO_OP_PPO_LOSS = 5,
  SAO_OP_EXPLAINED_VARIANCE = 6,
  SAO_OP_STEP_ADVANTAGE = 7,
  SAO_OP_GROUP_ADVANTAGE = 8,
  SAO_OP_RUNNING_MEAN_ADVANTAGE = 9
} sao_op_t;

/* Step value of sao_step_advantage (App. A.1). */
typedef enum {
  SAO_STEP_AVERAGE = 0,  /* mean of the step's token values            */
  SAO_STEP_LAST = 1      /* value of the step's last token              */
} sao_step_value_t;

/* Bits of the optional device status word. */
#define SAO_STATUS_TARGET_RANGE 1  /* a loss-mask token's target is outside [0, V)   */
#define SAO_STATUS_SEGMENTS     2  /* cu_seqlens is not non-decreasing from 0 to T    */
#define SAO_STATUS_NONFINITE    4  /* a log-sum-exp came out NaN or infinite          */
#define SAO_STATUS_KEY_RANGE    8  /* a running-mean key is outside [0, n_keys)        */

/* Per-token flags written by sao_clipped_loss (sao_ppo_loss: see there). */
#define SAO_FLAG_MASKED    0  /* mask == 0                                       */
#define SAO_FLAG_USED      1  /* max(0, 1 - eps_low) < rho < 1 + eps_high         */
#define SAO_FLAG_LOW       2  /* rho <= max(0, 1 - eps_low)                       */
#define SAO_FLAG_HIGH      3  /* rho >= 1 + eps_high                              */
#define SAO_FLAG_NONFINITE 4  /* rho is NaN                                       */

const char* sao_status_string(sao_status_t status);
const char* sao_last_error_message(void);
/* Library version as "major.minor.patch". */
const char* sao_version(void);

/* Bytes of `ws` that `op` needs for T tokens, hidden size H and vocabulary V
 * (0 if none). Returns 0 for invalid arguments as well. The backward's share is
 * dominated by one vocabulary block of the logit gradient, round_up(T, 256) x Vb
 * elements of the hidden dtype. Vb comes from a target Vt = 32768 rows, doubled
 * (up to 65536) while (round_up(T, 256) / 256) x (Vt / 256) < 8192: V is cut into
 * n = ceil(V / Vt) blocks of b = ceil(ceil(V / n) / 256) tiles of 256 rows. When
 * n > 1, b is then rounded up to a multiple m of 256 / gcd(256, ceil(H / 256)) if
 * that stays within Vt / 256 tiles and 256 x b x H elements fit in 256 MiB, and
 * otherwise rounded down to a multiple of m if b >= m. Vb = 256 b (32768 rows for
 * V = 151936, H = 2048 bf16 at T = 65536; 24576 for V = 151552, H = 6144 at
 * T = 32768). */
size_t sao_workspace_size(sao_op_t op, int64_t T, int64_t H, int64_t V, sao_dtype_t dtype);

/*
 * Per-token log-probabilities of the current policy, Sec. 3.1, Eq. (1)-(2):
 *   z_{t,v} = hidden[t] . w_head[v],  lse[t] = log sum_v exp(z_{t,v}),
 *   logp[t] = z_{t,target[t]} - lse[t]            (temperature 1, full vocabulary).
 * Rows with mask[t] == 0 are skipped and get logp = lse = 0; mask == NULL means
 * every row. The T x V logits never reach memory: each tile of logits is reduced
 * to a running (max, sum of exponentials) per token inside the kernel.
 * Outputs: logp[T], lse[T] float32 (overwritten). lse is the input of
 * sao_loss_backward.
 */
sao_status_t sao_token_logprob(const void* hidden, int64_t ld_hidden, const void* w_head,
                               int64_t ld_w, const int32_t* target, const uint8_t* mask,
                               int64_t T, int64_t H, int64_t V, sao_dtype_t dtype, float* logp,
                               float* lse, int32_t* status, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Skip-observation token-level GAE, Sec. 3.2, Eq. (4)-(5), over B packed
 * trajectories; trajectory b is tokens [cu_seqlens[b], cu_seqlens[b+1]).
 * For its action tokens tau_0 < ... < tau_{n-1} (mask 1), with tau_n = end:
 *   r~_k    = sum of rewards[tau_k .. tau_{k+1}-1]   (observation rewards fold into
 *             the preceding action; rewards before the first action are dropped)
 *   delta_k = r~_k + gamma * values[tau_{k+1}] - values[tau_k]   (0 after the last action)
 *   adv[tau_k] = delta_k + gamma * lambda_b * adv[tau_{k+1}]
 *   ret[tau_k] = r~_k + gamma * ret[tau_{k+1}]                   (critic lambda = 1)
 * lambda_b = max(0, 1 - 1/(alpha * L_b)) with L_b the trajectory's token count
 * when alpha > 0 (length-adaptive GAE, Sec. 4.1); alpha == 0 selects the fixed
 * `lam` (alpha < 0 is SAO_ERR_VALUE).
 * Arithmetic is float64 inside; adv/ret are float32, 0 where mask == 0
 * (overwritten). n_tokens (nullable, device int64) receives sum(mask), the
 * token-mean denominator N of sao_clipped_loss (overwritten).
 * values, rewards, mask are [T]; cu_seqlens is int32 [B+1]. If cu_seqlens does
 * not rise from 0 to T without decreasing, every adv/ret is NaN and the status
 * word gets SAO_STATUS_SEGMENTS. ws: sao_workspace_size(SAO_OP_ADVANTAGE, ...) bytes.
 */
sao_status_t sao_advantage(const float* values, const float* rewards, const uint8_t* mask,
                           const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma,
                           double lam, double alpha, float* adv, float* ret, int64_t* n_tokens,
                           int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Step-level GAE, App. A.1: one advantage per agentic step instead of per token.
 * A step is a maximal run of tokens with mask 1 inside a trajectory (one model
 * turn). For trajectory b with steps [a_0, z_0) ... [a_{n-1}, z_{n-1}) and a_n = end:
 *   V_i   = mean of values[a_i .. z_i)   (SAO_STEP_AVERAGE)  or  values[z_i - 1]  (SAO_STEP_LAST)
 *   R_i   = sum of rewards[a_i .. a_{i+1})   (observation rewards fold into the step
 *           before them; rewards before the first step are dropped)
 *   delta_i = R_i + gamma * V_{i+1} - V_i    (V_n = 0)
 *   A_i   = delta_i + gamma * lambda_b * A_{i+1},  G_i = R_i + gamma * G_{i+1}   (critic lambda = 1)
 * lambda_b = max(0, 1 - 1/(alpha * n)) with n the trajectory's number of steps when
 * alpha > 0, else (alpha == 0) `lam`; alpha < 0 is SAO_ERR_VALUE. Every token of
 * step i gets adv = A_i and ret = G_i; tokens with mask 0 get 0 (overwritten). last (nullable, uint8 [T], overwritten) is 1 on
 * each step's final token: the critic's loss mask in the last-token form.
 * n_tokens, status, the segment checks and their NaN outputs follow sao_advantage.
 * Arithmetic is float64 inside; reductions run in a fixed order.
 * ws: sao_workspace_size(SAO_OP_STEP_ADVANTAGE, T, 1, 1, SAO_F32) bytes (24 per token).
 */
sao_status_t sao_step_advantage(const float* values, const float* rewards, const uint8_t* mask,
                                const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma,
                                double lam, double alpha, sao_step_value_t step_value, float* adv,
                                float* ret, uint8_t* last, int64_t* n_tokens, int32_t* status,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * GRPO's group-normalised advantage, the critic-free baseline of Sec. 2.
 * Trajectories [g*group_size, (g+1)*group_size) answer one prompt (B must be a
 * multiple of group_size). With R_b the sum of trajectory b's rewards:
 *   mu_g = mean of the group's R,  sigma_g = sqrt(population variance + eps_stab),
 *   traj_adv[b] = (R_b - mu_g) / sigma_g      (eps_stab = 0 and equal rewards: NaN)
 *   adv[t] = traj_adv[b] on trajectory b's tokens with mask 1, else 0 (overwritten)
 * traj_reward[B] and traj_adv[B] are float64 outputs (required). n_tokens,
 * status and the segment checks follow sao_advantage (malformed segments: NaN
 * everywhere). ws: sao_workspace_size(SAO_OP_GROUP_ADVANTAGE, T, 1, 1, SAO_F32).
 */
sao_status_t sao_group_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens,
                                 int32_t B, int64_t T, int32_t group_size, double eps_stab,
                                 float* adv, double* traj_reward, double* traj_adv,
                                 int64_t* n_tokens, int32_t* status, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * Running-mean reward baseline: the 8 most recent rewards of each prompt in the
 * Sec. 4.3 ablation, the 128 most recent in the Sec. 4.5 online comparison.
 * Trajectories arrive in batch order; trajectory b has key keys[b] in [0, n_keys)
 * (its prompt; keys == NULL puts every trajectory under key 0). With R_b the sum
 * of trajectory b's rewards:
 *   traj_adv[b] = R_b - mean of the `window` most recent earlier rewards of its key
 *                 (the history, then earlier trajectories of this batch; the
 *                 trajectory's own reward excluded; an empty window gives 0)
 *   adv[t]      = traj_adv[b] on trajectory b's tokens with mask 1, else 0
 * history (float64 [n_keys][window], in/out) is a ring per key: the reward pushed
 * as the key's j-th (from 0) sits at slot j mod window; seen (int64 [n_keys],
 * in/out) counts the rewards pushed per key. Zero both before the first batch.
 * This call pushes the batch's rewards after computing the baselines. A key
 * outside [0, n_keys) sets SAO_STATUS_KEY_RANGE, gives that trajectory NaN and
 * pushes nothing for it. traj_reward and traj_adv are float64 [B] outputs
 * (required); n_tokens, status and the segment checks follow sao_advantage
 * (malformed segments: NaN outputs, history untouched). With keys, finding a
 * trajectory's earlier same-key trajectories scans the batch, so the work grows
 * as B^2 / 64 per call (negligible for batches of rollouts, B in the hundreds).
 * ws: sao_workspace_size(SAO_OP_RUNNING_MEAN_ADVANTAGE, T, 1, 1, SAO_F32) bytes.
 */
sao_status_t sao_running_mean_advantage(const float* rewards, const uint8_t* mask,
                                        const int32_t* cu_seqlens, int32_t B, int64_t T,
                                        const int32_t* keys, int32_t n_keys, int32_t window,
                                        double* history, int64_t* seen, float* adv,
                                        double* traj_reward, double* traj_adv, int64_t* n_tokens,
                                        int32_t* status, void* ws, size_t ws_bytes,
                                        hipStream_t stream);

/*
 * Direct double-sided importance sampling and the token-level mean,
 * Sec. 3.1, Eq. (1)-(3). For each token with mask 1 (in float64):
 *   rho_t = exp(logp[t] - logp_rollout[t])                         Eq. (2)
 *   flag  = NONFINITE if rho is NaN, LOW if rho <= max(0, 1-eps_low),
 *           HIGH if rho >= 1+eps_high, else USED                   Eq. (3), strict
 *           (a ratio is never negative: with eps_low >= 1 only rho = 0, i.e.
 *           log pi = -inf or an underflowing exp, is clipped low)
 *   loss[0] += -(1/N) sum_{USED} rho_t adv_t logp_t    (minus Eq. (1))
 *   loss[1] += -(1/N) sum_{USED} rho_t adv_t           (same gradient)
 *   g[t]     = -[USED] rho_t adv_t / N                 (d loss / d logp[t]; exactly 0
 *                                                       unless USED; overwritten)
 * f(r) is treated as a stop-gradient weight. N = *n_tokens (device int64, the
 * whole batch's loss-mask count, so chunked calls share one denominator); when
 * n_tokens is NULL, N = sum(mask) of this call. N == 0 gives zero loss and g.
 * flags[T] uint8 (overwritten), counts[5] int64 (+=): {sum(mask), USED, LOW,
 * HIGH, NONFINITE}. loss[2] is float64 (+=). Reductions are deterministic.
 */
sao_status_t sao_clipped_loss(const float* logp, const float* logp_rollout, const float* adv,
                              const uint8_t* mask, int64_t T, float eps_low, float eps_high,
                              const int64_t* n_tokens, double* loss, float* g, uint8_t* flags,
                              int64_t* counts, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * sao_clipped_loss without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Same arguments, outputs, accumulation and
 * results as sao_clipped_loss (the same kernels; bit-identical outputs), minus
 * ws and ws_bytes. The kernels' scratch (per-block partials and the mask count)
 * is a static array of 114,944 bytes in device memory, one per GPU, which the
 * library obtains on its first call on each device (with that device current)
 * and holds until the process ends; no call allocates or frees anything. That
 * maximum covers every T, since the loss uses at most 2048 blocks of partials;
 * a T whose scratch would not fit is rejected with SAO_ERR_WORKSPACE. `stream`
 * must belong to the current device (else SAO_ERR_DEVICE). Every call on a GPU
 * shares that GPU's array, and each call writes every part of the scratch it
 * reads, so nothing carries over between calls; but calls that overlap on one
 * GPU (on different streams, or from different host threads without ordering)
 * race on it and must not be issued.
 */
sao_status_t sao_clipped_loss_noalloc(const float* logp, const float* logp_rollout, const float* adv,
                                      const uint8_t* mask, int64_t T, float eps_low, float eps_high,
                                      const int64_t* n_tokens, double* loss, float* g, uint8_t* flags,
                                      int64_t* counts, hipStream_t stream);

/*
 * The clipped surrogate the paper compares DIS with: the unified objective of
 * Sec. 2 with separate clip widths (eps_low == eps_high is standard PPO,
 * eps_high > eps_low is clip-higher) and, when logp_behav is given, the
 * decoupled three-policy form of Sec. 3.1. For each token with mask 1 (in float64):
 *   r_t  = exp(logp[t] - logp_old[t])
 *   w_t  = exp(logp_old[t] - logp_behav[t])          (1 when logp_behav is NULL;
 *                                                     a constant, not truncated)
 *   flag = NONFINITE if r or w is NaN; HIGH if adv > 0 and r > 1+eps_high;
 *          LOW if adv < 0 and r < 1-eps_low; else USED (unclipped)
 *   loss[0] += -(1/N) sum_t w_t min(r_t adv_t, clip(r_t, 1-eps_low, 1+eps_high) adv_t)
 *              over tokens that are not NONFINITE
 *   g[t]     = -[USED] w_t r_t adv_t / N     (d loss / d logp[t]; overwritten)
 * Strict comparisons: at r = 1+eps_high or 1-eps_low the two products agree and
 * the gradient flows. N, flags[T] (overwritten), counts[5] (+=: {sum(mask), USED,
 * LOW, HIGH, NONFINITE}, so (LOW + HIGH) / N is the clip ratio) and the
 * workspace follow sao_clipped_loss; loss[1] is float64 (+=). logp_behav is
 * nullable; every other array is required. Reductions are deterministic.
 */
sao_status_t sao_ppo_loss(const float* logp, const float* logp_old, const float* logp_behav,
                          const float* adv, const uint8_t* mask, int64_t T, float eps_low,
                          float eps_high, const int64_t* n_tokens, double* loss, float* g,
                          uint8_t* flags, int64_t* counts, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * Explained variance of the critic, Sec. 4.4, over tokens with mask 1:
 *   EV = 1 - Var(R - V) / Var(R)        (R = ret of sao_advantage, V = values)
 * moments[5] (device float64, in/out) is a running state {n, mean of R,
 * sum of squared deviations of R, mean of R - V, sum of squared deviations of
 * R - V}; this call's tokens are combined into it, so chunked calls cover the
 * whole batch (zero it before the first). ev (nullable, device float64,
 * overwritten) = 1 - moments[4] / moments[2] after the combination, NaN when
 * n == 0 or Var(R) == 0. Arithmetic is float64; the combination runs in a fixed
 * order. ws: sao_workspace_size(SAO_OP_EXPLAINED_VARIANCE, T, 1, 1, SAO_F32) bytes.
 * T == 0 leaves moments and ev untouched.
 */
sao_status_t sao_explained_variance(const float* values, const float* ret, const uint8_t* mask,
                                    int64_t T, double* moments, double* ev, void* ws,
                                    size_t ws_bytes, hipStream_t stream);

/*
 * Backward of the DIS loss through the log-softmax of Eq. (1)-(2):
 *   dz_{t,v}   = g[t] * (1[v == target[t]] - exp(z_{t,v} - lse[t]))
 *   dhidden[t] = sum_v dz_{t,v} w_head[v]      (dtype of hidden, dense [T][H]; rows with
 *                                               g == 0 are exact zeros; overwritten)
 *   dw_head[v] += sum_t dz_{t,v} hidden[t]     (float32, dense [V][H], +=)
 * g and lse come from sao_clipped_loss and sao_token_logprob. Rows with g == 0
 * cost no work. Logits are recomputed on the fly; their gradient is staged in
 * `ws` one vocabulary block at a time (see sao_workspace_size).
 */
sao_status_t sao_loss_backward(const void* hidden, int64_t ld_hidden, const void* w_head,
                               int64_t ld_w, const int32_t* target, const float* lse,
                               const float* g, int64_t T, int64_t H, int64_t V, sao_dtype_t dtype,
                               void* dhidden, float* dw_head, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Critic head for the PPO-style update with a learned value model (Sec. 2): a
 * bias-free H -> 1 projection of the hidden states,
 *   v[t] = hidden[t] . w_v                        (float32 [T], overwritten)
 * w_v is H elements of `dtype`, 16-byte aligned. All T rows are computed. No
 * workspace is needed (ws may be NULL). Use v, detached, as the `values` of
 * sao_advantage.
 */
sao_status_t sao_value_forward(const void* hidden, int64_t ld_hidden, const void* w_v, int64_t T,
                               int64_t H, sao_dtype_t dtype, float* v, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Squared-error loss of the critic against the lambda = 1 returns `ret` of
 * sao_advantage (Sec. 2 and Sec. 4.1), token-level mean with the same N:
 *   loss_v[0]    += (1/N) sum_t mask[t] (v[t] - ret[t])^2        (float64, +=)
 *   dv_t          = 2 mask[t] (v[t] - ret[t]) / N
 *   dhidden_v[t]  = dv_t w_v          (dtype of hidden, dense [T][H]; rows with
 *                                      mask 0 are exact zeros; overwritten)
 *   dw_v         += sum_t dv_t hidden[t]                          (float32 [H], +=)
 * N = *n_tokens (device int64) or, when n_tokens is NULL, sum(mask) of this
 * call; N == 0 adds nothing and writes zero rows. No gradient flows through the
 * advantages. Reductions are deterministic. Workspace:
 * sao_workspace_size(SAO_OP_VALUE, T, H, 1, dtype).
 */
sao_status_t sao_value_loss(const void* hidden, int64_t ld_hidden, const void* w_v, const float* v,
                            const float* ret, const uint8_t* mask, int64_t T, int64_t H,
                            const int64_t* n_tokens, sao_dtype_t dtype, double* loss_v,
                            void* dhidden_v, float* dw_v, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * Measurement hook, not part of the pass. For the calling thread, records the
 * caller's HIP events `start_event` and `stop_event` (hipEvent_t, created by
 * the caller with timing enabled) on the launch stream immediately before and
 * after the next launches of kernel `kernel`; SAO_KERNEL_NONE (or NULL events)
 * disables it. Each launch re-records the same pair, so the pair brackets the
 * most recent launch. The library never creates, waits on or destroys these
 * events.
 */
#define SAO_KERNEL_NONE         0
#define SAO_KERNEL_HEAD_FORWARD 1  /* the MFMA head-forward kernel of sao_token_logprob */
#define SAO_KERNEL_BACKWARD_DZ  2  /* sao_loss_backward's logit recompute (dz), first vocabulary block */
#define SAO_KERNEL_BACKWARD_DH  3  /* its dH += dz . W product, first vocabulary block */
#define SAO_KERNEL_BACKWARD_DW  4  /* its dW += dz^T . H product, first vocabulary block */
void sao_debug_time_kernel(int kernel, void* start_event, void* stop_event);

/*
 * Measurement hook, not part of the pass. For the calling thread, makes the next
 * launches of kernel `kernel` (one of the SAO_KERNEL_* above; the backward ones
 * on their first vocabulary block) record, for each workgroup b < slots, eight
 * int64 values in the caller's device buffer `records` (8 * slots int64): the
 * hardware ids of its first wave (XCC_ID << 32 | HW_ID), its start and end on the
 * device's constant-rate wall clock (s_memrealtime), the shader clock (s_memtime)
 * at its start, after its prologue, after its K loop and at its end, and its
 * tile (M tile << 32 | N tile of the product, -1 for none; for the head forward
 * the vocabulary tile and the token tile). Workgroup b is blockIdx.x plus
 * blockIdx.y times the grid's x size. At up to 8192 tokens the head forward and
 * the backward's logit recompute run one launch (per vocabulary block) of a fixed
 * grid of workgroups that each take many tiles, the partial last vocabulary tile's
 * included; there the records are per tile instead, tile (v, t) of the launch's
 * vocabulary range in slot b = v x ceil(T / 256) + t, and the launch clears all
 * slots first. Summed cycles over summed wall-clock time give the
 * clock the kernel ran at. SAO_KERNEL_NONE, NULL or slots <= 0 disables it. Each
 * launch overwrites the records of the previous one.
 */
void sao_debug_clock_samples(int kernel, void* records, int64_t slots);

#ifdef __cplusplus
}
#endif
#endif /* SAO_H */
