/* libdart — the trainer-side hot path of DART's policy update on MI355X (gfx950).
 *
 * Paper: "Efficient Multi-turn RL for GUI Agents via Decoupled Training and
 * Adaptive Data Curation" (DART), arXiv 2509.23866.
 *
 * The path maps the policy's vocabulary logits for every action token of a
 * step group (all steps of the N rollouts of one task, Sec. 3.3) to:
 *   1. per-token log-prob of the generated token and entropy   dart_tok_stats
 *   2. per-step mean entropy and the high-entropy step mask     dart_step_select
 *   3. the truncated-importance-sampling-weighted clipped
 *      policy-gradient loss and its gradient w.r.t. the logits  dart_tis_loss_fwd_bwd
 *
 * Conventions shared by every call
 * --------------------------------
 * - Array arguments are DEVICE pointers unless a comment says otherwise. The
 *   caller owns every buffer; the library allocates no memory and keeps no
 *   state between calls, so concurrent calls on different streams are safe
 *   (dart_tis_loss_fwd_bwd_noalloc, which has a fixed scratch array per
 *   device, says how its calls may overlap).
 * - Every call is asynchronous on `stream` (0 = the null stream): it checks its
 *   scalar arguments on the host, enqueues its kernels and returns. Outputs are
 *   valid once the stream is synchronised. Device data (target ids in range,
 *   strictly increasing offsets with the documented ends, 0/1 step masks) is a
 *   precondition and is not checked, unless the environment has DART_CHECK=1:
 *   then every call first validates the device arrays it reads, waits for the
 *   result (the call synchronises the stream, so this is a debugging mode: on
 *   a stream that is being captured into a graph every call returns
 *   DART_ERR_UNSUPPORTED) and returns DART_ERR_INVALID_ARG, with nothing of
 *   the call enqueued, on a violation.
 * - Logits are row-major [T, ld] with ld >= V (elements, not bytes). Rows whose
 *   start is 16-byte aligned (base aligned and ld * element size a multiple of
 *   16) take the vectorised path; other rows are still correct, only slower.
 * - Status codes: DART_OK; DART_ERR_INVALID_ARG for a bad scalar argument or a
 *   null required pointer (nothing is enqueued); DART_ERR_UNSUPPORTED, with
 *   nothing enqueued, for sizes beyond what a launch can hold (a dispatch holds
 *   at most 2^32 - 1 work-items): more than 67,108,863 steps (selection),
 *   4,194,303 groups (per-group selection) or 16,777,215 groups (GRPO
 *   advantage), more than 8,388,607 tiles of 256 x 256 logits or 268,435,455
 *   rows (LM head); DART_ERR_HIP when HIP reports a launch error. No call
 *   aborts or throws. The token statistics take any T up to INT32_MAX (rows
 *   are launched 2^22 at a time).
 * - Results are deterministic: no atomics on any floating-point result, fixed
 *   reduction orders; identical rows at identical alignment give bit-identical
 *   entropies.
 */
#ifndef DART_H
#define DART_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DART_OK = 0,
    DART_ERR_INVALID_ARG = 1,
    DART_ERR_UNSUPPORTED = 2,
    DART_ERR_HIP = 3
} dart_status_t;

typedef enum { DART_F32 = 0, DART_BF16 = 1 } dart_dtype_t;

/* Token statistics (Sec. 4.3, definition of the token entropy H_{t,i} and of
 * p = pi_theta(v | ...); Eq. (1), log pi_theta of the generated token).
 *
 * For every row t of `logits` ([T, ld], dtype `dtype`, first V columns used):
 *   lse[t]     = log sum_v exp(z_tv)                        (natural log)
 *   logp[t]    = z_{t, target[t]} - lse[t]
 *   entropy[t] = -sum_v p_tv log p_tv,  p_tv = exp(z_tv - lse[t])   (nats, >= 0)
 * computed in one streaming pass in float32 (online max / normaliser /
 * entropy). logp stays accurate when p_target is close to 1.
 *   target:  [T] int32, 0 <= target[t] < V (precondition).
 *   logp, entropy, lse: [T] float32 outputs.
 * Errors: INVALID_ARG if a pointer is null, T < 1, V < 1, ld < V or dtype is
 * unknown. Finite logits are required; -inf entries are allowed (probability
 * 0) as long as each row has a finite entry; NaN gives undefined results. */
dart_status_t dart_tok_stats(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                             int64_t ld, const int32_t* target, float* logp, float* entropy,
                             float* lse, hipStream_t stream);

/* Step entropy and high-entropy step selection (Sec. 4.3: the step entropy is
 * the mean token entropy over the step's thought and action tokens; only the
 * top-rho fraction of steps of the group by step entropy is trained, rho = 0.8
 * in the paper; the indicator of Eq. (2)).
 *   entropy:       [T] float32 token entropies (from dart_tok_stats).
 *   step_offsets:  [S+1] int32, step s = tokens [off[s], off[s+1]),
 *                  0 = off[0] < off[1] < ... < off[S] = T (precondition).
 *   rho:           kept fraction in [0, 1]; k = dart_kept_steps(S, rho) steps are kept.
 *   step_entropy:  [S] float32 output, the mean (summed in float64, rounded once).
 *   step_mask:     [S] uint8 output, 1 = kept. Exactly k ones: the k largest
 *                  step entropies, ties broken towards the lower step index.
 *   n_kept_steps:  [1] int32 output (k), may be NULL.
 * Errors: INVALID_ARG if a required pointer is null, T < 1, S < 1, S > T or
 * rho is outside [0, 1] or NaN. */
dart_status_t dart_step_select(const float* entropy, int64_t T, const int32_t* step_offsets,
                               int64_t S, double rho, float* step_entropy, uint8_t* step_mask,
                               int32_t* n_kept_steps, hipStream_t stream);

/* TIS-weighted clipped policy-gradient loss and its gradient w.r.t. the logits
 * (Eq. (2) without the KL term; the truncated importance weight of Sec. 4.4;
 * the clipped ratio of Eq. (1) with the asymmetric bounds of Appendix A.4).
 *
 * Per token t of step s(t), with M = step_mask[s(t)] and N = number of tokens
 * in kept steps:
 *   r = exp(logp - logp_old),  w = min(exp(logp_old - logp_rollout), C)
 *   u = r A,  c = clip(r, 1 - eps_low, 1 + eps_high) A
 *   loss      = -(1/N) sum_t M w min(u, c)                 (token mean over kept tokens)
 *   tok_coef  = dloss/dlogp_t = -(M w A r / N) if u <= c else 0
 *   dlogits   = tok_coef_t * (onehot(target_t) - softmax(z_t))
 * w, M and N are constants of the differentiation; N = 0 gives loss 0 and a
 * zero gradient.
 *   logits, dtype, T, V, ld, target: as for dart_tok_stats.
 *   logp, lse:   [T] float32 from dart_tok_stats on the same logits.
 *   logp_old, logp_rollout, adv: [T] float32 (old trainer policy, rollout
 *                policy log-probs of the targets; per-token advantages).
 *   step_offsets, S: as for dart_step_select; step_mask: [S] uint8 (0/1).
 *   eps_low, eps_high: clip bounds >= 0; C > 0 (may be +INFINITY: no truncation).
 *   dlogits:     [T, ld_out] output of dtype `dtype` (bf16 rounded to nearest
 *                even). It may be the logits buffer itself (in place) when
 *                ld_out == ld; any other overlap with logits is rejected.
 *   loss:        [1] float64 output (summed in float64 in a fixed order).
 *   tok_coef:    [T] float32 output (required: it carries the coefficient from
 *                the loss kernel to the gradient kernel).
 *   stats:       [4] float32 output or NULL: clip fraction, mean TIS weight,
 *                fraction of weights at the cap, N (all over kept tokens).
 *   workspace, workspace_bytes: device memory owned by the caller, or NULL.
 *                With a workspace of at least dart_tis_loss_workspace_bytes(T)
 *                bytes (8-byte aligned; contents on entry do not matter) the
 *                loss runs on many workgroups that leave partial sums there,
 *                added in a fixed order by a second kernel. With NULL one
 *                workgroup computes it (no workspace; slower beyond ~8k
 *                tokens). Calls that share a workspace must be ordered (one
 *                stream); the library allocates nothing.
 * Errors: INVALID_ARG for a null required pointer, T < 1, V < 1, ld < V,
 * ld_out < V, S < 1, S > T, eps < 0 or NaN, C <= 0 or NaN, an unknown dtype,
 * a partial overlap of dlogits with logits, or a workspace that is too small
 * or misaligned; HIP when a launch fails. */
dart_status_t dart_tis_loss_fwd_bwd(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                                    int64_t ld, const int32_t* target, const float* logp,
                                    const float* lse, const float* logp_old,
                                    const float* logp_rollout, const float* adv,
                                    const int32_t* step_offsets, int64_t S,
                                    const uint8_t* step_mask, float eps_low, float eps_high,
                                    float C, void* dlogits, int64_t ld_out, double* loss,
                                    float* tok_coef, float* stats, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace the loss kernels use for T tokens (at most 41,000; 0 for
 * T < 1 or T > INT32_MAX). Host only. */
size_t dart_tis_loss_workspace_bytes(int64_t T);

/* dart_tis_loss_fwd_bwd for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation, checks, kernels and results, bit for bit,
 * with the loss workspace taken from a fixed array in the library's device
 * memory instead of a caller argument. The call allocates nothing and calls
 * no allocating routine.
 *   Arguments: as for dart_tis_loss_fwd_bwd, without workspace and
 *              workspace_bytes. The caller still owns every input and output.
 *   Scratch:   40,976 bytes per GPU (the largest loss workspace), held
 *              from the first call on that GPU until the process ends; it
 *              covers every T the call accepts (T <= INT32_MAX), and its
 *              contents on entry do not matter.
 *   Races:     every call on one GPU uses that GPU's one array, so calls that
 *              may run at the same time on one GPU (two streams, two host
 *              threads) race and give undefined results: order them on one
 *              stream, or use dart_tis_loss_fwd_bwd with a workspace each.
 * Errors: those of dart_tis_loss_fwd_bwd; UNSUPPORTED if T needs more scratch
 * than the array holds (not reachable for T <= INT32_MAX); HIP if the array's
 * device address cannot be obtained. */
dart_status_t dart_tis_loss_fwd_bwd_noalloc(const void* logits, dart_dtype_t dtype, int64_t T,
                                            int64_t V, int64_t ld, const int32_t* target,
                                            const float* logp, const float* lse,
                                            const float* logp_old, const float* logp_rollout,
                                            const float* adv, const int32_t* step_offsets,
                                            int64_t S, const uint8_t* step_mask, float eps_low,
                                            float eps_high, float C, void* dlogits, int64_t ld_out,
                                            double* loss, float* tok_coef, float* stats,
                                            hipStream_t stream);

/* The two halves of dart_tis_loss_fwd_bwd, for callers that want the loss
 * without the gradient, or that time the two kernels separately.
 * dart_tis_loss_fwd computes loss, tok_coef and stats exactly as above (the
 * logits are not read); dart_tis_grad then writes
 *   dlogits[t, v] = tok_coef[t] * (onehot(target[t])[v] - exp(z_tv - lse[t]))
 * (Eq. (2) through the softmax derivative) from the coefficients of the first
 * half. Same argument meanings, layouts and error rules as
 * dart_tis_loss_fwd_bwd. */
dart_status_t dart_tis_loss_fwd(int64_t T, const float* logp, const float* logp_old,
                                const float* logp_rollout, const float* adv,
                                const int32_t* step_offsets, int64_t S, const uint8_t* step_mask,
                                float eps_low, float eps_high, float C, double* loss,
                                float* tok_coef, float* stats, void* workspace,
                                size_t workspace_bytes, hipStream_t stream);

dart_status_t dart_tis_grad(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                            int64_t ld, const int32_t* target, const float* logp,
                            const float* lse, const float* tok_coef, void* dlogits,
                            int64_t ld_out, hipStream_t stream);

/* dart_step_select followed by dart_tis_loss_fwd on the mask it selects: the
 * step means and top-rho selection of Sec. 4.3, then the coefficients and loss
 * of Eq. (2), in one launch of one workgroup when T <= 4096 and S <= 8192
 * (both calls' work back to back, without the kernel boundaries between them;
 * beyond ~5000 tokens the one workgroup is slower than the two calls' launches);
 * larger problems make the two calls in turn.
 *   Arguments: entropy, T, step_offsets, S, rho, step_entropy, step_mask,
 *              n_kept_steps as for dart_step_select (step_mask is an output);
 *              logp, logp_old, logp_rollout, adv, eps_low, eps_high, C, loss,
 *              tok_coef, stats, workspace, workspace_bytes as for
 *              dart_tis_loss_fwd. The workspace is used only when the problem
 *              is too large for one workgroup.
 *   Results:   step_entropy, step_mask, n_kept_steps and tok_coef equal those
 *              of the two calls bit for bit; loss and stats are the same sums
 *              in float64 in the one-workgroup order (the two calls with a
 *              workspace sum over several workgroups, so the last bits of the
 *              loss may differ).
 * Errors: the rules of both calls, all checked before anything is enqueued
 * (INVALID_ARG); HIP when a launch fails. */
dart_status_t dart_select_tis_loss_fwd(int64_t T, const float* entropy, const float* logp,
                                       const float* logp_old, const float* logp_rollout,
                                       const float* adv, const int32_t* step_offsets, int64_t S,
                                       double rho, float eps_low, float eps_high, float C,
                                       float* step_entropy, uint8_t* step_mask,
                                       int32_t* n_kept_steps, double* loss, float* tok_coef,
                                       float* stats, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/* ------------------------------------------------------------------------
 * Objective variants and options (same two passes over the logits)
 * ------------------------------------------------------------------------ */

/* KL estimator of D_KL(pi_theta || pi_ref) (the -beta D_KL term of Eq. (1) and
 * Eq. (2); beta = 0.1 in Appendix A.4; the paper does not state the estimator).
 * With delta = logp_ref - logp on the sampled token: K1 = -delta,
 * K2 = delta^2 / 2, K3 = exp(delta) - delta - 1 (the GRPO estimator). */
typedef enum { DART_KL_NONE = 0, DART_KL_K1 = 1, DART_KL_K2 = 2, DART_KL_K3 = 3 } dart_kl_t;

/* Aggregation weight om_t of a kept token: TOKEN_MEAN = 1/N (N tokens in kept
 * steps; the default), TOKEN_MEAN_ALL = 1/T, STEP_MEAN = 1/(K |s|) (mean over
 * the K kept steps of each step's token mean). */
typedef enum {
    DART_AGG_TOKEN_MEAN = 0,
    DART_AGG_TOKEN_MEAN_ALL = 1,
    DART_AGG_STEP_MEAN = 2
} dart_agg_t;

/* Importance ratio level: per token (default), or per step (Eq. (1) is written
 * for the whole action) as the geometric mean or the product of the step's
 * token ratios; the TIS weight and the advantage are then taken per step too
 * (the same mean or sum of token log-ratios; the mean advantage of the step). */
typedef enum {
    DART_RATIO_TOKEN = 0,
    DART_RATIO_STEP_GEOMEAN = 1,
    DART_RATIO_STEP_PRODUCT = 2
} dart_ratio_t;

/* Loss configuration (host memory, read during the call). */
typedef struct {
    float eps_low, eps_high; /* clip bounds, >= 0 */
    float C;                 /* TIS cap, > 0, may be +INFINITY */
    int32_t kl;              /* dart_kl_t */
    float beta;              /* KL coefficient, >= 0 (ignored for DART_KL_NONE) */
    int32_t aggregation;     /* dart_agg_t */
    int32_t ratio;           /* dart_ratio_t */
} dart_loss_config_t;

/* Gradient flag: a row whose coefficient is exactly 0 (dropped step, clipped
 * token, zero advantage) is written as zeros without reading its logits. The
 * result is the same (+0 in place of -0); HBM traffic drops by the share of
 * such rows. */
#define DART_GRAD_SKIP_ZERO_ROWS 1u

/* dart_tok_stats for softmax(inv_temp * z): inv_temp is an inverse sampling
 * temperature (1 in the paper, Appendix A.4); finite and > 0. */
dart_status_t dart_tok_stats_ex(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                                int64_t ld, const int32_t* target, float inv_temp, float* logp,
                                float* entropy, float* lse, hipStream_t stream);

/* The loss of Eq. (2) including its KL term, under the configuration above:
 *   loss = -sum_t M om_t (w o - beta kl_t),  o = min(r A, clip(r) A)
 *   tok_coef[t] = dloss/dlogp_t
 * (the KL term sits inside the step indicator and outside the TIS weight, as in
 * Eq. (2)). logp_ref: [T] float32 reference-policy log-probs of the targets,
 * required when config->kl != DART_KL_NONE, else ignored (may be NULL).
 * stats: [6] float32 or NULL: clip fraction, mean TIS weight, fraction at the
 * cap, N, mean KL, K (over kept tokens / steps). Other arguments and errors as
 * dart_tis_loss_fwd (step-level ratios run on one workgroup and leave the
 * workspace unused); also INVALID_ARG for a null config, an unknown enum value,
 * or beta < 0 / non-finite. */
dart_status_t dart_tis_loss_fwd_ex(int64_t T, const float* logp, const float* logp_old,
                                   const float* logp_rollout, const float* logp_ref,
                                   const float* adv, const int32_t* step_offsets, int64_t S,
                                   const uint8_t* step_mask, const dart_loss_config_t* config,
                                   double* loss, float* tok_coef, float* stats, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* dart_tis_grad at inverse temperature inv_temp (the same value given to
 * dart_tok_stats_ex): dlogits = inv_temp * tok_coef * (onehot - softmax(inv_temp z)).
 * flags: 0 or DART_GRAD_SKIP_ZERO_ROWS; other bits are INVALID_ARG. */
dart_status_t dart_tis_grad_ex(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                               int64_t ld, const int32_t* target, const float* logp,
                               const float* lse, const float* tok_coef, float inv_temp,
                               uint32_t flags, void* dlogits, int64_t ld_out, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Around the path: the advantage and several task groups per call
 * ------------------------------------------------------------------------ */

/* Step-wise GRPO advantage (Sec. 3.3). A task's step group D holds every step
 * of its N trajectories, each step carrying its trajectory's reward R_i; over
 * D, Rbar = mean(R) and sigma = the population standard deviation, and every
 * token of every step of trajectory i gets A = (R_i - Rbar) / sigma (0 when
 * sigma == 0, i.e. all rewards equal).
 *   reward:              [n_traj] float32, one reward per trajectory.
 *   traj_step_offsets:   [n_traj+1] int32, steps of trajectory i are
 *                        [traj_step_offsets[i], traj_step_offsets[i+1]) (ends at S).
 *   group_traj_offsets:  [G+1] int32, trajectories of group g are
 *                        [group_traj_offsets[g], group_traj_offsets[g+1]) (ends at n_traj).
 *   step_offsets:        [S+1] int32 token offsets of the steps (ends at T).
 *   adv:                 [T] float32 output (the per-token advantage the loss takes).
 *   group_mean, group_std: [G] float32 outputs or NULL.
 * Offsets are preconditions (monotone, consistent ends); malformed ones give
 * meaningless values but never an out-of-bounds access. Errors: INVALID_ARG for
 * a null required pointer, n_traj < 1, G < 1 or G > n_traj, S < 1, S > T. */
dart_status_t dart_grpo_advantage(const float* reward, int64_t n_traj,
                                  const int32_t* traj_step_offsets,
                                  const int32_t* group_traj_offsets, int64_t G,
                                  const int32_t* step_offsets, int64_t S, int64_t T, float* adv,
                                  float* group_mean, float* group_std, hipStream_t stream);

/* dart_step_select for G task groups in one call (one workgroup per group):
 * group g is steps [group_step_offsets[g], group_step_offsets[g+1]) and keeps
 * dart_kept_steps(S_g, rho) of its own steps, by the same rule (the paper selects
 * each task group on its own, Sec. 4.3). n_kept_steps: [G] int32 or NULL. Errors as
 * dart_step_select; also INVALID_ARG for a null group_step_offsets, G < 1 or
 * G > S. */
dart_status_t dart_step_select_groups(const float* entropy, int64_t T,
                                     const int32_t* step_offsets, int64_t S,
                                     const int32_t* group_step_offsets, int64_t G, double rho,
                                     float* step_entropy, uint8_t* step_mask,
                                     int32_t* n_kept_steps, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The LM head fused in: statistics without materialised logits
 * ------------------------------------------------------------------------ */

/* dart_tok_stats for the logits z = h W^T of the LM head, computed tile by tile
 * on the matrix cores and reduced to the same per-row statistics (Sec. 4.3,
 * Eq. 1) without writing the [T, V] logits anywhere. h: the final hidden
 * states of the T tokens, W: the LM-head weight of the policy.
 *   hidden:     [T, ld_h] bfloat16, row-major (row t = h_t); ld_h >= d.
 *   weight:     [V, ld_w] bfloat16, row-major (row v = W_v, torch.nn.Linear's
 *               [out_features, in_features] layout); ld_w >= d.
 *   d:          hidden size, a multiple of 8; ld_h and ld_w multiples of 8;
 *               hidden, weight and workspace 16-byte aligned.
 *   target, logp, entropy, lse: as for dart_tok_stats.
 *   workspace:  device memory of at least dart_lmhead_stats_workspace_bytes(T, V)
 *               bytes, owned by the caller (per-row partial statistics of every
 *               256-column slice of the vocabulary, T * ceil(V/256) * 16 + T * 4
 *               bytes); contents on entry do not matter.
 * z is accumulated in fp32 from the bf16 inputs. Errors: INVALID_ARG for a null
 * pointer, T < 1, V < 1, d < 8, a violated multiple-of-8 or alignment rule, or a
 * workspace that is too small; UNSUPPORTED when ceil(T/256) * ceil(V/256)
 * exceeds INT32_MAX or ld_h or ld_w exceeds 2^22; HIP when a launch fails. */
dart_status_t dart_lmhead_tok_stats(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                    const void* weight, int64_t V, int64_t ld_w,
                                    const int32_t* target, float* logp, float* entropy,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/* dart_lmhead_tok_stats for softmax(inv_temp * h W^T), as dart_tok_stats_ex
 * is for materialised logits: lse, logp and entropy are those of inv_temp * z
 * for the fp32 z (inv_temp enters the kernel's base-2 exponent and the row
 * maximum; inv_temp = 1 gives the bits of dart_lmhead_tok_stats). inv_temp:
 * finite and > 0, else INVALID_ARG. Other arguments and errors as
 * dart_lmhead_tok_stats. */
dart_status_t dart_lmhead_tok_stats_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                       const void* weight, int64_t V, int64_t ld_w,
                                       const int32_t* target, float inv_temp, float* logp,
                                       float* entropy, float* lse, void* workspace,
                                       size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace dart_lmhead_tok_stats (and _ex) needs (0 for T or V
 * outside [1, INT32_MAX]). Host only. */
size_t dart_lmhead_stats_workspace_bytes(int64_t T, int64_t V);

/* The gradient pass of the fused head, part one: dlogits of the logits
 * z = h W^T, recomputed tile by tile on the matrix cores exactly as
 * dart_lmhead_tok_stats forms them, then
 *   dlogits[t, v] = tok_coef[t] * (onehot(target[t])[v] - exp(z_tv - lse[t]))
 * (the chain rule through Eq. 1's log-softmax; the target element is
 * tok_coef[t] * -expm1(logp[t]), accurate when p_y is near 1), written in
 * bfloat16 (round to nearest even).
 *   hidden, weight, d, ld_h, ld_w, target: as for dart_lmhead_tok_stats.
 *   lse, logp:  [T] float32, the outputs of dart_lmhead_tok_stats for these rows.
 *   tok_coef:   [T] float32, dloss/dlogp_t from a loss forward (dart_tis_loss_fwd
 *               or dart_tis_loss_fwd_ex).
 *   dlogits:    [T, ld_out] bfloat16 output, row-major; ld_out >= V and a
 *               multiple of 8; 16-byte aligned. Columns [V, ld_out) are not
 *               written.
 * Errors: as for dart_lmhead_tok_stats (INVALID_ARG also for a bad ld_out or
 * dlogits alignment). */
dart_status_t dart_lmhead_dlogits(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                  const void* weight, int64_t V, int64_t ld_w,
                                  const int32_t* target, const float* lse, const float* logp,
                                  const float* tok_coef, void* dlogits, int64_t ld_out,
                                  hipStream_t stream);

/* dart_lmhead_dlogits at inverse temperature inv_temp (the value given to
 * dart_lmhead_tok_stats_ex for lse and logp):
 *   dlogits[t, v] = inv_temp * tok_coef[t] * (onehot(target[t])[v] - exp(inv_temp z_tv - lse[t]))
 * as dart_tis_grad_ex defines it for materialised logits (inv_temp = 1 gives
 * the bits of dart_lmhead_dlogits). inv_temp: finite and > 0, else
 * INVALID_ARG. Other arguments and errors as dart_lmhead_dlogits. */
dart_status_t dart_lmhead_dlogits_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                     const void* weight, int64_t V, int64_t ld_w,
                                     const int32_t* target, const float* lse, const float* logp,
                                     const float* tok_coef, float inv_temp, void* dlogits,
                                     int64_t ld_out, hipStream_t stream);

/* The gradient pass of the fused head, whole: the gradients of the loss with
 * respect to the hidden states and the LM-head weight,
 *   dhidden = dlogits W        [T, d]
 *   dweight = dlogits^T h      [V, d]
 * with dlogits as dart_lmhead_dlogits defines it. The rows are taken
 * chunk_rows at a time: the chunk's dlogits go to the workspace in bfloat16,
 * then two GEMMs on the matrix cores (bf16 inputs, fp32 accumulation and
 * output) form the chunk's rows of dhidden and add its share to dweight, so the
 * [T, V] dlogits never exist whole.
 *   dhidden:    [T, ld_dh] float32 output, row-major; ld_dh >= d.
 *   dweight:    [V, ld_dw] float32 output, row-major; ld_dw >= d; overwritten
 *               (not accumulated into).
 *   chunk_rows: rows per chunk, >= 1 (values above T are taken as T).
 *   workspace:  device memory of at least
 *               dart_lmhead_backward_workspace_bytes(min(chunk_rows, T), V)
 *               bytes, 16-byte aligned, owned by the caller; contents on entry
 *               do not matter.
 * Errors: as for dart_lmhead_dlogits, INVALID_ARG also for a null output, bad
 * ld_dh/ld_dw, chunk_rows < 1 or a workspace that is too small; UNSUPPORTED
 * for a leading dimension (ld_h, ld_w, ld_dh, ld_dw, or the dlogits block's
 * ceil8 of its vocabulary entries) above 2^22 elements, where the tiles'
 * 32-bit row offsets end; HIP when a launch fails. */
dart_status_t dart_lmhead_backward(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                   const void* weight, int64_t V, int64_t ld_w,
                                   const int32_t* target, const float* lse, const float* logp,
                                   const float* tok_coef, float* dhidden, int64_t ld_dh,
                                   float* dweight, int64_t ld_dw, int64_t chunk_rows,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace dart_lmhead_backward needs for chunks of chunk_rows rows:
 * chunk_rows * ceil8(V) * 2 (0 for arguments outside [1, INT32_MAX]). Host
 * only. */
size_t dart_lmhead_backward_workspace_bytes(int64_t chunk_rows, int64_t V);

/* Flags of dart_lmhead_backward_ex (bitwise or). */
enum { DART_LMHEAD_SKIP_ZERO_ROWS = 1u, DART_LMHEAD_BF16_GRADS = 4u };

/* dart_lmhead_backward in blocks of chunk_rows rows x chunk_cols vocabulary
 * entries, with flags, at an inverse temperature. dart_lmhead_backward(...,
 * chunk_rows, ...) is this call with inv_temp = 1, chunk_cols = V and
 * flags = 0.
 *
 * inv_temp: the value given to dart_lmhead_tok_stats_ex for lse and logp
 * (finite and > 0, else INVALID_ARG); the dlogits are
 *   inv_temp * tok_coef[t] * (onehot(target[t])[v] - exp(inv_temp z_tv - lse[t]))
 * as dart_tis_grad_ex defines them for materialised logits.
 *
 * Each block forms its dlogits (bf16, in the workspace), adds its share to
 * its rows of dhidden (summed over the vocabulary blocks) and to its entries'
 * rows of dweight (summed over the row blocks), with the GEMMs of
 * dart_lmhead_backward. Summing costs traffic: every row block reads and
 * rewrites the [V, d] dweight, every vocabulary block the [T, d] dhidden. For
 * a given workspace (chunk_rows * chunk_cols bf16) whole rows suit T >> V,
 * whole vocabulary rows (chunk_rows = T) suit T << V, such as a step group of
 * a few thousand tokens against a vocabulary of 152k, and square blocks suit
 * T ~ V.
 *
 * DART_LMHEAD_BF16_GRADS: dhidden and dweight are bfloat16 (round to nearest
 * even) instead of float32, as an autograd caller needs them for bf16
 * parameters. An output that several blocks add to is summed in float32 in the
 * workspace and rounded once at the end; an element that one block writes is
 * that GEMM's fp32 result rounded once.
 *
 * DART_LMHEAD_SKIP_ZERO_ROWS: rows t with tok_coef[t] == 0 have dlogits = 0
 * (the step mask of Sec. 4.3 drops whole steps, and a clipped ratio in
 * Eq. (2) has zero gradient), so they add nothing to dweight and their rows of
 * dhidden are 0. The call gathers the other rows (hidden rows, target, lse,
 * logp, tok_coef) into the workspace, runs the blocked backward over those
 * rows only, and scatters their dhidden rows back; the rows it skipped are set
 * to 0. The result equals the dense call's up to the order of the GEMMs'
 * fp32 sums. The kernels read the kept-row count on the device (the launches
 * cover all T rows; work past the count ends at once), so the call stays
 * asynchronous and can be captured into a HIP graph, whose replays follow the
 * coefficients the replay finds. With or without this flag the call can be
 * captured (unless DART_CHECK=1).
 *
 *   dhidden:    [T, ld_dh] output, float32, or bfloat16 with
 *               DART_LMHEAD_BF16_GRADS; ld_dh >= d.
 *   dweight:    [V, ld_dw] output, as dhidden; ld_dw >= d; overwritten.
 *   chunk_rows, chunk_cols: the block, each >= 1; values above T (or V) are
 *               taken as T (or V).
 *   flags:      a combination of the two flags; other bits are INVALID_ARG.
 *   workspace:  device memory of at least
 *               dart_lmhead_backward_ex_workspace_bytes(T, d, V, chunk_rows,
 *               chunk_cols, flags) bytes, 16-byte aligned, owned by the
 *               caller; contents on entry do not matter.
 * Other arguments: as for dart_lmhead_backward. Errors: as for
 * dart_lmhead_backward; UNSUPPORTED also when the sizes are too large for the
 * workspace arithmetic. */
dart_status_t dart_lmhead_backward_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                      const void* weight, int64_t V, int64_t ld_w,
                                      const int32_t* target, const float* lse, const float* logp,
                                      const float* tok_coef, float inv_temp, void* dhidden,
                                      int64_t ld_dh, void* dweight, int64_t ld_dw,
                                      int64_t chunk_rows, int64_t chunk_cols, uint32_t flags,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/* Bytes of workspace dart_lmhead_backward_ex needs (host only; 0 for bad
 * arguments or flags). The parts, each starting 256-byte aligned: the dlogits
 * block, R * ceil8(C) bf16 with R = min(chunk_rows, T), C = min(chunk_cols,
 * V); with DART_LMHEAD_BF16_GRADS, an fp32 accumulator of V * d when R < T and
 * one of T * d when C < V (none when rows are skipped: the compact fp32
 * dhidden rows serve); with DART_LMHEAD_SKIP_ZERO_ROWS, T compact hidden rows
 * (bf16), their fp32 dhidden, five [T] int/float arrays and a counter. With
 * chunk_cols >= V and flags = 0 the value is that of
 * dart_lmhead_backward_workspace_bytes(min(chunk_rows, T), V). */
size_t dart_lmhead_backward_ex_workspace_bytes(int64_t T, int64_t d, int64_t V,
                                               int64_t chunk_rows, int64_t chunk_cols,
                                               uint32_t flags);

/* Host helper (no device work): k = clamp(ceil(rho * S - 1e-6), 0, S), the
 * number of steps dart_step_select keeps (the guard absorbs the representation
 * error of rho: 0.8 * 240 gives 192). Returns -1 for S < 0 or rho outside
 * [0, 1]. */
int64_t dart_kept_steps(int64_t S, double rho);

/* Host helper: a static, human-readable name for a status code. */
const char* dart_status_string(dart_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* DART_H */
