/*
 * ff_loss.h -- the objectives that consume a rollout (libff.so).
 *
 *   forward noising x_t = (1 - t) x_0 + t eps (Sec. 3.2)       -> ff_flow_noise
 *   Advantage Weighted Matching loss (Sec. 3.2, Eq. 3)         -> ff_awm_loss
 *   DiffusionNFT loss (Sec. 3.2, Eq. 2)                        -> ff_nft_loss
 *   clipped-ratio GRPO objective on stored trajectories
 *   (Sec. 3.1: policy gradient on the SDE log-probabilities)   -> ff_grpo_loss
 *
 * Conventions (ownership, asynchrony on `stream`, host-side validation,
 * status codes, ff_last_error) are those of ff.h.  The velocities these
 * losses read come from ff_dit_forward; the log-probabilities from
 * ff_logprob / ff_sde_step.
 *
 * Readings where the paper is silent:
 *   - time runs from t = 1 (noise) to t = 0 (data), as in the rollout; the
 *     forward-process velocity d x_t / dt = eps - x_0 is the target v of
 *     Eq. 2 and Eq. 3;
 *   - ||.||^2 is the squared L2 norm over the D elements of a sample and the
 *     expectation is the mean over the B samples of the batch;
 *   - Eq. 2's implicit positive / negative velocities v+ and v- are inputs;
 *   - the GRPO objective is the clipped ratio surrogate
 *       loss = -sum_{k,b} w_k min(r A_b, clip(r, 1 - eps_c, 1 + eps_c) A_b) / (S B),
 *       r = exp(logp_new[k, b] - logp_old[k, b]),
 *     with per-SDE-step weights w_k (a timestep reweighting such as
 *     GRPO-Guard's; NULL = unit weights).
 *
 * Sums over D are accumulated in float32 within a thread and float64 across
 * threads and blocks in a fixed order: results are bitwise reproducible.
 */
#ifndef FF_LOSS_H
#define FF_LOSS_H

#include "ff.h"

#ifdef __cplusplus
extern "C" {
#endif

/* x_t[b, :] = (1 - t[b]) x0[b, :] + t[b] eps[b, :], computed in float32 and
 * stored in `dtype`.  x0, eps, xt: device [B, D] of dtype (xt may not alias
 * x0 or eps); t: device float32 [B], each in [0, 1] (not checked on device).
 * B = 0 or D = 0 is a no-op.  Pointers 16-byte aligned. */
int ff_flow_noise(const void* x0, const void* eps, const float* t, void* xt, int64_t B, int64_t D,
                  int32_t dtype, void* stream);

/* Workspace bytes needed by ff_awm_loss / ff_nft_loss for a [B, D] batch. */
int ff_loss_workspace_size(int64_t B, int64_t D, size_t* bytes /* host, out */);

/* Eq. 3.  per_sample[b] = adv[b] * ||v[b] - (eps[b] - x0[b])||^2 (device
 * float64 [B], may be NULL), loss = mean_b per_sample[b] (device float64 [1]).
 * v, eps, x0: device [B, D] of dtype; adv: device float32 [B]. */
int ff_awm_loss(const void* v, const void* eps, const void* x0, const float* adv, int64_t B, int64_t D,
                int32_t dtype, double* per_sample, double* loss, void* workspace, size_t ws_bytes,
                void* stream);

/* Eq. 2.  per_sample[b] = r[b] ||v_pos[b] - v[b]||^2 + (1 - r[b]) ||v_neg[b] - v[b]||^2
 * with v = eps - x0 (device float64 [B], may be NULL); loss = mean over b.
 * v_pos, v_neg, eps, x0: device [B, D] of dtype; r: device float32 [B]. */
int ff_nft_loss(const void* v_pos, const void* v_neg, const void* eps, const void* x0, const float* r,
                int64_t B, int64_t D, int32_t dtype, double* per_sample, double* loss, void* workspace,
                size_t ws_bytes, void* stream);

/* Clipped-ratio GRPO objective.  logp_new, logp_old: device float64 [S, B]
 * (SDE step major, as the rollout stores them); adv: device float32 [B];
 * step_w: device float32 [S] or NULL; clip_eps > 0 (FF_EDOMAIN otherwise).
 * loss: device float64 [1]; n_clipped: device int32 [1] or NULL, the number
 * of (k, b) with r outside [1 - clip_eps, 1 + clip_eps].  S * B <= 65536. */
int ff_grpo_loss(const double* logp_new, const double* logp_old, const float* adv, const float* step_w,
                 int64_t B, int32_t S, double clip_eps, double* loss, int32_t* n_clipped, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FF_LOSS_H */
