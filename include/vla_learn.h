/*
 * vla_learn.h -- C ABI of the learning-phase kernels of VLA-RL (arXiv
 * 2505.18719): the advantage estimation that follows the rollout loop of
 * Alg. 1 and the PPO-clip objective of Eq. 2 on the action log-probabilities
 * of Eq. 1, with the gradients that carry that objective back to the logits
 * of the teacher-forced pass (vla_token_logprobs).
 *
 * These calls need no model handle.  Conventions are those of vla.h: device
 * pointers, `hipStream_t` passed as `void*`, asynchronous on that stream,
 * no device allocation, status codes VLA_* with vla_last_error().
 */
#ifndef VLA_LEARN_H_
#define VLA_LEARN_H_

#include "vla.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Generalised advantage estimates of Alg. 1 ("GAE(B_k, V_M, gamma, lambda)")
 * over a window of M = n_steps steps of N = n_env environments, time-major:
 *   rewards     fp32 [M, N]     r_t of Alg. 1
 *   values      fp32 [M + 1, N] V_t; row M is V_M, the value after the window
 *   dones       uint8 [M + 1, N] d_t of Alg. 1 (nonzero: o_t starts a new
 *               episode); transition t continues the episode iff d_{t+1} == 0,
 *               row 0 enters no transition of the window
 *   gamma, lam  discount and GAE parameter, each finite in [0, 1]
 *   advantages  fp32 [M, N] out:
 *               A_t = delta_t + gamma lam (1 - d_{t+1}) A_{t+1},  A_M = 0,
 *               delta_t = r_t + gamma (1 - d_{t+1}) V_{t+1} - V_t
 *   returns     fp32 [M, N] out, or NULL: A_t + V_t
 * n_env == 0 or n_steps == 0 is a no-op.  fp32 arithmetic; the scan is
 * evaluated in 16 time slices whose affine maps are chained, so results match
 * the sequential recursion to fp32 rounding, not bitwise. */
int vla_gae(int32_t n_env, int32_t n_steps, const float* rewards, const float* values, const uint8_t* dones,
            float gamma, float lam, float* advantages, float* returns, void* stream);

/* PPO-clip objective of Eq. 2 over n actions of n_tokens tokens each.  The
 * action log-probability is the sum of its token log-probabilities (Eq. 1),
 * rho_t = exp(sum_i logp_new[t, i] - sum_i logp_old[t, i]), and
 *     J = (1/n) sum_t min(rho_t A_t, clip(rho_t, 1 - eps, 1 + eps) A_t).
 *   logp_new, logp_old  fp32 [n, n_tokens] (e.g. vla_token_logprobs under the
 *                       current weights, and the rollout's vla_decode_actions)
 *   advantages          fp32 [n]
 *   eps                 clipping parameter, finite and >= 0
 *   stats               fp32 [2] out: stats[0] = -J (the loss a minimiser
 *                       uses), stats[1] = fraction of actions whose clipped
 *                       term is the minimum (A > 0 and rho > 1 + eps, or
 *                       A < 0 and rho < 1 - eps)
 *   dlogp               fp32 [n, n_tokens] out: d(-J)/d logp_new[t, i], which
 *                       is 0 for a clipped action and -rho_t A_t / n otherwise
 * 1 <= n_tokens <= 16, n >= 1 (else VLA_EINVAL).  The clipping decision is
 * taken in fp32; the loss is reduced in a fixed order (same bits every run). */
int vla_ppo_clip(int32_t n, int32_t n_tokens, const float* logp_new, const float* logp_old,
                 const float* advantages, float eps, float* stats, float* dlogp, void* stream);

/* Backward of the token log-probabilities over the action bins (the scoring
 * of vla_token_logprobs): for row r with logits z_r and token k_r,
 *     dlogits[r, j] = dlogp[r] (1[j = k_r] - softmax(z_r / T)_j) / T.
 *   rows          rows to process (batch * n_actions for a teacher-forced pass)
 *   bins          action bins per row, 1 <= bins <= 256
 *   action_begin  vocabulary id of bin 0; k_r = tokens[r] - action_begin
 *   logits        fp32 [rows, bins] raw logits (before temperature)
 *   tokens        int32 [rows] vocabulary ids; one outside the bins gives a
 *                 row of NaN
 *   temperature   T > 0
 *   dlogp         fp32 [rows] gradient arriving at each token log-probability
 *   dlogits       fp32 [rows, bins] out
 * rows == 0 is a no-op. */
int vla_logprob_backward(int32_t rows, int32_t bins, int32_t action_begin, const float* logits,
                         const int32_t* tokens, float temperature, const float* dlogp, float* dlogits,
                         void* stream);

#ifdef __cplusplus
}
#endif
#endif /* VLA_LEARN_H_ */
