/*
 * vla_learn.h -- C ABI of the learning-phase kernels of VLA-RL (arXiv
 * 2505.18719): the advantage estimation that follows the rollout loop of
 * Alg. 1 and the PPO-clip objective of Eq. 2 on the action log-probabilities
 * of Eq. 1, with the gradients that carry that objective back to the logits
 * of the teacher-forced pass (vla_token_logprobs).
 *
 * All calls but vla_ppo_lora_grads (which runs the decoder held by a model
 * handle) need no handle.  Conventions are those of vla.h: device
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

/* LoRA adapters of the policy (Sec. 3.3: the policy is trained through LoRA
 * adapters, merged as W = W0 + scale * B A) and the buffers for their
 * gradients: host arrays of n_layers * 7 device pointers, layer-major, the
 * projections in VLA_PROJ_* order (q, k, v, o, gate, up, down).  A NULL entry
 * of `a` marks a projection without an adapter; its gradients are not written. */
typedef struct vla_lora {
  int32_t rank;            /* 1 <= rank <= 64 */
  float scale;             /* alpha / rank */
  const void* const* a;    /* bf16 [rank, in] row-major */
  const void* const* b;    /* bf16 [out, rank] row-major */
  float* const* grad_a;    /* fp32 [rank, in] out: dL/dA */
  float* const* grad_b;    /* fp32 [out, rank] out: dL/dB */
} vla_lora;

/* Training modes, by what the forward of vla_ppo_lora_grads keeps per layer. */
#define VLA_TRAIN_RECOMPUTE 0 /* the layer's input only; the backward recomputes the layer's
                                 forward from it before its gradients */
#define VLA_TRAIN_KEEP 1      /* also the normed inputs, rotated queries, attention output and
                                 log-sum-exp, mid residual and fp32 gate/up pre-activations:
                                 no recompute (about 2.9 GB per layer at d = 4096, d_ffn =
                                 11008 and 64 x 320 rows) */

/* Bytes of the training workspace vla_ppo_lora_grads needs for a handle of
 * this configuration in `mode` (VLA_TRAIN_*), for max_batch * max_seq rows:
 * what the forward keeps per layer, one layer's gradients, transposed
 * operands.  Unknown mode: VLA_EINVAL. */
int vla_train_workspace_size(const vla_config* cfg, int32_t mode, size_t* bytes_host);

/* Gradient of one PPO update (Eq. 2, Sec. 3.3 Learning Phase) with respect to
 * the LoRA factors.  The handle's packed weights must be the policy being
 * updated, i.e. the merge of these adapters (vla_lora_merge).  Runs the
 * teacher-forced pass over [visual ; prompt ; stored actions] (as
 * vla_token_logprobs, every row of every layer), the PPO-clip loss on the
 * action log-probabilities (vla_ppo_clip) and its gradient down to the
 * action logits (vla_logprob_backward), then the backward of the whole pass:
 * the head and final RMSNorm of the scoring rows, and for each layer from the
 * top (after recomputing its forward from its input in VLA_TRAIN_RECOMPUTE
 * mode) the gradient GEMMs against its transposed weights, RMSNorm, SwiGLU
 * and causal-attention (with rotary) backward, and the LoRA gradients dL/dB = scale dY^T (X A^T),
 * dL/dA = scale (dY B)^T X of each adapted projection (X its input rows, dY
 * the gradient of its output rows: the rank-r reductions of its weight
 * gradient dY^T X, taken without forming it).
 *   batch, vis_emb, prompt_ids, prompt_lens_host, action_tokens  as in
 *                vla_token_logprobs
 *   logp_old     fp32 [batch, n_actions] token log-probs of the rollout policy
 *   advantages   fp32 [batch]
 *   eps, temperature  clipping parameter (>= 0) and sampling temperature (> 0)
 *   lora         adapters and gradient buffers (see vla_lora)
 *   train_ws     device memory, 256-byte aligned: with at least
 *                vla_train_workspace_size(VLA_TRAIN_KEEP) bytes the call keeps every
 *                layer's activations, else with at least the VLA_TRAIN_RECOMPUTE size
 *                it recomputes them (same results, bit for bit), else VLA_EWORKSPACE
 *   stats        fp32 [2] out: loss -J and clipped fraction
 *   logp_new     fp32 [batch, n_actions] out, or NULL: the teacher-forced log-probs
 * Gradient operands of the GEMMs, and the rank-r products X A^T and
 * dY B, are rounded to bf16 as the forward's activations are (fp32
 * accumulation).  Overwrites the handle's prefill state. */
int vla_ppo_lora_grads(struct vla_model* m, int32_t batch, const void* vis_emb, const int32_t* prompt_ids,
                       const int32_t* prompt_lens_host, const int32_t* action_tokens, const float* logp_old,
                       const float* advantages, float eps, float temperature, const vla_lora* lora,
                       void* train_ws, size_t train_ws_bytes, float* stats, float* logp_new, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* VLA_LEARN_H_ */
