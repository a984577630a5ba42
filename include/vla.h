/*
 * vla.h -- C ABI of the MI355X (gfx950) batched VLA rollout-inference library.
 *
 * The library runs the policy step of VLA-RL's rollout phase (arXiv
 * 2505.18719, Alg. 1 and Sec. 3.3): for a batch of environments it prefills
 * [projected visual patch embeddings ; instruction prompt tokens] through an
 * OpenVLA-style Llama-2 decoder (Sec. 3.1), then generates the |A| = 7 action
 * tokens auto-regressively with a paged KV cache, sampling each token among
 * the action bins (the last `action_bins` vocabulary ids, one bin per action
 * dimension, Sec. 3.1) by Gumbel-max with caller-supplied noise, and returns
 * the per-token log-probabilities whose sum is the action log-probability of
 * Eq. 1, plus per-token entropies.  A teacher-forced entry point recomputes
 * log-probabilities of stored action tokens, the numerator of the PPO ratio
 * (Eq. 2).  Rollout runs in bf16 (Sec. 3.5, "Infrastructure"): weights and
 * stored activations are bf16, accumulation and the residual stream fp32.
 *
 * Conventions
 *  - Every pointer is a DEVICE pointer unless its name ends in `_host`.
 *  - Streams are `hipStream_t` passed as `void*` (NULL = the default stream).
 *    All work is enqueued asynchronously on that stream; outputs are valid
 *    once the stream has been synchronised.  No call synchronises the host
 *    with the device except `vla_read_device_flags`.
 *  - The library never allocates device memory: the caller provides one
 *    workspace of `vla_workspace_size` bytes and owns every buffer.
 *  - Matrices are row-major.  Linear weights are `[out_features, in_features]`.
 *  - Every call returns a status (0 = success, negative = error) and sets a
 *    thread-local message readable with `vla_last_error`.  No C++ exception
 *    crosses this boundary.
 *  - A model handle is not thread-safe; use one handle per stream.
 */
#ifndef VLA_H_
#define VLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define VLA_OK 0
#define VLA_EINVAL -1        /* null pointer, non-positive size, bad temperature, ... */
#define VLA_ESHAPE -2        /* batch > max_batch or a sequence longer than max_seq */
#define VLA_EWORKSPACE -3    /* workspace smaller than vla_workspace_size() or misaligned */
#define VLA_EHIP -4          /* a HIP runtime call failed; the message holds HIP's text */
#define VLA_ESTATE -6        /* decode without a matching prefill on this handle */
#define VLA_EUNSUPPORTED -7  /* configuration outside what the kernels implement */

/* device-side flags (see vla_read_device_flags) */
#define VLA_FLAG_BAD_PROMPT_ID 1u   /* a prompt id outside [0, vocab): a zero row was used */
#define VLA_FLAG_BAD_ACTION 2u      /* a teacher-forced token outside the action range: scored as NaN */
#define VLA_FLAG_SYNC_TIMEOUT 4u    /* a grid barrier of the persistent decode kernel timed out: that decode's
                                       outputs are invalid */

/* Decoder shape and capacity.
 *   d_model = n_heads * head_dim, head_dim in {64, 128}, d_model % 256 == 0,
 *   d_model <= 8192; d_ffn >= 1 (padded internally to a multiple of 64);
 *   1 <= action_bins <= 256; action_begin + action_bins <= vocab;
 *   1 <= n_actions <= 16; max_seq <= 320 (prefix + n_actions rows of one env);
 *   page_size == 16; 1 <= max_batch <= 512. */
typedef struct vla_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t head_dim;
  int32_t d_ffn;
  int32_t vocab;
  int32_t action_bins;   /* number of action bins (256 for OpenVLA) */
  int32_t action_begin;  /* vocabulary id of bin 0 (vocab - action_bins for OpenVLA) */
  int32_t n_actions;     /* action tokens per environment step, |A| = 7 (Eq. 1) */
  int32_t n_visual;      /* visual patch embeddings per observation (256) */
  float rope_base;       /* rotary base, 10000 */
  float rms_eps;         /* RMSNorm epsilon, 1e-6 */
  int32_t max_batch;     /* largest batch passed to any call on the handle */
  int32_t max_seq;       /* longest sequence: n_visual + prompt + n_actions */
  int32_t page_size;     /* KV-cache page size in tokens (16) */
} vla_config;

/* Decoder weights, all bf16 device memory, read only during vla_create.
 * Per-layer entries are HOST arrays of n_layers device pointers. */
typedef struct vla_weights {
  const void* embed;              /* [vocab, d_model] token embedding */
  const void* lm_head;            /* [vocab, d_model] output projection (untied) */
  const void* final_norm;         /* [d_model] RMSNorm gain */
  const void* const* attn_norm;   /* [d_model] per layer */
  const void* const* wq;          /* [d_model, d_model] per layer */
  const void* const* wk;          /* [d_model, d_model] */
  const void* const* wv;          /* [d_model, d_model] */
  const void* const* wo;          /* [d_model, d_model] */
  const void* const* mlp_norm;    /* [d_model] */
  const void* const* wgate;       /* [d_ffn, d_model] */
  const void* const* wup;         /* [d_ffn, d_model] */
  const void* const* wdown;       /* [d_model, d_ffn] */
} vla_weights;

typedef struct vla_model vla_model;  /* opaque handle */

/* Bytes of device workspace a model with this configuration needs: repacked
 * weights, the paged KV pool for max_batch * max_seq tokens, activations and
 * split-K partials.  Returns VLA_EINVAL / VLA_EUNSUPPORTED for a bad config. */
int vla_workspace_size(const vla_config* cfg, size_t* bytes_host);

/* Validate `cfg`, lay out `workspace` (256-byte aligned, >= vla_workspace_size
 * bytes, owned by the caller and kept alive until vla_destroy) and repack the
 * weights into it on `stream`: fused [Wq;Wk;Wv] with the rotary pairs of each
 * head arranged for the fused RoPE epilogue, interleaved [Wgate;Wup], the
 * action-bin rows of the LM head, fp32 norm gains and a rotary table computed
 * on the host in double precision.  The caller may free `weights` once
 * `stream` has completed.  On success *out receives the handle. */
int vla_create(const vla_config* cfg, const vla_weights* weights, void* workspace,
               size_t workspace_bytes, void* stream, vla_model** out);

/* Prefill (Alg. 1, the policy-generation step, first half): for environment b
 * the sequence is its n_visual rows of `vis_emb` followed by the embedding
 * rows of its prompt ids, at positions 0 .. L_b-1 with L_b = n_visual +
 * prompt_lens_host[b] (causal attention over the whole prefix, no special
 * tokens).  Environments are packed without padding (ragged prefill) and each
 * gets its own KV-cache pages.
 *   vis_emb          bf16 [batch, n_visual, d_model]
 *   prompt_ids       int32 [sum(prompt_lens_host)], environment b's ids follow env b-1's
 *   prompt_lens_host int32 [batch] on the host, each >= 0, L_b + n_actions <= max_seq
 *   action_logits    fp32 [batch, action_bins] out: logits of the action bins at
 *                    the last prefix row (raw, before temperature)
 * The handle keeps the KV cache and these logits for vla_decode_actions. */
int vla_prefill(vla_model* m, int32_t batch, const void* vis_emb, const int32_t* prompt_ids,
                const int32_t* prompt_lens_host, float* action_logits, void* stream);

/* Decode the n_actions action tokens of the batch prefilled last (Alg. 1,
 * policy generation and the sum of token log-probabilities, Eq. 1).  Token i
 * is bin k_i = argmax_j (z_ij / T + g_ij) (lowest j on exact ties), i.e. a
 * draw from softmax(z_i / T) over the action bins, where z_i are the logits
 * at position L_b - 1 + i; tokens 0 .. n_actions-2 are fed back through the
 * KV-cached decoder.
 *   batch        must equal the last vla_prefill's batch (else VLA_ESTATE)
 *   gumbel       fp32 [batch, n_actions, action_bins] standard Gumbel noise g
 *   temperature  T > 0 (VLA-RL samples at T = 1.5)
 *   tokens       int32 [batch, n_actions] out: vocabulary ids action_begin + k_i
 *   logp         fp32 [batch, n_actions] out: log softmax(z_i / T)[k_i]
 *   entropy      fp32 [batch, n_actions] out, or NULL: entropy of softmax(z_i / T)
 *   step_logits  fp32 [batch, n_actions, action_bins] out, or NULL: z_i
 * The decode consumes the prefill state: a second call needs a new prefill.
 * Batches above 128 environments run the decoder layers once per chunk of
 * at most 128 environments (each chunk streams the weights again); results
 * do not depend on the chunking. */
int vla_decode_actions(vla_model* m, int32_t batch, const float* gumbel, float temperature,
                       int32_t* tokens, float* logp, float* entropy, float* step_logits,
                       void* stream);

/* Action extraction a_t = f(v_out) of Alg. 1 (Sec. 3.3: each action token
 * is a discrete bin of one dimension of the robot action space).  Token i of
 * an environment's sequence is dimension i; its bin k = token - action_begin
 * of `bins` uniform bins over [range_lo[i], range_hi[i]] maps to the bin
 * centre
 *     actions[r, i] = range_lo[i] + (k + 1/2) (range_hi[i] - range_lo[i]) / bins
 * (fp32).  The ranges are those the policy's actions were discretised over
 * (for OpenVLA the 1st and 99th percentiles of each dimension of the
 * training actions); the caller supplies them.  Needs no model handle.
 *   n                 environments (rows); n_dims  action dimensions per row
 *   tokens            int32 [n, n_dims] vocabulary ids (e.g. from vla_decode_actions)
 *   bins              1 <= bins <= 256
 *   range_lo, range_hi fp32 [n_dims]
 *   actions           fp32 [n, n_dims] out; NaN where a token is outside the bins
 * n == 0 is a no-op. */
int vla_extract_actions(int32_t n, int32_t n_dims, const int32_t* tokens, int32_t action_begin, int32_t bins,
                        const float* range_lo, const float* range_hi, float* actions, void* stream);

/* Value estimates V_t = V(o_t, v_in) of Alg. 1 by a value model of the
 * policy's own architecture (the "homogeneous value model" of Fig. 2): the
 * decoder held by `m` (create the handle with the value model's weights) runs
 * over [visual ; prompt] as in vla_prefill, then
 *     values[b] = value_head . RMSNorm_final(h_b)     (fp32 accumulation)
 * where h_b is the hidden state at the last prefix row L_b - 1 and the normed
 * state is rounded to bf16 as at the action head's input.
 *   vis_emb, prompt_ids, prompt_lens_host  as in vla_prefill
 *   value_head  bf16 [d_model], read only
 *   values      fp32 [batch] out
 * Overwrites the handle's prefill state (a later decode needs a new prefill). */
int vla_value(vla_model* m, int32_t batch, const void* vis_emb, const int32_t* prompt_ids,
              const int32_t* prompt_lens_host, const void* value_head, float* values, void* stream);

/* LoRA merge before a rollout (Sec. 3.3, Rollout Phase: the updated LoRA
 * weights are merged with the original checkpoint): replaces one projection
 * of one decoder layer in the handle's packed weights by
 *     W = bf16(W0 + scale * B A)            (round to nearest even)
 * where W0 is the ORIGINAL checkpoint weight of that projection (so repeated
 * merges never accumulate: each starts from W0) and B A the adapter's rank-r
 * update, summed over r in fp32.  Every other weight is left as it is.
 *   layer       0 .. n_layers-1
 *   projection  VLA_PROJ_* (q, k, v, o, gate, up, down)
 *   w0          bf16 [out, in] row-major, the checkpoint weight as given to
 *               vla_create (q, k, v, o: [d, d]; gate, up: [d_ffn, d];
 *               down: [d, d_ffn]); read only
 *   lora_a      bf16 [rank, in] row-major; lora_b bf16 [out, rank] row-major
 *   rank        8 <= rank <= 64, a multiple of 8 (else VLA_EUNSUPPORTED)
 *   scale       alpha / rank of the adapter (finite, else VLA_EINVAL)
 * Asynchronous on `stream`; later calls on the same stream see the merged
 * weights.  All pointers are device pointers owned by the caller. */
#define VLA_PROJ_Q 0
#define VLA_PROJ_K 1
#define VLA_PROJ_V 2
#define VLA_PROJ_O 3
#define VLA_PROJ_GATE 4
#define VLA_PROJ_UP 5
#define VLA_PROJ_DOWN 6
int vla_lora_merge(vla_model* m, int32_t layer, int32_t projection, const void* w0, const void* lora_a,
                   const void* lora_b, int32_t rank, float scale, void* stream);

/* Every projection of one layer in one launch: vla_lora_merge for each
 * projection p (VLA_PROJ_* order, arrays of 7 device pointers held in host
 * memory) whose w0[p] is not NULL, the others left as they are; the merged
 * weights are the bits the seven separate calls give.  Same argument rules
 * and errors as vla_lora_merge (checked for every merged projection before
 * anything is launched); rank and scale are shared by the layer's adapters. */
int vla_lora_merge_layer(vla_model* m, int32_t layer, const void* const* w0, const void* const* lora_a,
                         const void* const* lora_b, int32_t rank, float scale, void* stream);

/* Teacher-forced pass (numerator of the PPO ratio, Eq. 2): one causal forward
 * over [visual ; prompt ; the n_actions given action tokens] per environment,
 * with no KV reuse, scoring token i by the logits at row L_b - 1 + i.
 *   vis_emb, prompt_ids, prompt_lens_host  as in vla_prefill
 *   action_tokens  int32 [batch, n_actions] vocabulary ids in
 *                  [action_begin, action_begin + action_bins); others raise
 *                  VLA_FLAG_BAD_ACTION and are scored as NaN
 *   logp, entropy  fp32 [batch, n_actions] out (entropy may be NULL)
 *   logits         fp32 [batch, n_actions, action_bins] out, or NULL
 * Overwrites the handle's prefill state (a later decode needs a new prefill). */
int vla_token_logprobs(vla_model* m, int32_t batch, const void* vis_emb, const int32_t* prompt_ids,
                       const int32_t* prompt_lens_host, const int32_t* action_tokens,
                       float temperature, float* logp, float* entropy, float* logits, void* stream);

/* Synchronise `stream`, return the OR of VLA_FLAG_* raised by kernels since
 * the last read into *flags_host, and clear them. */
int vla_read_device_flags(vla_model* m, void* stream, uint32_t* flags_host);

/* Live kernel timing.  vla_profile_begin(m, mask) starts recording a pair of
 * HIP events on the launch stream around every kernel launch of the selected
 * categories (bit i of `mask` selects category i) together with the
 * launch's algorithmic work (flops for VLA_PROF_PREFILL_*, HBM bytes for
 * VLA_PROF_DECODE_*: weights, activations and KV read once, no split-K
 * partials).  vla_profile_end waits for the recorded events and, for each
 * category, writes the summed kernel time in milliseconds, the summed work
 * and the number of launches into arrays of VLA_PROF_CATEGORIES entries, then
 * stops recording.  At most 16384 launches are recorded per begin/end. */
#define VLA_PROF_PREFILL_GEMM 0
#define VLA_PROF_PREFILL_ATTN 1
#define VLA_PROF_DECODE_GEMM 2
#define VLA_PROF_DECODE_ATTN 3
#define VLA_PROF_DECODE_LAYER 4  /* persistent decode layer kernel: HBM bytes of its four projections */
#define VLA_PROF_CATEGORIES 5
int vla_profile_begin(vla_model* m, uint32_t mask);
int vla_profile_end(vla_model* m, double* ms_host, double* work_host, int64_t* launches_host);

/* Release the handle (not the caller's workspace).  Safe on NULL. */
void vla_destroy(vla_model* m);

/* Message of the last failed call on this thread ("" if none). */
const char* vla_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* VLA_H_ */
