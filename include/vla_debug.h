/*
 * vla_debug.h -- test hooks of libvla.so: single kernels of the rollout path
 * exposed for kernel-level parity tests.  Not part of the rollout API; same
 * conventions as vla.h (device pointers, async on `stream`, status codes).
 */
#ifndef VLA_DEBUG_H_
#define VLA_DEBUG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Prefill MFMA GEMM: C[M, N] fp32 = A[M, K] bf16 * W[N, K]^T bf16, A and W in
 * frag layout (vla_debug_pack_frag).  Requires K % 32 == 0, N % 64 == 0. */
int vla_debug_gemm(const void* A, const void* W, int32_t M, int32_t N, int32_t K, float* C, void* stream);

/* Decode skinny GEMM: C[M, N] fp32 = A * W^T for M <= 128, A [M, K] and W
 * [N, K] in frag layout, on a persistent grid of at most `workgroups`
 * workgroups; tile segments' partial sums go to `scratch` (16 * M * N floats).
 * Requires N % 64 == 0, K % 256 == 0, N * K < 2^30. */
int vla_debug_skinny(const void* A, const void* W, int32_t M, int32_t N, int32_t K, int32_t workgroups,
                     float* scratch, float* C, void* stream);

/* vla_debug_skinny without a scratch argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops, hosts
 * that forbid allocation): the split-K partials live in a fixed device array
 * of 2^23 floats (32 MiB) that the library holds on each GPU it runs on until
 * the process ends.  Same plan and kernels as vla_debug_skinny, so C gets the
 * same bits.  Requires M <= 128, N % 64 == 0, K % 256 == 0 (else
 * VLA_EUNSUPPORTED) and slots * M * N <= 2^23, where slots (<= 16) is the
 * plan's largest number of partial slots of a column tile (else VLA_ESHAPE;
 * e.g. M = 64 with N = 12288, K = 4096 fits).  Allocates nothing; every call
 * on a GPU shares that GPU's array, so calls that overlap on one GPU (on
 * different streams, or from different threads) race and give wrong results;
 * calls on one stream run in order.  Every partial slot the reduction reads
 * is written by the same call first, so nothing needs clearing. */
int vla_debug_skinny_noalloc(const void* A, const void* W, int32_t M, int32_t N, int32_t K, int32_t workgroups,
                             float* C, void* stream);

/* Repack a row-major bf16 matrix src [rows, K] (row stride ld) into the frag
 * layout the GEMMs read: 16 x 32 blocks of 1 KB; 16-row block r / 16 holds
 * K / 32 + 1 consecutive blocks (the last one spare), K block k / 32 at
 * element ((r / 16) * (K / 32 + 1) + k / 32) * 512, and in it the 8 elements
 * (r, 8 (k % 32 / 8) .. + 8) at element 8 (r % 16 + 16 (k % 32 / 8)).  dst
 * holds ceil(rows / 16) * (K / 32 + 1) * 512 elements; rows past `rows` and
 * the spare blocks are left unwritten.  Requires K % 32 == 0. */
int vla_debug_pack_frag(const void* src, int32_t rows, int32_t K, int32_t ld, void* dst, void* stream);

/* Sampler on given logits z[B, A] at step `step` of gumbel[B, n_actions, A]:
 * writes tokens / logp / entropy / logits at [b, step] exactly as
 * vla_decode_actions does.  `next_tok` receives the sampled vocabulary ids. */
int vla_debug_sample(const float* z, int32_t B, int32_t A, int32_t n_actions, int32_t step, int32_t action_begin,
                     const float* gumbel, float temperature, int32_t* tokens, int32_t* next_tok, float* logp,
                     float* entropy, float* logits_out, void* stream);

/* Copy `bytes` of an internal buffer of the handle to `dst` (device):
 * which = 0 residual x fp32 [rows, d], 1 rotated q bf16 [rows, d], 2 / 3 the K / V
 * page pool of `layer` (bf16, page layouts of the KV cache), 4 the bf16
 * activation buffer [rows, d] in frag layout (see vla_debug_pack_frag); the
 * packed projection weights of `layer`, bf16 in frag layout: 5 [Wq; Wk; Wv]
 * [3 d, d] (q and k rows of each head ordered so that each 64-row block holds
 * rotary pairs 32 rows apart: block b = head rows [32b, 32b+32) then
 * [hd/2 + 32b, hd/2 + 32b + 32)), 6 Wo [d, d], 7 [Wgate; Wup] [2 Fp, d]
 * interleaved in blocks of 32 rows (gate rows 32 (r / 64) + r % 32 at r % 64 < 32,
 * the matching up rows after them; rows past d_ffn zero), 8 Wdown [d, Fp]
 * (columns past d_ffn zero); Fp = d_ffn rounded up to a multiple of 256;
 * 9 the SwiGLU output h, bf16 [rows, Fp] in frag layout. */
struct vla_model;
int vla_debug_read(struct vla_model* m, int32_t which, int32_t layer, void* dst, size_t bytes, void* stream);

/* Make later prefill / teacher-forced passes run only the first `n_layers`
 * decoder layers (0 restores all), so that the residual after any layer can
 * be read with vla_debug_read for layer-by-layer parity.  With a limit set
 * (even n_layers), every row of every layer run is computed; without one,
 * the last layer computes its attention output, O projection and MLP only
 * for the rows read afterwards (the same bits for those rows). */
int vla_debug_set_layer_limit(struct vla_model* m, int32_t n_layers);

/* With a layer limit set, end the last layer run at a stage, so that each
 * rounding point of the layer (Sec. 3.5: the rollout runs in bf16) can be read
 * on its own: 0 the layer's end (x: its output, buffer 9: its SwiGLU output h);
 * 1 before the QKV projection (x: the layer input, buffer 4: the attention
 * norm's output); 2 after attention (buffer 1: rotated q, buffers 2 / 3: the
 * layer's K / V pages, buffer 4: the attention output); 3 after the MLP norm
 * (x: the mid residual, buffer 4: the MLP norm's output).  Stages 1..3 leave
 * the rest of the pass undone; the prefill logits are then not meaningful. */
int vla_debug_set_stop(struct vla_model* m, int32_t stage);

/* Decode path of later vla_decode_actions calls: 0 (the default) runs one
 * kernel per projection and per consumer; 1 (where the device supports
 * cooperative launches) runs each decoder layer's work after attention, and
 * the next projection, in one persistent launch with grid barriers between
 * its phases.  Both give the same bits; the persistent path measured slower
 * (grid barriers and the row phases cost more than the kernel boundaries they
 * replace). */
int vla_debug_set_decode_path(struct vla_model* m, int32_t persistent);

/* Phase timing of the persistent decode layer kernel: the launch of decoder
 * layer `layer` at the first decode step of later vla_decode_actions calls
 * (first 128-row chunk) writes, per workgroup g, 14 wall-clock stamps (the
 * 100 MHz device clock) at stamps[16 g + k]: the start, then before and after
 * each of its 6 grid barriers, and the end.  `stamps` is device memory of
 * 16 * (compute units) uint64, or NULL to stop. */
int vla_debug_trace_decode_layer(struct vla_model* m, int32_t layer, void* stamps);

#ifdef __cplusplus
}
#endif
#endif /* VLA_DEBUG_H_ */
