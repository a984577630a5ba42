// Launch interface of the gfx950 kernels (host side).  Every launcher takes
// plain device pointers and a stream and returns the launch's hipError_t.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vla {

typedef uint16_t bf16_t;

// Paged KV cache of one layer.  K pages are [page][head][slot][head_dim]
// (each key row contiguous); V pages are stored transposed,
// [page][head][head_dim][slot], so that 8 consecutive keys of one feature are
// one 16-byte load for the attention P*V products.  page_size is 16 tokens.
constexpr int kPage = 16;

struct KvCache {
  bf16_t* k;
  bf16_t* v;
};

// Per-row metadata of a packed ragged batch (device arrays).
struct RowMeta {
  const int32_t* row_pos;     // [M] position of the row inside its environment
  const int32_t* row_env;     // [M] environment of the row
  const int32_t* page_table;  // [B, max_pages] physical page of each 16-token block
  int max_pages;
};

// Prefill GEMM, C = A * W^T with A [M, K] bf16 (row stride lda) and W [N, K]
// bf16, fp32 accumulation on MFMA, and one of these epilogues:
enum GemmEpilogue {
  kEpiStoreF32 = 0,  // C[m, n] = acc                         (fp32, ldc)
  kEpiResidual = 1,  // C[m, n] = (R ? R : C)[m, n] + acc     (fp32 residual stream, ldc)
  kEpiSwiGlu = 2,    // H[m, j] = bf16(silu(gate) * up)  for W = interleaved [gate; up] blocks of 32 rows;
                     //   H in frag layout with K = ldh
  kEpiQkvRope = 3,   // rotate q, k by RoPE, store q bf16 [M, d] and K/V into the page pool
  kEpiSwiGluKeep = 4,  // kEpiSwiGlu, and the fp32 pre-activations C[m, n] = acc kept (ldc) for a backward
};

struct GemmArgs {
  const bf16_t* A;  // [M, K] in frag layout
  const bf16_t* W;  // [N, K] in frag layout
  int M, N, K;
  int ka, kw;       // K of A's and W's frag allocations when wider than the contraction (0: K)
  float* C;
  int ldc;
  const float* R;   // kEpiResidual: the residual read (row stride ldc), or null for C itself
  bf16_t* H;
  int ldh;
  // kEpiQkvRope
  bf16_t* q;
  int ldq;
  KvCache kv;
  RowMeta meta;
  const float2* rope;  // [pos][head_dim / 2] (cos, sin)
  int d_model, n_heads, head_dim;
};

hipError_t launch_gemm(const GemmArgs& a, GemmEpilogue epi, hipStream_t s);

// Skinny GEMM for decode: C = A[M, K] * W[N, K]^T for M <= 128 rows, N % 64 == 0,
// K % 256 == 0, N * K < 2^30.  The work is cut into units of 64 columns
// (a tile) x 256 K; a persistent grid of `G` workgroups takes whole tiles one
// per workgroup per round while at least G remain (tiles [0, dp_tiles)), then
// splits the remaining tiles' units evenly, in tile order, over the G
// workgroups.  Each tile segment a workgroup computes is stored as an fp32
// partial sum at part[slot, m, n]; tile t has skinny_slots(plan, t) slots and
// its result is their sum in slot order.
struct SkinnyArgs {
  const bf16_t* A;  // [M, K] in frag layout
  int M;
  const bf16_t* W;  // [N, K] in frag layout
  int N, K;
  float* part;      // [plan.slots, M, N]
};
struct SkinnyPlan {
  int tiles;     // N / 64
  int chunks;    // K / 256 units per tile
  int G;         // workgroups
  int dp_tiles;  // tiles computed whole (a multiple of G)
  int slots;     // most partial slots of any tile
};
// workgroup whose stream-K run holds unit u of U (runs [g U / G, (g+1) U / G))
__host__ __device__ inline int skinny_owner(int u, int U, int G) { return ((u + 1) * G + U - 1) / U - 1; }
__host__ __device__ inline int skinny_slots(const SkinnyPlan& p, int tile) {
  if (tile < p.dp_tiles) return 1;
  const int U = (p.tiles - p.dp_tiles) * p.chunks, t = tile - p.dp_tiles;
  return skinny_owner((t + 1) * p.chunks - 1, U, p.G) - skinny_owner(t * p.chunks, U, p.G) + 1;
}
// Partial slots loaded together before they are summed (more slots: summed one by one after).
constexpr int kSlotsAhead = 8;

// v + the sum of ns partial slots (slot s at p[s * stride]), added in slot order.
__device__ inline float sum_slots(const float* __restrict__ p, size_t stride, int ns, float v) {
  float q[kSlotsAhead];
#pragma unroll
  for (int s = 0; s < kSlotsAhead; ++s)
    if (s < ns) q[s] = p[s * stride];
#pragma unroll
  for (int s = 0; s < kSlotsAhead; ++s)
    if (s < ns) v += q[s];
  for (int s = kSlotsAhead; s < ns; ++s) v += p[s * stride];
  return v;
}
__device__ inline float4 sum_slots4(const float* __restrict__ p, size_t stride, int ns, float4 v) {
  float4 q[kSlotsAhead];
#pragma unroll
  for (int s = 0; s < kSlotsAhead; ++s)
    if (s < ns) q[s] = *reinterpret_cast<const float4*>(p + s * stride);
#pragma unroll
  for (int s = 0; s < kSlotsAhead; ++s)
    if (s < ns) {
      v.x += q[s].x; v.y += q[s].y; v.z += q[s].z; v.w += q[s].w;
    }
  for (int s = kSlotsAhead; s < ns; ++s) {
    const float4 t = *reinterpret_cast<const float4*>(p + s * stride);
    v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
  }
  return v;
}

// Sum of the partial slots of column n of a skinny GEMM (N columns) at row m.
__device__ inline float skinny_sum(const float* __restrict__ part, const SkinnyPlan& p, int M, int N, int m, int n) {
  return sum_slots(part + (size_t)m * N + n, (size_t)M * N, skinny_slots(p, n >> 6), 0.f);
}
// The plan for `workgroups` workgroups, with fewer if needed to keep every tile within `max_slots`.
SkinnyPlan skinny_plan(int N, int K, int workgroups, int max_slots);
hipError_t launch_skinny(const SkinnyArgs& a, const SkinnyPlan& p, hipStream_t s);

// Persistent decode layer (decode_layer.hip): everything of a decoder layer
// after attention at one decode step, plus the next projection, in one
// cooperative launch of G workgroups (one per CU).
struct DecodeLayerArgs {
  SkinnyArgs o, gu, dn, nx;            // O, [gate; up], down, and the next (QKV or action head) projections
  SkinnyPlan p_o, p_gu, p_dn, p_nx;
  float* x;                            // residual [M, d] fp32
  const float* g_mlp;                  // MLP RMSNorm gain
  const float* g_next;                 // the next RMSNorm's gain (next layer's attention norm, or the final norm)
  bf16_t* ua;                          // MLP norm output [M, d] frag (gu.A)
  bf16_t* h;                           // SwiGLU output [M, Fp] frag (dn.A)
  bf16_t* ub;                          // next norm output [M, d] frag (nx.A)
  int M, d, Fp;
  float eps;
  unsigned* bar;                       // barrier block: [0] global count, [1] abort word, [16 (1 + g % 8)] group counts
  unsigned bar_base;                   // barriers passed before this launch in the current decode call
  uint32_t* flags;                     // VLA flags (4: a barrier wait timed out)
  unsigned long long* trace;           // test hook, or null: per workgroup 16 wall-clock stamps of its phases
};
constexpr int kDecodeLayerBarriers = 6;  // grid barriers per launch
hipError_t launch_decode_layer(const DecodeLayerArgs& a, int G, hipStream_t s);
// Whether the current device can run it: cooperative launches, and one workgroup
// of every row-block variant resident per CU.
bool decode_layer_supported();

// Set the calling thread's message for vla_last_error and return `code`.
int set_error(int code, const char* msg);

// Elementwise / reduction kernels
struct EmbedArgs {
  float* x;                     // [M, d] out
  const bf16_t* emb;            // [vocab, d]
  const bf16_t* vis;            // [B, n_visual, d]
  const int32_t* prompt_ids;    // packed
  const int32_t* actions;       // [B, n_actions] or null
  const int32_t* row_pos;
  const int32_t* row_env;
  const int32_t* env_prefix;    // [B] L_b
  const int32_t* env_prompt_off;// [B]
  int M, d, n_visual, n_actions, vocab;
  uint32_t* flags;
};
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);

// u[i] = bf16(rmsnorm(x[rows ? rows[i] : i]) * g), i < M; u row-major with row
// stride ldu, or in frag layout (K = d, d % 256 == 0, d <= 8192) when `frag` is
// set, where the rows of the last 16-row block past M are written as zeros
hipError_t launch_rmsnorm(const float* x, int ldx, const int32_t* rows, const float* g, float eps,
                          bf16_t* u, int ldu, int M, int d, hipStream_t s, bool frag = false);

// Decode step input: x[b] = emb[tok[b]], u[b] = bf16(rmsnorm(x[b]) * g), u in frag layout
hipError_t launch_embed_token_norm(const int32_t* tok, const bf16_t* emb, float* x, bf16_t* u,
                                   const float* g, float eps, int B, int d, int vocab,
                                   uint32_t* flags, hipStream_t s);

// Consumers of a skinny GEMM's partial sums (plan `p`, partial rows of p.tiles * 64 floats):
// x[m] += C[m, :];  u[m] = bf16(rmsnorm(x[m]) * g)   (M rows of d; u in frag layout)
hipError_t launch_reduce_residual_norm(const float* part, const SkinnyPlan& p, float* x, bf16_t* u,
                                       const float* g, float eps, int M, int d, hipStream_t s);
// z[m, n] = C[m, n] for n < N (z rows of N floats)
hipError_t launch_reduce_sum(const float* part, const SkinnyPlan& p, float* z, int M, int N, hipStream_t s);
// h[m, j] = bf16(silu(C[m, gate_j]) * C[m, up_j]) for j < F (h in frag layout, K = ldh),
// C's columns interleaved
// as [32 gate; 32 up] blocks (column 64 (j / 32) + j % 32 and 32 further)
hipError_t launch_reduce_swiglu(const float* part, const SkinnyPlan& p, bf16_t* h, int ldh, int M, int F,
                                hipStream_t s);

// Attention
struct PrefillAttnArgs {
  const bf16_t* q;  // [M, d]
  bf16_t* o;        // [M, d] in frag layout
  KvCache kv;
  const int32_t* page_table;
  int max_pages;
  const int32_t* env_row0;    // [B] first packed row of env b
  const int32_t* env_len;     // [B] rows of env b in this pass (<= 320)
  int n_env, d, n_heads, head_dim;
  float scale;
  const int32_t* env_q0;      // [B] first query row of env b whose output is needed, or null for all;
                              // the 16-row query tiles below its tile are skipped
  float* lse;                 // [M, n_heads, 2] or null: [row, head, 0] receives log sum_j exp(scale q.k_j)
};
hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t s);

// Decode attention fused with the QKV projection's consumer: each workgroup
// (head, environment) first sums the partial slots of its q, k, v columns,
// rotates q and k, appends k and v to the page pool at the token's position,
// then attends over keys 0 .. env_prefix[b] + step - 1 (the last one is the
// token itself, taken from LDS with the same bf16 rounding).
struct DecodeAttnArgs {
  const float* part;   // QKV projection partial slots [plan.slots, B, 3 d] (q, k rows permuted per head)
  SkinnyPlan plan;
  const float2* rope;  // [pos][head_dim / 2] (cos, sin)
  bf16_t* o;           // [B, d] in frag layout
  KvCache kv;
  const int32_t* page_table;
  int max_pages;
  const int32_t* env_prefix;
  int step;  // 1-based decode step: token position = env_prefix[b] + step - 1
  int B, d, n_heads, head_dim;
  float scale;
};
hipError_t launch_attn_decode(const DecodeAttnArgs& a, hipStream_t s);

// Sampler over the action bins (one wave per row).
struct SamplerArgs {
  const float* z;          // [rows, A] logits
  int A;
  float temperature;
  // sampling mode (gumbel != null): row b, step i
  const float* gumbel;     // [B, n_actions, A]
  int step, n_actions, action_begin;
  int32_t* tokens;         // [B, n_actions]
  int32_t* next_tok;       // [B]
  // teacher-forced mode (gumbel == null): row r = b * n_actions + i scores given[r]
  const int32_t* given;    // [rows]
  float* logp;             // sampling: [B, n_actions] at step; TF: [rows]
  float* entropy;          // same layout, may be null
  float* logits_out;       // same layout times A, may be null
  int rows;
  uint32_t* flags;
};
hipError_t launch_sampler(const SamplerArgs& a, hipStream_t s);

// Weight packing (one-time, at create): dst [rows, K] in frag layout (see frag_index)
enum PackMode { kPackRows = 0, kPackQk = 1, kPackGateUp = 2 };
// Source row of destination row r under a packing mode, or -1 for a zero
// row; for kPackGateUp `part` receives 0 (gate) or 1 (up).
__device__ inline int pack_src_row(int mode, int r, int head_dim, int src_rows, int& part) {
  part = 0;
  if (mode == kPackRows) return r < src_rows ? r : -1;
  if (mode == kPackQk) {
    const int head = r / head_dim, p = r % head_dim, half = head_dim / 2;
    const int blk = p / 64, c = p % 64;
    return head * head_dim + (c < 32 ? 32 * blk + c : half + 32 * blk + c - 32);
  }
  part = (r % 64) < 32 ? 0 : 1;
  const int j = 32 * (r / 64) + (r % 32);
  return j < src_rows ? j : -1;
}
struct PackArgs {
  bf16_t* dst;
  int rows, K;
  const bf16_t* src;   // row-major source, row stride src_ld
  const bf16_t* src2;  // up projection (kPackGateUp)
  int src_ld, src_rows, src_cols;
  int mode, head_dim;
};
hipError_t launch_pack_frag(const PackArgs& a, hipStream_t s);
// LoRA merge into a packed weight (frag layout, rows placed as launch_pack_frag
// places them for `mode`): destination row r of source row j gets
// bf16(w0[j, :] + scale * (b[j, :] a)) with a [rank, src_cols], b [src_rows, rank]
// row-major bf16 and the rank sum accumulated in fp32.  For kPackGateUp only
// the rows of `part` (0 gate, 1 up) are computed and written (rows % 64 == 0).  Requires K % 64 == 0,
// rank % 8 == 0, 8 <= rank <= 64, src_ld and src_cols multiples of 8.
struct MergeArgs {
  bf16_t* dst;
  int rows, K;
  const bf16_t* w0;
  int src_ld, src_rows, src_cols;
  int mode, head_dim, part;
  const bf16_t* a;
  const bf16_t* b;
  int rank;
  float scale;
};
hipError_t launch_lora_merge(const MergeArgs& a, hipStream_t s);
// Up to seven merges (e.g. every projection of one layer) in one launch; each
// item as launch_lora_merge requires it, item results as if merged one by one.
constexpr int kMergeBatchMax = 7;
struct MergeBatch {
  MergeArgs item[kMergeBatchMax];
  int wg0[kMergeBatchMax + 1];  // first workgroup of each item; wg0[n] = the launch's workgroups
  int n;
};
hipError_t launch_lora_merge_batch(MergeBatch b, hipStream_t s);
// Value head: values[r] = sum_k u[r, k] * head[k] for R rows of u (bf16,
// frag layout with K = d) and head bf16 [d]; fp32, fixed summation order.
hipError_t launch_value_head(const bf16_t* u, int R, int d, const bf16_t* head, float* values, hipStream_t s);
// Learning phase.  GAE over a window of n_steps steps of n_env environments,
// time-major: rewards [M, N], values [M + 1, N] (row M the bootstrap value),
// dones [M + 1, N] (row t = d_t; transition t continues iff d_{t+1} == 0);
// advantages and returns (may be null) [M, N].
struct GaeArgs {
  const float* rewards;
  const float* values;
  const uint8_t* dones;
  int n_env, n_steps;
  float gamma, lam;
  float* advantages;
  float* returns;
};
hipError_t launch_gae(const GaeArgs& a, hipStream_t s);
// PPO-clip over n actions of n_tokens tokens: stats[0] = -mean surrogate,
// stats[1] = clipped fraction, dlogp [n, n_tokens] = d stats[0] / d logp_new.
struct PpoArgs {
  const float* logp_new;
  const float* logp_old;
  const float* advantages;
  int n, n_tokens;
  float eps;
  float* stats;
  float* dlogp;
};
hipError_t launch_ppo_clip(const PpoArgs& a, hipStream_t s);
// dlogits[r, j] = dlogp[r] (1[j = k_r] - softmax(z_r / T)_j) / T, k_r = tokens[r] - action_begin
// (a token outside [0, bins) gives a NaN row); bins <= 256.
struct LogprobBwdArgs {
  const float* logits;
  const int32_t* tokens;
  const float* dlogp;
  int rows, bins, action_begin;
  float temperature;
  float* dlogits;
};
hipError_t launch_logprob_backward(const LogprobBwdArgs& a, hipStream_t s);

// Action extraction: actions[r, i] = lo[i] + (k + 1/2) (hi[i] - lo[i]) / bins, k = tokens[r, i] - action_begin
// (NaN outside the bins); tokens and actions [n, n_dims].
hipError_t launch_extract_actions(const int32_t* tokens, int n, int n_dims, int action_begin, int bins,
                                  const float* lo, const float* hi, float* actions, hipStream_t s);
// Gather R rows: xc[i] = x[rows[i]] (fp32, d columns) and row i of oc = row rows[i] of o
// (both bf16 frag layout with K = d; d % 8 == 0).
hipError_t launch_gather_rows(const float* x, const bf16_t* o, const int32_t* rows, int R, int d, float* xc,
                              bf16_t* oc, hipStream_t s);
// Backward of the teacher-forced pass.
// dst (bf16 frag [R, kdst]) = fp32 row-major x (row stride ld), columns >= n zero
hipError_t launch_to_frag(const float* x, int ld, int R, int n, int kdst, bf16_t* dst, hipStream_t s);
// dst (bf16 frag [K rows, Kd]) = transpose of src [R, K]: fp32 row-major (src_f32, row
// stride ld) or bf16 frag of frag width ld; columns R .. Kd zero (Kd % 32 == 0, Kd >= R)
hipError_t launch_transpose_frag(const void* src, bool src_f32, int ld, int R, int K, int Kd, bf16_t* dst,
                                 hipStream_t s);
// dx = dres + RMSNorm backward of dy at x (gain g), one row per workgroup; dres, dx_frag may be null
hipError_t launch_rmsnorm_bwd(const float* x, const float* g, float eps, const float* dy, const float* dres,
                              float* dx, bf16_t* dx_frag, int M, int d, hipStream_t s);
// SwiGLU backward from the fp32 interleaved gate/up pre-activations and dh: d[g; up] (bf16 frag,
// K = 2 Fp, the packed interleaved order) and the forward h (bf16 frag, K = Fp)
hipError_t launch_swiglu_bwd(const float* cgu, int ldc, const float* dh, int ldh, int M, int F, int Fp, bf16_t* dgu,
                             bf16_t* h, hipStream_t s);
struct AttnBwdArgs {
  const bf16_t* q;        // [M, d] rotated queries of the forward
  const bf16_t* o;        // [M, d] attention output of the forward (bf16 frag, K = d)
  const float* dout;      // [M, d] gradient of the attention output
  KvCache kv;             // rotated keys and values of the forward
  const int32_t* page_table;
  int max_pages;
  const int32_t* env_row0;
  const int32_t* env_len;  // <= 320 rows (max_pages <= 64)
  int n_env, d, n_heads, head_dim;
  float scale;
  const float2* rope;     // [pos][head_dim / 2] (cos, sin)
  float* stats;           // [M, n_heads, 2]: log-sum-exp of each query row (from the forward's
                          // PrefillAttnArgs::lse) in, D_t = dO_t . O_t written by the first pass
  bf16_t* dqkv;           // [M, 3 d] bf16 frag (K = 3 d): gradients of q, k (before rotation, packed order), v
  bf16_t* do16;           // [M, d] row-major scratch: dO rounded to bf16 (written by the first pass)
};
hipError_t launch_attn_bwd(const AttnBwdArgs& a, hipStream_t s);
// LoRA gradients of one projection by the low-rank route: with X its input rows and
// dY the gradient of its output rows, dB = s dY^T (X A^T) and dA = s (dY B)^T X on the
// skinny GEMM (r <= 64 output rows), the four products chained through bf16 frag operands.
struct LoraGradArgs {
  int o0, n_cols;    // this projection's columns o0 .. o0 + n_cols of the packed output order
  int in, out;       // natural sizes of the projection
  int mode, head_dim, part;  // PackMode of its packed rows; part 0 gate / 1 up for kPackGateUp
  const bf16_t* a;   // [r, in] row-major
  const bf16_t* b;   // [out, r] row-major
  int r;             // 1 .. 64
  float scale;
  float* da;         // [r, in] fp32 out
  float* db;         // [out, r] fp32 out
};
// B^T as a bf16 frag [rows, K] operand: row c, column o0 + o = B[natural row of packed
// output o, c] for o < n_cols, c < r; zero elsewhere (K % 32 == 0, rows % 16 == 0, r <= rows <= 128)
hipError_t launch_pack_bt(const LoraGradArgs& a, int K, int rows, bf16_t* dst, hipStream_t s);
// dB[natural row of o, c] = s C[c, o] for o < n_cols (to_b), or dA[c, i] = s C[c, i] for i < in;
// C fp32 [64, ldc] row-major
hipError_t launch_lora_finalize(const LoraGradArgs& a, const float* C, int ldc, bool to_b, hipStream_t s);
// fp32 rows of d: dst[rows[i]] = src[i] (scatter) or dst[i] = src[rows[i]] (gather), i < R
hipError_t launch_move_rows(const float* src, const int32_t* rows, int R, int d, float* dst, bool scatter,
                            hipStream_t s);
hipError_t launch_bf16_to_f32(float* dst, const bf16_t* src, int n, hipStream_t s);
hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s);

}  // namespace vla
