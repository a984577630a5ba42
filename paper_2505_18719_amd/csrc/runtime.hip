// Host runtime of the VLA library: C ABI, argument validation, workspace
// layout, one-time weight repacking, ragged-batch metadata and page tables,
// and the launch sequences of prefill, KV-cached action decode and the
// teacher-forced pass.  No device memory is allocated here: every buffer is a
// slice of the caller's workspace.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"
#include "kernels.h"
#include "vla.h"
#include "vla_learn.h"

using namespace vla;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

}  // namespace

int vla::set_error(int code, const char* msg) { return fail(code, msg); }

namespace {

#define VLA_CK(expr)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(VLA_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr int kMaxSplits = 16;
constexpr int kSkinnyRows = 128;
constexpr int kMetaRing = 4;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int round_up(int v, int a) { return (v + a - 1) / a * a; }

// Sizes derived from a configuration.
struct Dims {
  int d, H, hd, F, Fp, A, Ap, V, L, nact, nvis;
  int Bmax, Smax, max_pages, n_pages;
  size_t Mmax;      // packed rows of the largest pass
  int Nmax;         // widest skinny GEMM
  size_t meta_ints;
};

int check_config(const vla_config* c, Dims* o) {
  if (!c) return fail(VLA_EINVAL, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->head_dim < 1 || c->d_ffn < 1 || c->vocab < 1 ||
      c->action_bins < 1 || c->n_actions < 1 || c->n_visual < 0 || c->max_batch < 1 || c->max_seq < 1)
    return fail(VLA_EINVAL, "config has a non-positive size");
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(VLA_EUNSUPPORTED, "head_dim must be 64 or 128");
  if (c->d_model != c->n_heads * c->head_dim) return fail(VLA_EINVAL, "d_model != n_heads * head_dim");
  if (c->d_model > 8192 || c->d_model % 256 != 0)
    return fail(VLA_EUNSUPPORTED, "d_model must be a multiple of 256, at most 8192");
  if (c->action_bins > 256) return fail(VLA_EUNSUPPORTED, "action_bins must be <= 256");
  if (c->action_begin < 0 || c->action_begin + c->action_bins > c->vocab)
    return fail(VLA_EINVAL, "action range outside the vocabulary");
  if (c->n_actions > 16) return fail(VLA_EUNSUPPORTED, "n_actions must be <= 16");
  if (c->page_size != kPage) return fail(VLA_EUNSUPPORTED, "page_size must be 16");
  if (c->max_seq > 320) return fail(VLA_EUNSUPPORTED, "max_seq must be <= 320");
  if (c->max_seq < c->n_visual + c->n_actions + (c->n_visual == 0 ? 1 : 0))
    return fail(VLA_EINVAL, "max_seq smaller than n_visual + n_actions");
  if (c->max_batch > 512) return fail(VLA_EUNSUPPORTED, "max_batch must be <= 512");
  if (!(c->rope_base > 1.f) || !(c->rms_eps >= 0.f)) return fail(VLA_EINVAL, "bad rope_base or rms_eps");
  Dims& D = *o;
  D.d = c->d_model;
  D.H = c->n_heads;
  D.hd = c->head_dim;
  D.F = c->d_ffn;
  D.Fp = round_up(c->d_ffn, 256);  // decode GEMM K units are 256 wide
  D.A = c->action_bins;
  D.Ap = round_up(c->action_bins, 64);
  D.V = c->vocab;
  D.L = c->n_layers;
  D.nact = c->n_actions;
  D.nvis = c->n_visual;
  D.Bmax = c->max_batch;
  D.Smax = c->max_seq;
  D.max_pages = (c->max_seq + kPage - 1) / kPage;
  D.n_pages = D.max_pages * D.Bmax;
  D.Mmax = (size_t)D.Bmax * D.Smax;
  D.Nmax = std::max(std::max(3 * D.d, 2 * D.Fp), D.Ap);
  D.meta_ints = 2 * D.Mmax + 5 * (size_t)D.Bmax + (size_t)D.Bmax * D.max_pages +
                (size_t)D.Bmax * D.nact;
  return VLA_OK;
}

// Workspace layout; with base == nullptr only the size is computed.
struct Layout {
  size_t off = 0;
  char* base = nullptr;
  template <class T>
  T* take(size_t count) {
    off = align_up(off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

struct LayerW {
  bf16_t *wqkv, *wo, *wgu, *wd;
  float *attn_norm, *mlp_norm;
};

}  // namespace

struct vla_model {
  vla_config cfg;
  Dims D;
  bf16_t* emb;
  bf16_t* lm_act;  // [Ap, d], rows past A are zero
  float* final_norm;
  std::vector<LayerW> lw;
  std::vector<KvCache> kv;
  float2* rope;
  float* x;
  bf16_t* u;
  bf16_t* q;
  bf16_t* h;
  float* part;
  float* logits_pre;  // [Bmax, A]
  float* logits_dec;  // [Bmax, A]
  float* logits_tf;   // [Bmax * nact, A]
  bf16_t* u_head;     // [Bmax * nact, d]
  // the last layer's rows that are read afterwards (at most Bmax * nact), compacted
  float* xc;          // residual [Bmax * nact, d]
  bf16_t* uc;         // attention output / norm output, frag layout
  bf16_t* hc;         // SwiGLU output, frag layout (K = Fp)
  int32_t* next_tok;  // [Bmax]
  uint32_t* flags;
  int32_t* meta_dev;
  // pinned host staging of the per-call metadata: a ring of kMetaRing buffers, so that the
  // host waits for a buffer's upload only when it runs kMetaRing calls ahead of the device
  int32_t* meta_host;  // kMetaRing * meta_ints
  hipEvent_t meta_event[kMetaRing];
  bool meta_pending[kMetaRing];
  int meta_slot;
  // device views into meta_dev
  int32_t *row_pos, *row_env, *env_row0, *env_len, *env_prefix, *env_prompt_off, *env_q0, *page_table, *head_rows;
  // decode state
  int state_batch;
  bool state_valid;
  std::vector<int> prefix_host;  // L_b of the last prefill
  int layer_limit;               // test hook: run only the first layer_limit layers (0 = all)
  int debug_stop;                // test hook: with a layer limit, where the last layer run stops (0 = its end)
  float scale;
  // decode GEMM work splits (one persistent workgroup per CU)
  SkinnyPlan plan_qkv, plan_o, plan_gu, plan_d, plan_head;
  int cus;  // compute units: the skinny GEMM's persistent grid
  // persistent decode layer kernel: its buffers, and whether the device runs it
  float *part_o, *part_gu, *part_dn, *part_nx;  // split-K partials of each projection of a layer launch
  bf16_t *dec_ua, *dec_ub;                      // [Bmax, d] frag: MLP norm output, next norm output
  unsigned* dec_bar;                            // barrier block (zeroed per decode call)
  bool fused_ok;                                // cooperative launch of one workgroup per CU is possible
  int decode_path;                              // test hook: 1 = persistent layer kernel, 0 = per-kernel (default)
  unsigned long long* trace_buf;                // test hook: phase stamps of one layer launch, or null
  int trace_layer;
  // live profiling
  struct ProfSlot {
    hipEvent_t a, b;
    int cat;
    double work;
  };
  std::vector<ProfSlot> prof;
  int prof_used;
  uint32_t prof_mask;
};

namespace {

void plan(Layout& L, vla_model* m, const Dims& D, int n_layers) {
  vla_model tmp;
  vla_model& M = m ? *m : tmp;
  M.emb = L.take<bf16_t>((size_t)D.V * D.d);
  M.lm_act = L.take<bf16_t>(frag_elems(D.Ap, D.d));
  M.final_norm = L.take<float>(D.d);
  M.lw.resize(n_layers);
  M.kv.resize(n_layers);
  for (int l = 0; l < n_layers; ++l) {
    LayerW& w = M.lw[l];
    w.wqkv = L.take<bf16_t>(frag_elems(3 * D.d, D.d));
    w.wo = L.take<bf16_t>(frag_elems(D.d, D.d));
    w.wgu = L.take<bf16_t>(frag_elems(2 * D.Fp, D.d));
    w.wd = L.take<bf16_t>(frag_elems(D.d, D.Fp));
    w.attn_norm = L.take<float>(D.d);
    w.mlp_norm = L.take<float>(D.d);
  }
  const size_t kv_elems = (size_t)D.n_pages * D.H * kPage * D.hd;
  for (int l = 0; l < n_layers; ++l) {
    M.kv[l].k = L.take<bf16_t>(kv_elems);
    M.kv[l].v = L.take<bf16_t>(kv_elems);
  }
  M.rope = L.take<float2>((size_t)D.Smax * (D.hd / 2));
  M.x = L.take<float>(D.Mmax * D.d);
  M.u = L.take<bf16_t>(frag_elems(D.Mmax, D.d));  // activations in frag layout
  M.q = L.take<bf16_t>(D.Mmax * D.d);
  M.h = L.take<bf16_t>(frag_elems(D.Mmax, D.Fp));
  M.part = L.take<float>((size_t)kMaxSplits * kSkinnyRows * D.Nmax);
  M.logits_pre = L.take<float>((size_t)D.Bmax * D.A);
  M.logits_dec = L.take<float>((size_t)D.Bmax * D.A);
  M.logits_tf = L.take<float>((size_t)D.Bmax * D.nact * D.A);
  M.u_head = L.take<bf16_t>(frag_elems((size_t)D.Bmax * D.nact, D.d));
  M.xc = L.take<float>((size_t)D.Bmax * D.nact * D.d);
  M.uc = L.take<bf16_t>(frag_elems((size_t)D.Bmax * D.nact, D.d));
  M.hc = L.take<bf16_t>(frag_elems((size_t)D.Bmax * D.nact, D.Fp));
  M.next_tok = L.take<int32_t>(D.Bmax);
  M.flags = L.take<uint32_t>(4);
  // persistent decode layer: one partial region per projection of a launch (each is read
  // once per launch, so none needs cache maintenance between its phases)
  M.part_o = L.take<float>((size_t)kMaxSplits * kSkinnyRows * D.d);
  M.part_gu = L.take<float>((size_t)kMaxSplits * kSkinnyRows * 2 * D.Fp);
  M.part_dn = L.take<float>((size_t)kMaxSplits * kSkinnyRows * D.d);
  M.part_nx = L.take<float>((size_t)kMaxSplits * kSkinnyRows * std::max(3 * D.d, D.Ap));
  M.dec_ua = L.take<bf16_t>(frag_elems(D.Bmax, D.d));
  M.dec_ub = L.take<bf16_t>(frag_elems(D.Bmax, D.d));
  M.dec_bar = L.take<unsigned>(256);
  M.meta_dev = L.take<int32_t>(D.meta_ints);
  L.off = align_up(L.off, 256);
}

size_t kv_region_bytes(const Dims& D, int n_layers) {
  return align_up((size_t)D.n_pages * D.H * kPage * D.hd * sizeof(bf16_t), 256) * 2 * n_layers;
}

void set_meta_views(vla_model* m, int32_t* base) {
  const Dims& D = m->D;
  int32_t* p = base;
  m->row_pos = p; p += D.Mmax;
  m->row_env = p; p += D.Mmax;
  m->env_row0 = p; p += D.Bmax;
  m->env_len = p; p += D.Bmax;
  m->env_prefix = p; p += D.Bmax;
  m->env_prompt_off = p; p += D.Bmax;
  m->env_q0 = p; p += D.Bmax;
  m->page_table = p; p += (size_t)D.Bmax * D.max_pages;
  m->head_rows = p;
}

// Index of a view inside the meta block (same for host staging and device).
template <class T>
size_t meta_index(const vla_model* m, const T* view) {
  return (size_t)(view - m->meta_dev);
}

RowMeta row_meta(const vla_model* m) { return RowMeta{m->row_pos, m->row_env, m->page_table, m->D.max_pages}; }

constexpr int kProfSlots = 16384;

// Start event of a profiled launch; returns the slot or -1 when not recorded.
int prof_start(vla_model* m, int cat, hipStream_t s) {
  if (!(m->prof_mask & (1u << cat)) || m->prof_used >= (int)m->prof.size()) return -1;
  const int i = m->prof_used++;
  m->prof[i].cat = cat;
  m->prof[i].work = 0.0;
  (void)hipEventRecord(m->prof[i].a, s);
  return i;
}

void prof_stop(vla_model* m, int slot, double work, hipStream_t s) {
  if (slot < 0) return;
  m->prof[slot].work = work;
  (void)hipEventRecord(m->prof[slot].b, s);
}

// Profiled launch wrapper: evaluates `launch` between the two events.
#define PROF_LAUNCH(cat, work, launch)              \
  do {                                              \
    const int slot_ = prof_start(m, (cat), s);      \
    VLA_CK(launch);                                 \
    prof_stop(m, slot_, (work), s);                 \
  } while (0)

double gemm_flops(double M, double N, double K) { return 2.0 * M * N * K; }
// algorithmic HBM bytes of a decode GEMM: the weights once plus the activations in
double skinny_bytes(double N, double K, double M) { return 2.0 * N * K + 2.0 * M * K; }

// Skinny GEMM over up to kSkinnyRows rows, followed by the logits reduction.
int head_logits(vla_model* m, const bf16_t* u, int R, float* logits, hipStream_t s) {
  const Dims& D = m->D;
  for (int r0 = 0; r0 < R; r0 += kSkinnyRows) {
    const int rows = std::min(kSkinnyRows, R - r0);
    SkinnyArgs sa{u + frag_index(r0, 0, D.d), rows, m->lm_act, D.Ap, D.d, m->part};
    VLA_CK(launch_skinny(sa, m->plan_head, s));
    VLA_CK(launch_reduce_sum(m->part, m->plan_head, logits + (size_t)r0 * D.A, rows, D.A, s));
  }
  return VLA_OK;
}

// One decode step (token position prefix + step - 1) on the persistent layer
// kernel: the token's embedding and first RMSNorm, layer 0's QKV projection,
// then per layer the decode attention (with the QKV consumer) and one
// decode_layer launch (everything after attention plus the next projection;
// after the last layer the action head's), and the head's reduction into
// logits_dec.  The arithmetic is that of the per-kernel path.
int decode_step_fused(vla_model* m, int B, int step, unsigned& bar_base, hipStream_t s) {
  const Dims& D = m->D;
  const float eps = m->cfg.rms_eps;
  VLA_CK(launch_embed_token_norm(m->next_tok, m->emb, m->x, m->dec_ub, m->lw[0].attn_norm, eps, B, D.d, D.V,
                                 m->flags, s));
  for (int r0 = 0; r0 < B; r0 += kSkinnyRows) {
    const int rows = std::min(kSkinnyRows, B - r0);
    float* x = m->x + (size_t)r0 * D.d;
    bf16_t* o = m->u + frag_index(r0, 0, D.d);  // r0 is a multiple of 16: whole frag blocks
    bf16_t* ua = m->dec_ua + frag_index(r0, 0, D.d);
    bf16_t* ub = m->dec_ub + frag_index(r0, 0, D.d);
    bf16_t* h = m->h + frag_index(r0, 0, D.Fp);
    const int32_t* ptab = m->page_table + (size_t)r0 * D.max_pages;
    const int32_t* eprefix = m->env_prefix + r0;
    double kv_bytes = 0.0;
    for (int b = r0; b < r0 + rows; ++b) kv_bytes += 2.0 * 2.0 * D.d * (double)(m->prefix_host[b] + step);
    SkinnyArgs sq{ub, rows, m->lw[0].wqkv, 3 * D.d, D.d, m->part_nx};
    PROF_LAUNCH(VLA_PROF_DECODE_GEMM, skinny_bytes(3.0 * D.d, D.d, rows), launch_skinny(sq, m->plan_qkv, s));
    for (int l = 0; l < D.L; ++l) {
      const LayerW& w = m->lw[l];
      DecodeAttnArgs da{m->part_nx, m->plan_qkv, m->rope, o, m->kv[l], ptab, D.max_pages, eprefix,
                        step, rows, D.d, D.H, D.hd, m->scale};
      PROF_LAUNCH(VLA_PROF_DECODE_ATTN, kv_bytes, launch_attn_decode(da, s));
      const bool last = l + 1 == D.L;
      DecodeLayerArgs a{};
      a.o = SkinnyArgs{o, rows, w.wo, D.d, D.d, m->part_o};
      a.gu = SkinnyArgs{ua, rows, w.wgu, 2 * D.Fp, D.d, m->part_gu};
      a.dn = SkinnyArgs{h, rows, w.wd, D.d, D.Fp, m->part_dn};
      a.nx = last ? SkinnyArgs{ub, rows, m->lm_act, D.Ap, D.d, m->part_nx}
                  : SkinnyArgs{ub, rows, m->lw[l + 1].wqkv, 3 * D.d, D.d, m->part_nx};
      a.p_o = m->plan_o; a.p_gu = m->plan_gu; a.p_dn = m->plan_d; a.p_nx = last ? m->plan_head : m->plan_qkv;
      a.x = x; a.g_mlp = w.mlp_norm; a.g_next = last ? m->final_norm : m->lw[l + 1].attn_norm;
      a.ua = ua; a.h = h; a.ub = ub;
      a.M = rows; a.d = D.d; a.Fp = D.Fp; a.eps = eps;
      a.bar = m->dec_bar; a.bar_base = bar_base; a.flags = m->flags;
      a.trace = (step == 1 && l == m->trace_layer && r0 == 0) ? m->trace_buf : nullptr;
      bar_base += kDecodeLayerBarriers;
      // algorithmic bytes: the four projections' weights (real F) and activations once
      const double bytes = skinny_bytes(D.d, D.d, rows) + skinny_bytes(2.0 * D.F, D.d, rows) +
                           skinny_bytes(D.d, D.F, rows) +
                           (last ? skinny_bytes(D.A, D.d, rows) : skinny_bytes(3.0 * D.d, D.d, rows));
      PROF_LAUNCH(VLA_PROF_DECODE_LAYER, bytes, launch_decode_layer(a, m->cus, s));
    }
    VLA_CK(launch_reduce_sum(m->part_nx, m->plan_head, m->logits_dec + (size_t)r0 * D.A, rows, D.A, s));
  }
  return VLA_OK;
}

// Shared forward over a packed ragged batch: prefill (actions == nullptr) or
// teacher-forced (each environment's rows extended by its action tokens).
// save_x (training): per-layer device buffers that receive each layer's input
// residual; a training pass computes every row of the last layer.
// Activations a training forward keeps per layer: the layer input always; with
// `full` also everything the backward would otherwise recompute from it.
struct SavedActs {
  std::vector<float*> xs;              // input residual [Mmax, d]
  bool full = false;
  std::vector<bf16_t*> u1, q, ob, u2;  // attention-norm output (frag), rotated queries (row-major),
                                       // attention output (frag), MLP-norm output (frag)
  std::vector<float*> xm, cgu, lse;    // mid residual [Mmax, d], gate/up pre-activations
                                       // [Mmax, 2 Fp] (interleaved), log-sum-exp stats [Mmax, H, 2]
};

int forward(vla_model* m, int B, const void* vis, const int32_t* prompt_ids, const int32_t* lens_host,
            const int32_t* actions, hipStream_t s, int* out_rows, const SavedActs* sv = nullptr,
            int* out_M = nullptr) {
  const Dims& D = m->D;
  const bool tf = actions != nullptr;
  std::vector<int> prefix(B), rows(B);
  size_t M = 0;
  for (int b = 0; b < B; ++b) {
    if (lens_host[b] < 0) return fail(VLA_EINVAL, "negative prompt length");
    prefix[b] = D.nvis + lens_host[b];
    if (prefix[b] < 1) return fail(VLA_EINVAL, "empty sequence (n_visual + prompt length == 0)");
    if (prefix[b] + D.nact > D.Smax) return fail(VLA_ESHAPE, "n_visual + prompt + n_actions exceeds max_seq");
    rows[b] = prefix[b] + (tf ? D.nact : 0);
    M += rows[b];
  }
  // host metadata -> pinned staging (the next buffer of the ring) -> one async upload
  const int ms = m->meta_slot;
  m->meta_slot = (ms + 1) % kMetaRing;
  if (m->meta_pending[ms]) {  // this buffer's previous upload: kMetaRing calls ago
    VLA_CK(hipEventSynchronize(m->meta_event[ms]));
    m->meta_pending[ms] = false;
  }
  int32_t* h = m->meta_host + (size_t)ms * D.meta_ints;
  int32_t* hp = h + meta_index(m, m->row_pos);
  int32_t* he = h + meta_index(m, m->row_env);
  int32_t* hr0 = h + meta_index(m, m->env_row0);
  int32_t* hl = h + meta_index(m, m->env_len);
  int32_t* hpre = h + meta_index(m, m->env_prefix);
  int32_t* hpo = h + meta_index(m, m->env_prompt_off);
  int32_t* hq0 = h + meta_index(m, m->env_q0);
  int32_t* hpt = h + meta_index(m, m->page_table);
  int32_t* hh = h + meta_index(m, m->head_rows);
  size_t r = 0;
  int po = 0;
  for (int b = 0; b < B; ++b) {
    hr0[b] = (int32_t)r;
    hl[b] = rows[b];
    hpre[b] = prefix[b];
    hq0[b] = prefix[b] - 1;  // the rows read after the last layer start at the last prefix row
    hpo[b] = po;
    po += lens_host[b];
    for (int t = 0; t < rows[b]; ++t, ++r) {
      hp[r] = t;
      he[r] = b;
    }
    // pages of env b are interleaved with the other environments' pages
    const int np = (prefix[b] + D.nact + kPage - 1) / kPage;
    for (int p = 0; p < D.max_pages; ++p) hpt[(size_t)b * D.max_pages + p] = p < np ? p * B + b : 0;
    if (tf) {
      for (int i = 0; i < D.nact; ++i) hh[b * D.nact + i] = hr0[b] + prefix[b] - 1 + i;
    } else {
      hh[b] = hr0[b] + prefix[b] - 1;
    }
  }
  VLA_CK(hipMemcpyAsync(m->meta_dev, h, D.meta_ints * sizeof(int32_t), hipMemcpyHostToDevice, s));
  VLA_CK(hipEventRecord(m->meta_event[ms], s));
  m->meta_pending[ms] = true;

  const int Mi = (int)M;
  // causal attention flops of one layer: q.k and p.v over (t + 1) keys per row
  double attn_flops = 0.0;
  for (int b = 0; b < B; ++b) attn_flops += 2.0 * D.d * (double)rows[b] * (rows[b] + 1);
  EmbedArgs ea{m->x, m->emb, static_cast<const bf16_t*>(vis), prompt_ids, actions, m->row_pos, m->row_env,
               m->env_prefix, m->env_prompt_off, Mi, D.d, D.nvis, D.nact, D.V, m->flags};
  VLA_CK(launch_embed(ea, s));
  const float eps = m->cfg.rms_eps;
  // the prefill GEMMs read their activations (u, attention output, h) in frag layout
  const bool full = sv && sv->full;
  VLA_CK(launch_rmsnorm(m->x, D.d, nullptr, m->lw[0].attn_norm, eps, full ? sv->u1[0] : m->u, D.d, Mi, D.d, s, true));
  const int n_layers = m->layer_limit > 0 ? std::min(m->layer_limit, D.L) : D.L;
  // Only the rows read afterwards (head_rows: the last prefix row, or the n_actions
  // scoring rows, of each environment) need the last layer's output; its other rows
  // only feed the KV cache through the QKV projection.  Every row's computation is
  // independent of which other rows run with it, so results are the same bits.
  // (A layer limit set through the debug interface computes every row.)
  const bool prune = m->layer_limit == 0 && sv == nullptr;
  const int R = tf ? B * D.nact : B;
  double attn_flops_last = 0.0;  // q.k and p.v of the needed query rows only
  for (int b = 0; b < B; ++b)
    for (int t = prefix[b] - 1; t < rows[b]; ++t) attn_flops_last += 4.0 * D.d * (t + 1);
  for (int l = 0; l < n_layers; ++l) {
    const LayerW& w = m->lw[l];
    const bool last = prune && l == D.L - 1;
    // debug stop points inside the last layer of a limited pass (every buffer read afterwards holds that stage)
    const int stop = m->layer_limit > 0 && l == n_layers - 1 ? m->debug_stop : 0;
    if (stop == 1) break;  // u: the attention norm's output, x: the layer input
    // keep mode chains the residual stream through the kept buffers (x_l -> xm_l -> x_{l+1}, the
    // residual epilogues reading one and writing the next); otherwise it is updated in place
    if (sv && !(full && l > 0))
      VLA_CK(hipMemcpyAsync(sv->xs[l], m->x, (size_t)Mi * D.d * sizeof(float), hipMemcpyDeviceToDevice, s));
    bf16_t* const qb = full ? sv->q[l] : m->q;
    GemmArgs g{};
    g.A = full ? sv->u1[l] : m->u; g.W = w.wqkv; g.M = Mi; g.N = 3 * D.d; g.K = D.d;
    g.q = qb; g.ldq = D.d; g.kv = m->kv[l]; g.meta = row_meta(m); g.rope = m->rope;
    g.d_model = D.d; g.n_heads = D.H; g.head_dim = D.hd;
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(Mi, 3.0 * D.d, D.d), launch_gemm(g, kEpiQkvRope, s));
    PrefillAttnArgs pa{qb, full ? sv->ob[l] : m->u, m->kv[l], m->page_table, D.max_pages, m->env_row0, m->env_len,
                       B, D.d, D.H, D.hd, m->scale, last ? m->env_q0 : nullptr, full ? sv->lse[l] : nullptr};
    PROF_LAUNCH(VLA_PROF_PREFILL_ATTN, last ? attn_flops_last : attn_flops, launch_attn_prefill(pa, s));
    if (stop == 2) break;  // u: the attention output; q and the layer's K/V pages written
    // the rest of the layer runs on all rows, or on the compacted needed rows of the last layer
    const int Ml = last ? R : Mi;
    float* x = m->x;
    bf16_t* u = full ? sv->ob[l] : m->u;
    bf16_t* hbuf = m->h;
    if (last) {
      VLA_CK(launch_gather_rows(m->x, m->u, m->head_rows, R, D.d, m->xc, m->uc, s));
      x = m->xc;
      u = m->uc;
      hbuf = m->hc;
    }
    GemmArgs go{};
    go.A = u; go.W = w.wo; go.M = Ml; go.N = D.d; go.K = D.d; go.C = x; go.ldc = D.d;
    if (full) {
      go.R = sv->xs[l];
      go.C = x = sv->xm[l];
    }
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(Ml, D.d, D.d), launch_gemm(go, kEpiResidual, s));
    if (full) u = sv->u2[l];
    VLA_CK(launch_rmsnorm(x, D.d, nullptr, w.mlp_norm, eps, u, D.d, Ml, D.d, s, true));
    if (stop == 3) break;  // x: the mid residual, u: the MLP norm's output
    GemmArgs gg{};
    // [gate; up] interleaved in 64-row blocks: only the blocks holding real rows are computed; the
    // down projection's contraction stops at the last real feature (h and Wdown stay Fp wide)
    gg.A = u; gg.W = w.wgu; gg.M = Ml; gg.N = 64 * ((D.F + 31) / 32); gg.K = D.d; gg.H = hbuf; gg.ldh = D.Fp;
    if (full) {  // h, and the fp32 pre-activations kept for the backward
      gg.C = sv->cgu[l]; gg.ldc = 2 * D.Fp;
      PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(Ml, 2.0 * D.F, D.d), launch_gemm(gg, kEpiSwiGluKeep, s));
    } else {
      PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(Ml, 2.0 * D.F, D.d), launch_gemm(gg, kEpiSwiGlu, s));
    }
    GemmArgs gd{};
    gd.A = hbuf; gd.W = w.wd; gd.M = Ml; gd.N = D.d; gd.K = 32 * ((D.F + 31) / 32); gd.ka = D.Fp; gd.kw = D.Fp;
    gd.C = x; gd.ldc = D.d;
    if (full) {
      gd.R = sv->xm[l];
      gd.C = x = l + 1 < D.L ? sv->xs[l + 1] : m->x;
    }
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(Ml, D.d, D.F), launch_gemm(gd, kEpiResidual, s));
    if (l + 1 < D.L)
      VLA_CK(launch_rmsnorm(x, D.d, nullptr, m->lw[l + 1].attn_norm, eps, full ? sv->u1[l + 1] : m->u, D.d, Mi, D.d,
                            s, true));
  }
  if (prune)
    VLA_CK(launch_rmsnorm(m->xc, D.d, nullptr, m->final_norm, eps, m->u_head, D.d, R, D.d, s, true));
  else
    VLA_CK(launch_rmsnorm(m->x, D.d, m->head_rows, m->final_norm, eps, m->u_head, D.d, R, D.d, s, true));
  *out_rows = R;
  if (out_M) *out_M = Mi;
  return VLA_OK;
}

// ---- training (backward of the teacher-forced pass) --------------------------
// Buffers of the caller's training workspace.
struct TrainBufs {
  SavedActs sv;  // what the forward keeps per layer
  float *dx, *dxm, *du, *dob, *xm, *cgu, *dh, *stats, *dz, *du_h, *xc, *dxc, *logp, *dlogp;
  float *t1, *t2, *cres, *spart;  // low-rank products and skinny-GEMM partials
  bf16_t *dxf, *dxmf, *u1, *ob, *u2, *hb, *dgu, *dqkv, *wt, *xt, *dyt, *dzf, *wact_t, *apk, *bpt, *t1f, *t2f, *do16;
};

// keep: every layer's activations are kept by the forward (no recompute in the backward)
void plan_train(Layout& L, const Dims& D, TrainBufs& t, bool keep) {
  const size_t Mx = D.Mmax, d = D.d;
  // rows padded to 64 (the skinny GEMM's column tiles run over them), the
  // row contraction padded to 256 (its K units)
  const size_t Mx64 = round_up((int)D.Mmax, 64);
  const int A32 = round_up(D.A, 32), Mk = round_up((int)D.Mmax, 256);
  const int Fg = 64 * ((D.F + 31) / 32), F64 = round_up(D.F, 64);
  const size_t Rh = (size_t)D.Bmax * D.nact;
  SavedActs& sv = t.sv;
  sv.full = keep;
  sv.xs.resize(D.L);
  for (int l = 0; l < D.L; ++l) sv.xs[l] = L.take<float>(Mx * d);
  if (keep) {
    for (int l = 0; l < D.L; ++l) {
      sv.u1.push_back(L.take<bf16_t>(frag_elems(Mx64, d)));
      sv.q.push_back(L.take<bf16_t>(Mx * d));
      sv.ob.push_back(L.take<bf16_t>(frag_elems(Mx64, d)));
      sv.u2.push_back(L.take<bf16_t>(frag_elems(Mx64, d)));
      sv.xm.push_back(L.take<float>(Mx * d));
      sv.cgu.push_back(L.take<float>(Mx * 2 * D.Fp));
      sv.lse.push_back(L.take<float>(Mx * D.H * 2));
    }
    t.xm = t.cgu = t.stats = nullptr;
    t.u1 = t.ob = t.u2 = nullptr;
  } else {
    t.xm = L.take<float>(Mx * d);
    t.cgu = L.take<float>(Mx * 2 * D.Fp);
    t.stats = L.take<float>(Mx * D.H * 2);
    t.u1 = L.take<bf16_t>(frag_elems(Mx64, d));
    t.ob = L.take<bf16_t>(frag_elems(Mx64, d));
    t.u2 = L.take<bf16_t>(frag_elems(Mx64, d));
  }
  t.dx = L.take<float>(Mx * d);
  t.dxm = L.take<float>(Mx * d);
  t.du = L.take<float>(Mx * d);
  t.dob = L.take<float>(Mx * d);
  t.dh = L.take<float>(Mx * D.Fp);
  t.dz = L.take<float>(Rh * D.A);
  t.du_h = L.take<float>(Rh * d);
  t.xc = L.take<float>(Rh * d);
  t.dxc = L.take<float>(Rh * d);
  t.logp = L.take<float>(Rh);
  t.dlogp = L.take<float>(Rh);
  const size_t ncol = std::max(std::max(Mx64, (size_t)Fg), std::max(d, (size_t)F64));
  // the low-rank products of up to 128 stacked factor rows (the skinny GEMM's A operand)
  t.t1 = L.take<float>(128 * Mx64);
  t.t2 = L.take<float>(128 * Mx64);
  t.cres = L.take<float>(128 * ncol);
  t.spart = L.take<float>((size_t)kMaxSplits * 128 * ncol);
  t.dxf = L.take<bf16_t>(frag_elems(Mx64, d));
  t.dxmf = L.take<bf16_t>(frag_elems(Mx64, d));
  t.hb = L.take<bf16_t>(frag_elems(Mx64, D.Fp));
  t.dgu = L.take<bf16_t>(frag_elems(Mx64, 2 * D.Fp));
  t.dqkv = L.take<bf16_t>(frag_elems(Mx64, 3 * D.d));
  t.do16 = L.take<bf16_t>(Mx * d);
  t.wt = L.take<bf16_t>(std::max(std::max(frag_elems(D.Fp, D.d), frag_elems(D.d, 2 * D.Fp)),
                                 std::max(frag_elems(D.d, D.d), frag_elems(D.d, 3 * D.d))));
  t.xt = L.take<bf16_t>(frag_elems(std::max(D.d, D.Fp), Mk));
  t.dyt = L.take<bf16_t>(frag_elems(std::max(3 * D.d, 2 * D.Fp), Mk));
  t.dzf = L.take<bf16_t>(frag_elems(Rh, A32));
  t.wact_t = L.take<bf16_t>(frag_elems(D.d, A32));
  t.apk = L.take<bf16_t>(frag_elems(128, std::max(D.d, D.Fp)));
  t.bpt = L.take<bf16_t>(frag_elems(128, std::max(3 * D.d, 2 * D.Fp)));
  t.t1f = L.take<bf16_t>(frag_elems(128, Mk));
  t.t2f = L.take<bf16_t>(frag_elems(128, Mk));
  L.off = align_up(L.off, 256);
}

// C (fp32, ldc) = A W^T on the prefill GEMM
hipError_t gemm_f32(const bf16_t* A, int ka, const bf16_t* W, int kw, int M, int N, int K, float* C, int ldc,
                    hipStream_t s) {
  GemmArgs g{};
  g.A = A; g.W = W; g.M = M; g.N = N; g.K = K; g.ka = ka; g.kw = kw; g.C = C; g.ldc = ldc;
  return launch_gemm(g, kEpiStoreF32, s);
}

// Backward of decoder layer l: t.dx holds dL/d(layer output) [M, d] and receives
// dL/d(layer input) (not for layer 0, whose input is the embeddings); LoRA gradients
// of the adapted projections are written.
int layer_backward(vla_model* m, TrainBufs& t, int l, int B, int M, const vla_lora* lora, hipStream_t s) {
  const Dims& D = m->D;
  const LayerW& w = m->lw[l];
  const float eps = m->cfg.rms_eps;
  const int d = D.d, Fp = D.Fp, F64 = round_up(D.F, 64), Fg = 64 * ((D.F + 31) / 32);
  const int Mp = round_up(M, 64), Mk = round_up(M, 256);
  const SavedActs& sv = t.sv;
  const float* const xs = sv.xs[l];
  // the layer's forward activations: kept by the forward, or recomputed here from its input
  bf16_t *u1 = t.u1, *ob = t.ob, *u2 = t.u2, *qb = m->q;
  float *xm = t.xm, *cgu = t.cgu, *stats = t.stats;
  if (sv.full) {
    u1 = sv.u1[l]; ob = sv.ob[l]; u2 = sv.u2[l]; qb = sv.q[l];
    xm = sv.xm[l]; cgu = sv.cgu[l]; stats = sv.lse[l];
  } else {
    VLA_CK(launch_rmsnorm(xs, d, nullptr, w.attn_norm, eps, u1, d, M, d, s, true));
    GemmArgs g{};
    g.A = u1; g.W = w.wqkv; g.M = M; g.N = 3 * d; g.K = d;
    g.q = qb; g.ldq = d; g.kv = m->kv[l]; g.meta = row_meta(m); g.rope = m->rope;
    g.d_model = d; g.n_heads = D.H; g.head_dim = D.hd;
    // the recompute of the layer's forward (recompute mode only) is profiled like the forward's launches
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(M, 3.0 * d, d), launch_gemm(g, kEpiQkvRope, s));
    PrefillAttnArgs pa{qb, ob, m->kv[l], m->page_table, D.max_pages, m->env_row0, m->env_len,
                       B, d, D.H, D.hd, m->scale, nullptr, stats};
    PROF_LAUNCH(VLA_PROF_PREFILL_ATTN, 0.0, launch_attn_prefill(pa, s));
    VLA_CK(hipMemcpyAsync(xm, xs, (size_t)M * d * sizeof(float), hipMemcpyDeviceToDevice, s));
    GemmArgs go{};
    go.A = ob; go.W = w.wo; go.M = M; go.N = d; go.K = d; go.C = xm; go.ldc = d;
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(M, d, d), launch_gemm(go, kEpiResidual, s));
    VLA_CK(launch_rmsnorm(xm, d, nullptr, w.mlp_norm, eps, u2, d, M, d, s, true));
    PROF_LAUNCH(VLA_PROF_PREFILL_GEMM, gemm_flops(M, 2.0 * D.F, d), gemm_f32(u2, 0, w.wgu, 0, M, Fg, d, cgu, 2 * Fp, s));
  }
  // MLP: dh = dy Wd, SwiGLU backward, du2 = d[g; up] Wgu, RMSNorm backward
  VLA_CK(launch_to_frag(t.dx, d, M, d, d, t.dxf, s));
  VLA_CK(launch_transpose_frag(w.wd, false, Fp, d, Fp, d, t.wt, s));
  VLA_CK(gemm_f32(t.dxf, 0, t.wt, 0, M, F64, d, t.dh, Fp, s));
  VLA_CK(launch_swiglu_bwd(cgu, 2 * Fp, t.dh, Fp, M, D.F, Fp, t.dgu, t.hb, s));
  VLA_CK(launch_transpose_frag(w.wgu, false, d, 2 * Fp, d, 2 * Fp, t.wt, s));
  VLA_CK(gemm_f32(t.dgu, 2 * Fp, t.wt, 2 * Fp, M, d, Fg, t.du, d, s));
  VLA_CK(launch_rmsnorm_bwd(xm, w.mlp_norm, eps, t.du, t.dx, t.dxm, t.dxmf, M, d, s));
  // attention: do = dxm Wo, attention backward, du1 = d[q; k; v] Wqkv
  VLA_CK(launch_transpose_frag(w.wo, false, d, d, d, d, t.wt, s));
  VLA_CK(gemm_f32(t.dxmf, 0, t.wt, 0, M, d, d, t.dob, d, s));
  AttnBwdArgs ab{qb, ob, t.dob, m->kv[l], m->page_table, D.max_pages, m->env_row0, m->env_len, B, d, D.H, D.hd,
                 m->scale, m->rope, stats, t.dqkv, t.do16};
  VLA_CK(launch_attn_bwd(ab, s));
  // the gradient of the first layer's input (the embeddings) feeds no trained parameter
  if (l > 0) {
    VLA_CK(launch_transpose_frag(w.wqkv, false, d, 3 * d, d, 3 * d, t.wt, s));
    VLA_CK(gemm_f32(t.dqkv, 0, t.wt, 0, M, d, 3 * d, t.du, d, s));
  }
  // LoRA gradients by the low-rank route on the skinny GEMM (<= 128 output rows; the
  // contractions over the M rows run with K = Mk, rows past M zero):
  //   T1^T = A X^T, T2^T = B^T dY^T (r x M);  dB^T = T1^T dY,  dA = T2^T X.
  // Projections that share X and dY (q, k, v; gate, up) stack their A and B^T
  // factors, 16-row aligned, into one operand, so X, dY and X^T stream once per
  // group for T1, T2 and dA.
  auto adapted = [&](int p) { return lora->a[l * 7 + p] != nullptr; };
  auto skinny_to = [&](const bf16_t* a_op, int rows, const bf16_t* w_op, int N, int K, float* out) {
    const SkinnyPlan sp = skinny_plan(N, K, m->cus, kMaxSplits);
    SkinnyArgs sa{a_op, rows, w_op, N, K, t.spart};
    hipError_t e = launch_skinny(sa, sp, s);
    return e != hipSuccess ? e : launch_reduce_sum(t.spart, sp, out, rows, N, s);
  };
  const int r16 = round_up(lora->rank, 16), per = 128 / r16;
  // one projection of a group: its packed output columns o0 .. o0 + n_cols of dY (the order
  // of `mode`), and dYT, the transposed dY rows of those columns
  struct Proj {
    int p, o0, n_cols, out, mode, part;
    const bf16_t* dYT;
  };
  // X frag [M, kx] (in real input features) with X^T rows in64 (XT); dY frag [M, ky]
  auto group = [&](const Proj* ps, int n, const bf16_t* X, int kx, int in, const bf16_t* XT, const bf16_t* dY,
                   int ky) -> hipError_t {
    hipError_t e;
    const int in64 = round_up(in, 64);
    for (int b0 = 0; b0 < n; b0 += per) {
      const int nb = std::min(per, n - b0), rows = nb * r16;
      LoraGradArgs la[3];
      for (int i = 0; i < nb; ++i) {
        const Proj& q = ps[b0 + i];
        la[i] = LoraGradArgs{q.o0, q.n_cols, in, q.out, q.mode, D.hd, q.part,
                             static_cast<const bf16_t*>(lora->a[l * 7 + q.p]),
                             static_cast<const bf16_t*>(lora->b[l * 7 + q.p]), lora->rank, lora->scale,
                             lora->grad_a[l * 7 + q.p], lora->grad_b[l * 7 + q.p]};
        PackArgs pa{t.apk + frag_index(i * r16, 0, kx), r16, kx, la[i].a, nullptr, in, lora->rank, in, kPackRows, D.hd};
        if ((e = launch_pack_frag(pa, s)) != hipSuccess) return e;
        if ((e = launch_pack_bt(la[i], ky, r16, t.bpt + frag_index(i * r16, 0, ky), s)) != hipSuccess) return e;
      }
      if ((e = skinny_to(t.apk, rows, X, Mp, kx, t.t1)) != hipSuccess) return e;
      if ((e = launch_to_frag(t.t1, Mp, rows, M, Mk, t.t1f, s)) != hipSuccess) return e;
      if ((e = skinny_to(t.bpt, rows, dY, Mp, ky, t.t2)) != hipSuccess) return e;
      if ((e = launch_to_frag(t.t2, Mp, rows, M, Mk, t.t2f, s)) != hipSuccess) return e;
      for (int i = 0; i < nb; ++i) {
        const Proj& q = ps[b0 + i];
        LoraGradArgs lb = la[i];
        lb.o0 = 0;  // q.dYT holds only this projection's rows
        if ((e = skinny_to(t.t1f + frag_index(i * r16, 0, Mk), r16, q.dYT, q.n_cols, Mk, t.cres)) != hipSuccess)
          return e;
        if ((e = launch_lora_finalize(lb, t.cres, q.n_cols, true, s)) != hipSuccess) return e;
      }
      if ((e = skinny_to(t.t2f, rows, XT, in64, Mk, t.cres)) != hipSuccess) return e;
      for (int i = 0; i < nb; ++i)
        if ((e = launch_lora_finalize(la[i], t.cres + (size_t)i * r16 * in64, in64, false, s)) != hipSuccess) return e;
    }
    return hipSuccess;
  };
  Proj ps[3];
  int n = 0;
  for (int p = VLA_PROJ_Q; p <= VLA_PROJ_V; ++p)
    if (adapted(p))
      ps[n++] = Proj{p, p * d, d, d, p == VLA_PROJ_V ? kPackRows : kPackQk, 0, t.dyt + frag_index(p * d, 0, Mk)};
  if (n) {
    VLA_CK(launch_transpose_frag(u1, false, d, M, d, Mk, t.xt, s));
    VLA_CK(launch_transpose_frag(t.dqkv, false, 3 * d, M, 3 * d, Mk, t.dyt, s));
    VLA_CK(group(ps, n, u1, d, d, t.xt, t.dqkv, 3 * d));
  }
  if (adapted(VLA_PROJ_O)) {
    VLA_CK(launch_transpose_frag(ob, false, d, M, d, Mk, t.xt, s));
    VLA_CK(launch_transpose_frag(t.dxmf, false, d, M, d, Mk, t.dyt, s));
    ps[0] = Proj{VLA_PROJ_O, 0, d, d, kPackRows, 0, t.dyt};
    VLA_CK(group(ps, 1, ob, d, d, t.xt, t.dxmf, d));
  }
  n = 0;
  for (int p = VLA_PROJ_GATE; p <= VLA_PROJ_UP; ++p)
    if (adapted(p)) ps[n++] = Proj{p, 0, Fg, D.F, kPackGateUp, p - VLA_PROJ_GATE, t.dyt};
  if (n) {
    VLA_CK(launch_transpose_frag(u2, false, d, M, d, Mk, t.xt, s));
    VLA_CK(launch_transpose_frag(t.dgu, false, 2 * Fp, M, Fg, Mk, t.dyt, s));
    VLA_CK(group(ps, n, u2, d, d, t.xt, t.dgu, 2 * Fp));
  }
  if (adapted(VLA_PROJ_DOWN)) {
    VLA_CK(launch_transpose_frag(t.hb, false, Fp, M, D.F, Mk, t.xt, s));
    VLA_CK(launch_transpose_frag(t.dxf, false, d, M, d, Mk, t.dyt, s));
    ps[0] = Proj{VLA_PROJ_DOWN, 0, d, d, kPackRows, 0, t.dyt};
    VLA_CK(group(ps, 1, t.hb, Fp, D.F, t.xt, t.dxf, d));
  }
  // dL/d(layer input) = dxm + RMSNorm backward of du1
  if (l > 0) VLA_CK(launch_rmsnorm_bwd(xs, w.attn_norm, eps, t.du, t.dxm, t.dx, nullptr, M, d, s));
  return VLA_OK;
}

}  // namespace

extern "C" {

int vla_workspace_size(const vla_config* cfg, size_t* bytes) {
  Dims D;
  int rc = check_config(cfg, &D);
  if (rc) return rc;
  if (!bytes) return fail(VLA_EINVAL, "bytes_host is NULL");
  Layout L;
  plan(L, nullptr, D, cfg->n_layers);
  *bytes = L.off;
  return VLA_OK;
}

int vla_create(const vla_config* cfg, const vla_weights* w, void* workspace, size_t ws_bytes, void* stream,
               vla_model** out) {
  Dims D;
  int rc = check_config(cfg, &D);
  if (rc) return rc;
  if (!w || !out || !workspace) return fail(VLA_EINVAL, "NULL weights, workspace or out");
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->wq || !w->wk || !w->wv || !w->wo ||
      !w->mlp_norm || !w->wgate || !w->wup || !w->wdown)
    return fail(VLA_EINVAL, "a weight pointer is NULL");
  for (int l = 0; l < cfg->n_layers; ++l)
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->mlp_norm[l] || !w->wgate[l] ||
        !w->wup[l] || !w->wdown[l])
      return fail(VLA_EINVAL, "a per-layer weight pointer is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return fail(VLA_EWORKSPACE, "workspace not 256-byte aligned");
  Layout L;
  L.base = static_cast<char*>(workspace);
  vla_model* m = new vla_model();
  m->cfg = *cfg;
  m->D = D;
  plan(L, m, D, cfg->n_layers);
  if (L.off > ws_bytes) {
    delete m;
    return fail(VLA_EWORKSPACE, "workspace smaller than vla_workspace_size()");
  }
  m->scale = 1.0f / std::sqrt((float)D.hd);
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      cus = 256;
    m->cus = cus;
    m->plan_qkv = skinny_plan(3 * D.d, D.d, cus, kMaxSplits);
    m->plan_o = skinny_plan(D.d, D.d, cus, kMaxSplits);
    m->plan_gu = skinny_plan(2 * D.Fp, D.d, cus, kMaxSplits);
    m->plan_d = skinny_plan(D.d, D.Fp, cus, kMaxSplits);
    m->plan_head = skinny_plan(D.Ap, D.d, cus, kMaxSplits);
    m->fused_ok = decode_layer_supported();
    m->decode_path = 0;  // the per-kernel path: measured faster than the persistent layer kernel
  }
  set_meta_views(m, m->meta_dev);
  m->state_batch = 0;
  m->state_valid = false;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int n_events = 0;
  auto cleanup = [&](int code) {
    for (int i = 0; i < n_events; ++i) (void)hipEventDestroy(m->meta_event[i]);
    if (m->meta_host) (void)hipHostFree(m->meta_host);
    delete m;
    return code;
  };
  m->meta_host = nullptr;
  if (hipHostMalloc(reinterpret_cast<void**>(&m->meta_host), kMetaRing * D.meta_ints * sizeof(int32_t),
                    hipHostMallocDefault) != hipSuccess)
    return cleanup(fail(VLA_EHIP, "hipHostMalloc of the metadata staging buffers failed"));
  std::memset(m->meta_host, 0, kMetaRing * D.meta_ints * sizeof(int32_t));
  for (; n_events < kMetaRing; ++n_events)
    if (hipEventCreateWithFlags(&m->meta_event[n_events], hipEventDisableTiming) != hipSuccess)
      return cleanup(fail(VLA_EHIP, "hipEventCreate failed"));

  auto ck = [&](hipError_t e, const char* what) -> int {
    if (e == hipSuccess) return VLA_OK;
    return fail(VLA_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  };
#define CREATE_CK(expr)                      \
  do {                                       \
    int r_ = ck((expr), #expr);              \
    if (r_) return cleanup(r_);              \
  } while (0)

  const bf16_t* emb = static_cast<const bf16_t*>(w->embed);
  const bf16_t* lm = static_cast<const bf16_t*>(w->lm_head);
  CREATE_CK(hipMemcpyAsync(m->emb, emb, (size_t)D.V * D.d * 2, hipMemcpyDeviceToDevice, s));
  // projection weights are stored in frag layout (see frag_index); the LM head keeps only the action rows.
  // The spare blocks are zeroed first, so that every byte of a packed weight is defined.
  auto pack = [&](bf16_t* dst, int rows, int K, const void* src, int src_ld, int src_rows, int src_cols, int mode,
                  const void* src2 = nullptr) {
    const hipError_t e = launch_fill_zero(dst, frag_elems(rows, K) * sizeof(bf16_t), s);
    if (e != hipSuccess) return e;
    PackArgs pa{dst, rows, K, static_cast<const bf16_t*>(src), static_cast<const bf16_t*>(src2), src_ld, src_rows,
                src_cols, mode, D.hd};
    return launch_pack_frag(pa, s);
  };
  CREATE_CK(pack(m->lm_act, D.Ap, D.d, lm + (size_t)cfg->action_begin * D.d, D.d, D.A, D.d, kPackRows));
  CREATE_CK(launch_bf16_to_f32(m->final_norm, static_cast<const bf16_t*>(w->final_norm), D.d, s));
  for (int l = 0; l < D.L; ++l) {
    LayerW& lw = m->lw[l];
    // [Wq; Wk; Wv] is 3d rows of one frag matrix: d is a multiple of 256, so each part starts on a 16-row block
    const size_t part = frag_elems(D.d, D.d);
    CREATE_CK(pack(lw.wqkv, D.d, D.d, w->wq[l], D.d, D.d, D.d, kPackQk));
    CREATE_CK(pack(lw.wqkv + part, D.d, D.d, w->wk[l], D.d, D.d, D.d, kPackQk));
    CREATE_CK(pack(lw.wqkv + 2 * part, D.d, D.d, w->wv[l], D.d, D.d, D.d, kPackRows));
    CREATE_CK(pack(lw.wo, D.d, D.d, w->wo[l], D.d, D.d, D.d, kPackRows));
    CREATE_CK(pack(lw.wgu, 2 * D.Fp, D.d, w->wgate[l], D.d, D.F, D.d, kPackGateUp, w->wup[l]));
    CREATE_CK(pack(lw.wd, D.d, D.Fp, w->wdown[l], D.F, D.d, D.F, kPackRows));
    CREATE_CK(launch_bf16_to_f32(lw.attn_norm, static_cast<const bf16_t*>(w->attn_norm[l]), D.d, s));
    CREATE_CK(launch_bf16_to_f32(lw.mlp_norm, static_cast<const bf16_t*>(w->mlp_norm[l]), D.d, s));
  }
  // zeroed KV pool: masked keys of a partly filled page then multiply finite values
  CREATE_CK(launch_fill_zero(m->kv[0].k, kv_region_bytes(D, D.L), s));
  CREATE_CK(launch_fill_zero(m->flags, 16, s));
  // rotary table: angle = pos * base^(-2i/hd), evaluated in double precision
  std::vector<float2> rope((size_t)D.Smax * (D.hd / 2));
  for (int p = 0; p < D.Smax; ++p)
    for (int i = 0; i < D.hd / 2; ++i) {
      const double ang = (double)p * std::pow((double)cfg->rope_base, -2.0 * i / D.hd);
      rope[(size_t)p * (D.hd / 2) + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
    }
  CREATE_CK(hipMemcpyAsync(m->rope, rope.data(), rope.size() * sizeof(float2), hipMemcpyHostToDevice, s));
  CREATE_CK(hipStreamSynchronize(s));
#undef CREATE_CK
  *out = m;
  g_err.clear();
  return VLA_OK;
}

int vla_prefill(vla_model* m, int32_t B, const void* vis, const int32_t* ids, const int32_t* lens_host,
                float* logits, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (B < 0) return fail(VLA_EINVAL, "negative batch");
  if (B > m->D.Bmax) return fail(VLA_ESHAPE, "batch > max_batch");
  m->state_valid = false;
  if (B == 0) {
    m->state_batch = 0;
    m->state_valid = true;
    return VLA_OK;
  }
  if (!lens_host || !logits || (m->D.nvis > 0 && !vis)) return fail(VLA_EINVAL, "NULL argument");
  long long np = 0;
  for (int b = 0; b < B; ++b) np += lens_host[b];
  if (np > 0 && !ids) return fail(VLA_EINVAL, "prompt_ids is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int R = 0;
  int rc = forward(m, B, vis, ids, lens_host, nullptr, s, &R);
  if (rc) return rc;
  rc = head_logits(m, m->u_head, R, m->logits_pre, s);
  if (rc) return rc;
  VLA_CK(hipMemcpyAsync(logits, m->logits_pre, (size_t)B * m->D.A * sizeof(float), hipMemcpyDeviceToDevice, s));
  m->prefix_host.assign(B, 0);
  for (int b = 0; b < B; ++b) m->prefix_host[b] = m->D.nvis + lens_host[b];
  m->state_batch = B;
  m->state_valid = true;
  g_err.clear();
  return VLA_OK;
}

int vla_decode_actions(vla_model* m, int32_t B, const float* gumbel, float T, int32_t* tokens, float* logp,
                       float* entropy, float* step_logits, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (!m->state_valid || B != m->state_batch) return fail(VLA_ESTATE, "decode needs a prefill of the same batch");
  if (B == 0) {
    m->state_valid = false;
    return VLA_OK;
  }
  if (!gumbel || !tokens || !logp) return fail(VLA_EINVAL, "NULL argument");
  if (!(T > 0.f) || !std::isfinite(T)) return fail(VLA_EINVAL, "temperature must be finite and > 0");
  const Dims& D = m->D;
  hipStream_t s = static_cast<hipStream_t>(stream);
  m->state_valid = false;
  const float eps = m->cfg.rms_eps;
  const bool fused = m->fused_ok && m->decode_path == 1;
  unsigned bar_base = 0;
  if (fused) VLA_CK(launch_fill_zero(m->dec_bar, 256 * sizeof(unsigned), s));
  for (int i = 0; i < D.nact; ++i) {
    const float* z = m->logits_pre;
    if (i > 0 && fused) {
      int rc = decode_step_fused(m, B, i, bar_base, s);
      if (rc) return rc;
      z = m->logits_dec;
    } else if (i > 0) {
      VLA_CK(launch_embed_token_norm(m->next_tok, m->emb, m->x, m->u, m->lw[0].attn_norm, eps, B, D.d, D.V, m->flags,
                                     s));
      // The decode GEMMs take at most kSkinnyRows rows: larger batches run the
      // layer stack once per chunk of environments (each chunk streams the weights).
      for (int r0 = 0; r0 < B; r0 += kSkinnyRows) {
        const int rows = std::min(kSkinnyRows, B - r0);
        float* x = m->x + (size_t)r0 * D.d;
        bf16_t* u = m->u + frag_index(r0, 0, D.d);  // r0 is a multiple of 16: whole frag blocks
        bf16_t* h = m->h + frag_index(r0, 0, D.Fp);
        const int32_t* ptab = m->page_table + (size_t)r0 * D.max_pages;
        const int32_t* eprefix = m->env_prefix + r0;
        // KV bytes read by one layer's decode attention at this step (K and V rows of every key)
        double kv_bytes = 0.0;
        for (int b = r0; b < r0 + rows; ++b) kv_bytes += 2.0 * 2.0 * D.d * (double)(m->prefix_host[b] + i);
        for (int l = 0; l < D.L; ++l) {
          const LayerW& w = m->lw[l];
          SkinnyArgs sq{u, rows, w.wqkv, 3 * D.d, D.d, m->part};
          PROF_LAUNCH(VLA_PROF_DECODE_GEMM, skinny_bytes(3.0 * D.d, D.d, rows), launch_skinny(sq, m->plan_qkv, s));
          DecodeAttnArgs da{m->part, m->plan_qkv, m->rope, u, m->kv[l], ptab, D.max_pages, eprefix,
                            i, rows, D.d, D.H, D.hd, m->scale};
          PROF_LAUNCH(VLA_PROF_DECODE_ATTN, kv_bytes, launch_attn_decode(da, s));
          SkinnyArgs so{u, rows, w.wo, D.d, D.d, m->part};
          PROF_LAUNCH(VLA_PROF_DECODE_GEMM, skinny_bytes(D.d, D.d, rows), launch_skinny(so, m->plan_o, s));
          VLA_CK(launch_reduce_residual_norm(m->part, m->plan_o, x, u, w.mlp_norm, eps, rows, D.d, s));
          SkinnyArgs sg{u, rows, w.wgu, 2 * D.Fp, D.d, m->part};
          PROF_LAUNCH(VLA_PROF_DECODE_GEMM, skinny_bytes(2.0 * D.F, D.d, rows), launch_skinny(sg, m->plan_gu, s));
          VLA_CK(launch_reduce_swiglu(m->part, m->plan_gu, h, D.Fp, rows, D.Fp, s));
          SkinnyArgs sd{h, rows, w.wd, D.d, D.Fp, m->part};
          PROF_LAUNCH(VLA_PROF_DECODE_GEMM, skinny_bytes(D.d, D.F, rows), launch_skinny(sd, m->plan_d, s));
          const float* gnext = (l + 1 < D.L) ? m->lw[l + 1].attn_norm : m->final_norm;
          VLA_CK(launch_reduce_residual_norm(m->part, m->plan_d, x, u, gnext, eps, rows, D.d, s));
        }
      }
      int rc = head_logits(m, m->u, B, m->logits_dec, s);
      if (rc) return rc;
      z = m->logits_dec;
    }
    SamplerArgs sa{};
    sa.z = z; sa.A = D.A; sa.temperature = T; sa.gumbel = gumbel; sa.step = i; sa.n_actions = D.nact;
    sa.action_begin = m->cfg.action_begin; sa.tokens = tokens; sa.next_tok = m->next_tok; sa.logp = logp;
    sa.entropy = entropy; sa.logits_out = step_logits; sa.rows = B; sa.flags = m->flags;
    VLA_CK(launch_sampler(sa, s));
  }
  g_err.clear();
  return VLA_OK;
}

int vla_token_logprobs(vla_model* m, int32_t B, const void* vis, const int32_t* ids, const int32_t* lens_host,
                       const int32_t* actions, float T, float* logp, float* entropy, float* logits, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (B < 0) return fail(VLA_EINVAL, "negative batch");
  if (B > m->D.Bmax) return fail(VLA_ESHAPE, "batch > max_batch");
  m->state_valid = false;
  if (B == 0) return VLA_OK;
  if (!lens_host || !actions || !logp || (m->D.nvis > 0 && !vis)) return fail(VLA_EINVAL, "NULL argument");
  if (!(T > 0.f) || !std::isfinite(T)) return fail(VLA_EINVAL, "temperature must be finite and > 0");
  long long np = 0;
  for (int b = 0; b < B; ++b) np += lens_host[b];
  if (np > 0 && !ids) return fail(VLA_EINVAL, "prompt_ids is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int R = 0;
  int rc = forward(m, B, vis, ids, lens_host, actions, s, &R);
  if (rc) return rc;
  rc = head_logits(m, m->u_head, R, m->logits_tf, s);
  if (rc) return rc;
  SamplerArgs sa{};
  sa.z = m->logits_tf; sa.A = m->D.A; sa.temperature = T; sa.gumbel = nullptr; sa.given = actions;
  sa.action_begin = m->cfg.action_begin; sa.logp = logp; sa.entropy = entropy; sa.logits_out = logits; sa.rows = R;
  sa.flags = m->flags;
  VLA_CK(launch_sampler(sa, s));
  g_err.clear();
  return VLA_OK;
}

int vla_value(vla_model* m, int32_t B, const void* vis, const int32_t* ids, const int32_t* lens_host,
              const void* value_head, float* values, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (B < 0) return fail(VLA_EINVAL, "negative batch");
  if (B > m->D.Bmax) return fail(VLA_ESHAPE, "batch > max_batch");
  m->state_valid = false;  // the pass overwrites the prefill state
  if (B == 0) return VLA_OK;
  if (!lens_host || !value_head || !values || (m->D.nvis > 0 && !vis)) return fail(VLA_EINVAL, "NULL argument");
  long long np = 0;
  for (int b = 0; b < B; ++b) np += lens_host[b];
  if (np > 0 && !ids) return fail(VLA_EINVAL, "prompt_ids is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int R = 0;
  int rc = forward(m, B, vis, ids, lens_host, nullptr, s, &R);
  if (rc) return rc;
  VLA_CK(launch_value_head(m->u_head, R, m->D.d, static_cast<const bf16_t*>(value_head), values, s));
  g_err.clear();
  return VLA_OK;
}

// The merge of one projection of one layer: its packed destination and row mode.
static int merge_args(vla_model* m, int32_t layer, int32_t projection, const void* w0, const void* lora_a,
                      const void* lora_b, int32_t rank, float scale, MergeArgs* out) {
  if (!w0 || !lora_a || !lora_b) return fail(VLA_EINVAL, "NULL argument");
  const Dims& D = m->D;
  if (layer < 0 || layer >= D.L) return fail(VLA_EINVAL, "layer out of range");
  if (projection < VLA_PROJ_Q || projection > VLA_PROJ_DOWN) return fail(VLA_EINVAL, "unknown projection");
  if (!std::isfinite(scale)) return fail(VLA_EINVAL, "scale must be finite");
  if (rank < 8 || rank > 64 || rank % 8 != 0) return fail(VLA_EUNSUPPORTED, "rank must be a multiple of 8 in [8, 64]");
  const LayerW& w = m->lw[layer];
  MergeArgs a{};
  a.w0 = static_cast<const bf16_t*>(w0);
  a.a = static_cast<const bf16_t*>(lora_a);
  a.b = static_cast<const bf16_t*>(lora_b);
  a.rank = rank;
  a.scale = scale;
  a.head_dim = D.hd;
  a.part = 0;
  const size_t qkv_part = frag_elems(D.d, D.d);  // [Wq; Wk; Wv] are consecutive d-row parts
  switch (projection) {
    case VLA_PROJ_Q: case VLA_PROJ_K: case VLA_PROJ_V:
      a.dst = w.wqkv + (size_t)projection * qkv_part;
      a.rows = D.d; a.K = D.d; a.src_ld = D.d; a.src_rows = D.d; a.src_cols = D.d;
      a.mode = projection == VLA_PROJ_V ? kPackRows : kPackQk;
      break;
    case VLA_PROJ_O:
      a.dst = w.wo; a.rows = D.d; a.K = D.d; a.src_ld = D.d; a.src_rows = D.d; a.src_cols = D.d; a.mode = kPackRows;
      break;
    case VLA_PROJ_GATE: case VLA_PROJ_UP:
      a.dst = w.wgu; a.rows = 2 * D.Fp; a.K = D.d; a.src_ld = D.d; a.src_rows = D.F; a.src_cols = D.d;
      a.mode = kPackGateUp; a.part = projection == VLA_PROJ_UP ? 1 : 0;
      break;
    default:  // VLA_PROJ_DOWN: K padded from d_ffn to Fp with zero columns
      a.dst = w.wd; a.rows = D.d; a.K = D.Fp; a.src_ld = D.F; a.src_rows = D.d; a.src_cols = D.F; a.mode = kPackRows;
      break;
  }
  if (a.src_cols % 8 != 0) return fail(VLA_EUNSUPPORTED, "input features must be a multiple of 8");
  *out = a;
  return VLA_OK;
}

int vla_lora_merge(vla_model* m, int32_t layer, int32_t projection, const void* w0, const void* lora_a,
                   const void* lora_b, int32_t rank, float scale, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  MergeArgs a;
  const int rc = merge_args(m, layer, projection, w0, lora_a, lora_b, rank, scale, &a);
  if (rc) return rc;
  VLA_CK(launch_lora_merge(a, static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_lora_merge_layer(vla_model* m, int32_t layer, const void* const* w0, const void* const* lora_a,
                         const void* const* lora_b, int32_t rank, float scale, void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (!w0 || !lora_a || !lora_b) return fail(VLA_EINVAL, "NULL array");
  MergeBatch b{};
  for (int32_t p = VLA_PROJ_Q; p <= VLA_PROJ_DOWN; ++p) {
    if (!w0[p]) continue;  // this projection is not merged
    const int rc = merge_args(m, layer, p, w0[p], lora_a[p], lora_b[p], rank, scale, &b.item[b.n]);
    if (rc) return rc;
    ++b.n;
  }
  if (b.n > 0) VLA_CK(launch_lora_merge_batch(b, static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_train_workspace_size(const vla_config* cfg, int32_t mode, size_t* bytes) {
  Dims D;
  int rc = check_config(cfg, &D);
  if (rc) return rc;
  if (!bytes) return fail(VLA_EINVAL, "bytes_host is NULL");
  if (mode != VLA_TRAIN_RECOMPUTE && mode != VLA_TRAIN_KEEP) return fail(VLA_EINVAL, "unknown training mode");
  Layout L;
  TrainBufs t;
  plan_train(L, D, t, mode == VLA_TRAIN_KEEP);
  *bytes = L.off;
  return VLA_OK;
}

int vla_ppo_lora_grads(vla_model* m, int32_t B, const void* vis, const int32_t* ids, const int32_t* lens_host,
                       const int32_t* actions, const float* logp_old, const float* advantages, float eps, float T,
                       const vla_lora* lora, void* train_ws, size_t train_bytes, float* stats, float* logp_new,
                       void* stream) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  const Dims& D = m->D;
  if (B < 1) return fail(VLA_EINVAL, "batch must be >= 1");
  if (B > D.Bmax) return fail(VLA_ESHAPE, "batch > max_batch");
  if (!lens_host || !actions || !logp_old || !advantages || !lora || !stats || !train_ws || (D.nvis > 0 && !vis))
    return fail(VLA_EINVAL, "NULL argument");
  if (!lora->a || !lora->b || !lora->grad_a || !lora->grad_b) return fail(VLA_EINVAL, "NULL adapter array");
  if (lora->rank < 1 || lora->rank > 64) return fail(VLA_EUNSUPPORTED, "rank must be in [1, 64]");
  if (!std::isfinite(lora->scale)) return fail(VLA_EINVAL, "scale must be finite");
  for (int i = 0; i < D.L * 7; ++i)
    if (lora->a[i] && (!lora->b[i] || !lora->grad_a[i] || !lora->grad_b[i]))
      return fail(VLA_EINVAL, "an adapted projection needs B and both gradient buffers");
  if (!(T > 0.f) || !std::isfinite(T)) return fail(VLA_EINVAL, "temperature must be finite and > 0");
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(VLA_EINVAL, "eps must be finite and >= 0");
  if (m->layer_limit != 0) return fail(VLA_ESTATE, "a debug layer limit is set");
  if (reinterpret_cast<uintptr_t>(train_ws) % 256 != 0) return fail(VLA_EWORKSPACE, "training workspace misaligned");
  // keep every layer's activations when the workspace holds them, else recompute
  Layout L;
  L.base = static_cast<char*>(train_ws);
  TrainBufs t;
  plan_train(L, D, t, true);
  if (train_bytes < L.off) {
    L = Layout{};
    L.base = static_cast<char*>(train_ws);
    t = TrainBufs{};
    plan_train(L, D, t, false);
    if (train_bytes < L.off)
      return fail(VLA_EWORKSPACE, "training workspace smaller than vla_train_workspace_size(VLA_TRAIN_RECOMPUTE)");
  }
  long long np = 0;
  for (int b = 0; b < B; ++b) np += lens_host[b];
  if (np > 0 && !ids) return fail(VLA_EINVAL, "prompt_ids is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  m->state_valid = false;
  // teacher-forced forward, every layer's input saved
  int R = 0, M = 0;
  int rc = forward(m, B, vis, ids, lens_host, actions, s, &R, &t.sv, &M);
  if (rc) return rc;
  rc = head_logits(m, m->u_head, R, m->logits_tf, s);
  if (rc) return rc;
  SamplerArgs sa{};
  sa.z = m->logits_tf; sa.A = D.A; sa.temperature = T; sa.gumbel = nullptr; sa.given = actions;
  sa.action_begin = m->cfg.action_begin; sa.logp = t.logp; sa.rows = R; sa.flags = m->flags;
  VLA_CK(launch_sampler(sa, s));
  if (logp_new) VLA_CK(hipMemcpyAsync(logp_new, t.logp, (size_t)R * sizeof(float), hipMemcpyDeviceToDevice, s));
  // loss and its gradient down to the action logits
  PpoArgs pp{t.logp, logp_old, advantages, B, D.nact, eps, stats, t.dlogp};
  VLA_CK(launch_ppo_clip(pp, s));
  LogprobBwdArgs lb{m->logits_tf, actions, t.dlogp, R, D.A, m->cfg.action_begin, T, t.dz};
  VLA_CK(launch_logprob_backward(lb, s));
  // head (the action rows of the LM head) and final RMSNorm of the scoring rows
  const int A32 = round_up(D.A, 32);
  VLA_CK(launch_to_frag(t.dz, D.A, R, D.A, A32, t.dzf, s));
  VLA_CK(launch_transpose_frag(m->lm_act, false, D.d, D.A, D.d, A32, t.wact_t, s));
  VLA_CK(gemm_f32(t.dzf, 0, t.wact_t, 0, R, D.d, A32, t.du_h, D.d, s));
  VLA_CK(launch_move_rows(m->x, m->head_rows, R, D.d, t.xc, false, s));
  VLA_CK(launch_rmsnorm_bwd(t.xc, m->final_norm, m->cfg.rms_eps, t.du_h, nullptr, t.dxc, nullptr, R, D.d, s));
  VLA_CK(launch_fill_zero(t.dx, (size_t)M * D.d * sizeof(float), s));
  VLA_CK(launch_move_rows(t.dxc, m->head_rows, R, D.d, t.dx, true, s));
  for (int l = D.L - 1; l >= 0; --l) {
    rc = layer_backward(m, t, l, B, M, lora, s);
    if (rc) return rc;
  }
  g_err.clear();
  return VLA_OK;
}

int vla_extract_actions(int32_t n, int32_t n_dims, const int32_t* tokens, int32_t action_begin, int32_t bins,
                        const float* range_lo, const float* range_hi, float* actions, void* stream) {
  if (n < 0 || n_dims < 1) return fail(VLA_EINVAL, "need n >= 0 and n_dims >= 1");
  if (bins < 1 || bins > 256) return fail(VLA_EUNSUPPORTED, "bins must be in [1, 256]");
  if ((size_t)n * n_dims >= (size_t)1 << 31) return fail(VLA_EUNSUPPORTED, "too many actions");
  if (n == 0) {
    g_err.clear();
    return VLA_OK;
  }
  if (!tokens || !range_lo || !range_hi || !actions) return fail(VLA_EINVAL, "NULL argument");
  VLA_CK(launch_extract_actions(tokens, n, n_dims, action_begin, bins, range_lo, range_hi, actions,
                                static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_gae(int32_t n_env, int32_t n_steps, const float* rewards, const float* values, const uint8_t* dones,
            float gamma, float lam, float* advantages, float* returns, void* stream) {
  if (n_env < 0 || n_steps < 0) return fail(VLA_EINVAL, "negative size");
  if (!(gamma >= 0.f && gamma <= 1.f) || !(lam >= 0.f && lam <= 1.f))
    return fail(VLA_EINVAL, "gamma and lambda must lie in [0, 1]");
  if ((size_t)(n_steps + 1) * (size_t)n_env >= (size_t)1 << 31) return fail(VLA_EUNSUPPORTED, "window too large");
  if (n_env == 0 || n_steps == 0) {
    g_err.clear();
    return VLA_OK;
  }
  if (!rewards || !values || !dones || !advantages) return fail(VLA_EINVAL, "NULL argument");
  GaeArgs a{rewards, values, dones, n_env, n_steps, gamma, lam, advantages, returns};
  VLA_CK(launch_gae(a, static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_ppo_clip(int32_t n, int32_t n_tokens, const float* logp_new, const float* logp_old,
                 const float* advantages, float eps, float* stats, float* dlogp, void* stream) {
  if (n < 1 || n_tokens < 1 || n_tokens > 16) return fail(VLA_EINVAL, "need n >= 1 and 1 <= n_tokens <= 16");
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(VLA_EINVAL, "eps must be finite and >= 0");
  if (!logp_new || !logp_old || !advantages || !stats || !dlogp) return fail(VLA_EINVAL, "NULL argument");
  if ((size_t)n * n_tokens >= (size_t)1 << 31) return fail(VLA_EUNSUPPORTED, "too many tokens");
  PpoArgs a{logp_new, logp_old, advantages, n, n_tokens, eps, stats, dlogp};
  VLA_CK(launch_ppo_clip(a, static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_logprob_backward(int32_t rows, int32_t bins, int32_t action_begin, const float* logits,
                         const int32_t* tokens, float temperature, const float* dlogp, float* dlogits,
                         void* stream) {
  if (rows < 0) return fail(VLA_EINVAL, "negative size");
  if (bins < 1 || bins > 256) return fail(VLA_EUNSUPPORTED, "bins must be in [1, 256]");
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(VLA_EINVAL, "temperature must be > 0");
  if (rows == 0) {
    g_err.clear();
    return VLA_OK;
  }
  if (!logits || !tokens || !dlogp || !dlogits) return fail(VLA_EINVAL, "NULL argument");
  LogprobBwdArgs a{logits, tokens, dlogp, rows, bins, action_begin, temperature, dlogits};
  VLA_CK(launch_logprob_backward(a, static_cast<hipStream_t>(stream)));
  g_err.clear();
  return VLA_OK;
}

int vla_read_device_flags(vla_model* m, void* stream, uint32_t* flags_host) {
  if (!m || !flags_host) return fail(VLA_EINVAL, "NULL argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint32_t v = 0;
  VLA_CK(hipMemcpyAsync(&v, m->flags, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  VLA_CK(hipStreamSynchronize(s));
  VLA_CK(launch_fill_zero(m->flags, 16, s));
  VLA_CK(hipStreamSynchronize(s));
  *flags_host = v;
  return VLA_OK;
}

int vla_profile_begin(vla_model* m, uint32_t mask) {
  if (!m) return fail(VLA_EINVAL, "model is NULL");
  if (m->prof.empty()) {
    m->prof.resize(kProfSlots);
    for (auto& p : m->prof) {
      VLA_CK(hipEventCreate(&p.a));
      VLA_CK(hipEventCreate(&p.b));
    }
  }
  m->prof_used = 0;
  m->prof_mask = mask;
  return VLA_OK;
}

int vla_profile_end(vla_model* m, double* ms, double* work, int64_t* launches) {
  if (!m || !ms || !work || !launches) return fail(VLA_EINVAL, "NULL argument");
  for (int c = 0; c < VLA_PROF_CATEGORIES; ++c) {
    ms[c] = 0.0;
    work[c] = 0.0;
    launches[c] = 0;
  }
  if (m->prof_used > 0) VLA_CK(hipEventSynchronize(m->prof[m->prof_used - 1].b));
  for (int i = 0; i < m->prof_used; ++i) {
    float t = 0.f;
    VLA_CK(hipEventElapsedTime(&t, m->prof[i].a, m->prof[i].b));
    const int c = m->prof[i].cat;
    ms[c] += t;
    work[c] += m->prof[i].work;
    launches[c] += 1;
  }
  m->prof_used = 0;
  m->prof_mask = 0;
  return VLA_OK;
}

void vla_destroy(vla_model* m) {
  if (!m) return;
  for (auto& p : m->prof) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  for (int i = 0; i < kMetaRing; ++i) {
    if (m->meta_pending[i]) (void)hipEventSynchronize(m->meta_event[i]);
    (void)hipEventDestroy(m->meta_event[i]);
  }
  if (m->meta_host) (void)hipHostFree(m->meta_host);
  delete m;
}

const char* vla_last_error(void) { return g_err.c_str(); }

int vla_debug_set_layer_limit(vla_model* m, int32_t n_layers) {
  if (!m || n_layers < 0) return fail(VLA_EINVAL, "bad argument");
  m->layer_limit = n_layers;
  return VLA_OK;
}

int vla_debug_set_decode_path(vla_model* m, int32_t persistent) {
  if (!m || persistent < 0 || persistent > 1) return fail(VLA_EINVAL, "bad argument");
  m->decode_path = persistent;
  return VLA_OK;
}

int vla_debug_trace_decode_layer(vla_model* m, int32_t layer, void* stamps) {
  if (!m || layer < 0 || layer >= m->D.L) return fail(VLA_EINVAL, "bad argument");
  m->trace_layer = layer;
  m->trace_buf = static_cast<unsigned long long*>(stamps);
  return VLA_OK;
}

int vla_debug_set_stop(vla_model* m, int32_t stage) {
  if (!m || stage < 0 || stage > 3) return fail(VLA_EINVAL, "bad argument");
  m->debug_stop = stage;
  return VLA_OK;
}

int vla_debug_read(vla_model* m, int32_t which, int32_t layer, void* dst, size_t bytes, void* stream) {
  if (!m || !dst || layer < 0 || layer >= m->D.L) return fail(VLA_EINVAL, "bad argument");
  const Dims& D = m->D;
  const void* src = nullptr;
  size_t avail = 0;
  const size_t kv = (size_t)D.n_pages * D.H * kPage * D.hd * sizeof(bf16_t);
  switch (which) {
    case 0: src = m->x; avail = D.Mmax * D.d * sizeof(float); break;
    case 1: src = m->q; avail = D.Mmax * D.d * sizeof(bf16_t); break;
    case 2: src = m->kv[layer].k; avail = kv; break;
    case 3: src = m->kv[layer].v; avail = kv; break;
    case 4: src = m->u; avail = frag_elems(D.Mmax, D.d) * sizeof(bf16_t); break;
    case 5: src = m->lw[layer].wqkv; avail = frag_elems(3 * D.d, D.d) * sizeof(bf16_t); break;
    case 6: src = m->lw[layer].wo; avail = frag_elems(D.d, D.d) * sizeof(bf16_t); break;
    case 7: src = m->lw[layer].wgu; avail = frag_elems(2 * D.Fp, D.d) * sizeof(bf16_t); break;
    case 8: src = m->lw[layer].wd; avail = frag_elems(D.d, D.Fp) * sizeof(bf16_t); break;
    case 9: src = m->h; avail = frag_elems(D.Mmax, D.Fp) * sizeof(bf16_t); break;
    default: return fail(VLA_EINVAL, "unknown buffer");
  }
  if (bytes > avail) return fail(VLA_EINVAL, "read larger than the buffer");
  VLA_CK(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream)));
  return VLA_OK;
}

}  // extern "C"
