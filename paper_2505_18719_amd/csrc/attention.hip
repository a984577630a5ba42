// Causal attention over the paged KV cache on gfx950.
//
// Prefill: one 512-thread workgroup per (environment, head); the head's whole
// K and V^T are copied into LDS once, then 16-query tiles are dealt to the 8
// waves.  Scores are computed transposed so that P stays in registers in the
// layout the P*V MFMA consumes, and a whole score row (<= 320 keys, the
// longest sequence of one environment) stays in registers, so the softmax is
// exact.
//
// Decode: one workgroup per (environment, head) and one query; scores and
// P*V in fp32 on the vector ALUs, streaming K rows and transposed V pages with
// 16-byte loads.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

// Prefill attention: one 512-thread workgroup (8 waves) per (environment,
// head).  The environment's whole K (key rows) and V^T (feature rows) for
// this head, <= 320 keys, are copied once into LDS with buffer_load ... lds
// (80 KB each at head_dim 128), then every wave takes 16-query tiles of the
// causal triangle in a balanced order.  Per tile, scores are computed
// transposed, S^T = K Q^T, with the keys of each 32-key chunk assigned to MFMA
// rows so that lane group g ends up holding keys 8g .. 8g+7 of the chunk for
// its query: exactly the B-operand fragment of P^T in O^T = V^T P^T.  P never
// leaves registers and enters the MFMA as P_hi + P_lo (two bf16 products,
// ~16 significant bits).  The whole score row (<= 320 keys) is kept, so the
// softmax is exact (true maximum, no online rescaling).
//
// LDS layouts (both conflict-free for the 16-byte operand reads, no padding):
//  K: row R holds key kperm(R), with the 32 keys of a chunk ordered as the
//     MFMA rows of its two 16-key tiles; 16-byte feature chunk j of row R is
//     stored at slot j ^ kswz(R).
//  V^T: the cache's own page layout, one 16-key page after the other (feature
//     f of a page: 16 keys, two 16-byte halves); half h of feature f is stored
//     at 16-byte unit 2f + (h ^ ((f >> 3) & 1)) of its page.
constexpr int kMaxKeys = 320;
constexpr int kMaxChunks = kMaxKeys / 32;
constexpr int kMaxPages = kMaxKeys / kPage;

// key held by LDS row R of K: MFMA row i of 16-key tile t of chunk c is key 32c + 8(i/4) + 4t + i%4
__device__ __forceinline__ int kperm(int R) {
  const int i = R & 15, t = (R >> 4) & 1, c = R >> 5;
  return 32 * c + 8 * (i >> 2) + 4 * t + (i & 3);
}
template <int HD>
__device__ __forceinline__ int kswz(int R) {
  return HD == 128 ? (R & 15) : ((R >> 1) & 7);
}

// One 16-query tile (queries 16 qt .. 16 qt + 15 of the environment) whose
// keys span NC 32-key chunks; only the last chunk holds keys that some query
// of the tile must not see (ncq = qt / 2 + 1 for every tile of a sequence).
// Straight-line code for a compile-time chunk count, so the scheduler can
// overlap the LDS reads of one chunk with the MFMAs of another.
template <int HD, int NC>
__device__ __forceinline__ void attn_tile(const PrefillAttnArgs& a, const char* klds, const char* vlds, int qt, int L,
                                          int row0, int head, int lane) {
  constexpr int KROW = HD * 2, VPAGE = HD * kPage * 2;
  constexpr int KS = HD / 32, NB = HD / 16;
  const int r16 = lane & 15, g = lane >> 4;
  const int qpos = qt * 16 + r16;
  uint4 qf[KS];  // B operand: query qpos, features 32 ks + 8g .. +8
  {
    const bf16_t* qp = a.q + (size_t)(row0 + min(qpos, L - 1)) * a.d + head * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const uint4*>(qp + ks * 32);
  }
  // scores: lane holds S(query qpos, key 32c + 8g + 4t + r) in sc[2c + t][r]
  f32x4 sc[2 * NC];
#pragma unroll
  for (int t = 0; t < 2 * NC; ++t) sc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int ct = 0; ct < 2 * NC; ++ct) {
      // LDS row 16 ct + r16 (chunk ct / 2, tile ct % 2); its swizzle is kswz<HD>(r16)
      const char* kr = klds + (16 * ct + r16) * KROW + 16 * ((4 * ks + g) ^ kswz<HD>(r16));
      sc[ct] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(kr)), as_bf16x8(qf[ks]), sc[ct]);
    }
  }
  const int klim = min(qpos, L - 1);  // last key this lane's query sees
  float mx = -INFINITY;
#pragma unroll
  for (int ct = 0; ct < 2 * NC; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = sc[ct][r] * a.scale;
      if (ct >= 2 * NC - 2) {
        const int key = 32 * (ct >> 1) + 8 * g + 4 * (ct & 1) + r;
        v = key <= klim ? v : -INFINITY;
      }
      sc[ct][r] = v;
      mx = fmaxf(mx, v);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
  mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
  float sum = 0.f;
#pragma unroll
  for (int ct = 0; ct < 2 * NC; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float pv = expf(sc[ct][r] - mx);  // masked: expf(-inf) = 0
      sc[ct][r] = pv;
      sum += pv;
    }
  sum += __shfl_xor(sum, 16, kWave);
  sum += __shfl_xor(sum, 32, kWave);
  if (a.lse && g == 0 && qpos < L) a.lse[((size_t)(row0 + qpos) * a.n_heads + head) * 2] = mx + logf(sum);

  // O^T = V^T P^T: A operand = V^T rows (feature nb*16 + r16), keys 32c + 8g .. +8,
  // i.e. page 2c + g/2, half g%2; (f >> 3) & 1 of feature 16nb + r16 is r16 >> 3
  f32x4 o[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const char* vp0 = vlds + (g >> 1) * VPAGE + 16 * (2 * r16 + ((g & 1) ^ (r16 >> 3)));
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 phi, plo;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pv = sc[2 * c + t][r];
        const __bf16 h = (__bf16)pv;
        phi[4 * t + r] = h;
        plo[4 * t + r] = (__bf16)(pv - (float)h);
      }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const uint4 vv = *reinterpret_cast<const uint4*>(vp0 + 2 * c * VPAGE + nb * 16 * 32);
      o[nb] = mfma16(as_bf16x8(vv), phi, o[nb]);
      o[nb] = mfma16(as_bf16x8(vv), plo, o[nb]);
    }
  }
  // o[nb][r] = O(query qpos, feature nb*16 + 4g + r)
  if (qpos < L) {
    const float inv = 1.f / sum;
    // frag layout (the O projection's A operand): 4 consecutive features stay contiguous
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      *reinterpret_cast<uint2*>(a.o + frag_index(row0 + qpos, head * HD + nb * 16 + 4 * g, a.d)) =
          make_uint2(pack2bf(o[nb][0] * inv, o[nb][1] * inv), pack2bf(o[nb][2] * inv, o[nb][3] * inv));
  }
}

// Tiles qt_lo .. qt_hi - 1, most expensive first, dealt to the 8 waves in snake order.
template <int HD>
__device__ __forceinline__ void attn_tiles(const PrefillAttnArgs& a, const char* klds, const char* vlds, int qt_lo,
                                           int qt_hi, int L, int row0, int head, int wave, int lane) {
  const int n = qt_hi - qt_lo;
  for (int p0 = 0; p0 < n; p0 += 8) {
    const int p = p0 + (((p0 >> 3) & 1) ? 7 - wave : wave);
    if (p >= n) continue;
    const int qt = qt_hi - 1 - p;
    switch (qt / 2 + 1) {  // live 32-key chunks
      case 1: attn_tile<HD, 1>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 2: attn_tile<HD, 2>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 3: attn_tile<HD, 3>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 4: attn_tile<HD, 4>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 5: attn_tile<HD, 5>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 6: attn_tile<HD, 6>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 7: attn_tile<HD, 7>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 8: attn_tile<HD, 8>(a, klds, vlds, qt, L, row0, head, lane); break;
      case 9: attn_tile<HD, 9>(a, klds, vlds, qt, L, row0, head, lane); break;
      default: attn_tile<HD, 10>(a, klds, vlds, qt, L, row0, head, lane); break;
    }
  }
}

template <int HD>
__global__ __launch_bounds__(512, 1) void attn_prefill_kernel(PrefillAttnArgs a) {
  constexpr int KROW = HD * 2;           // bytes per K row
  constexpr int KCH = HD / 8;            // 16-byte chunks per K row
  constexpr int VPAGE = HD * kPage * 2;  // bytes per V^T page
  __shared__ __attribute__((aligned(1024))) char lds[kMaxKeys * KROW + kMaxPages * VPAGE];
  char* const klds = lds;
  char* const vlds = lds + kMaxKeys * KROW;
  const int env = blockIdx.x, head = blockIdx.y;
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int H = a.n_heads;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nch = (L + 31) / 32;
  const int32_t* pt = a.page_table + env * a.max_pages;
  const int last_page = a.max_pages - 1;

  // ---- copy the K rows and V^T pages of the nch chunks into LDS, chunk by
  // chunk: copy i moves 1 KB of chunk i / CP (K rows first, then V^T pages);
  // wave w issues copies w, w + 8, ..., i.e. CP / 8 per chunk
  constexpr int KC = 32 * KROW / 1024, VC = 2 * VPAGE / 1024, CP = KC + VC;
  constexpr int KROWS_PER_KB = 1024 / KROW;
  static_assert(CP % 8 == 0, "copies per chunk must divide among the 8 waves");
  {
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)a.kv.k, (short)0, 0x7fffffff, 0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)a.kv.v, (short)0, 0x7fffffff, 0x00020000);
    const uint32_t kbase = (uint32_t)(uintptr_t)((lds_ptr_t*)klds), vbase = (uint32_t)(uintptr_t)((lds_ptr_t*)vlds);
    // the environment's page table, one entry per lane, read once: a copy must
    // not wait on a load of its own (the wait would also drain every copy
    // issued before it)
    int ptv = pt[min(lane, last_page)];
    // the copies below use ptv; passing it through an empty asm ends the load's
    // lifetime here, so the compiler waits for it once and not before each copy
    asm volatile("" : "+v"(ptv));
    for (int i = wave; i < CP * nch; i += 8) {
      const int c = i / CP, sub = i % CP;
      if (sub < KC) {
        const int kcopy = c * KC + sub;  // 1 KB of K rows, all in one 16-key page
        const int R = kcopy * KROWS_PER_KB + lane / KCH, slot = lane % KCH;
        const int key = kperm(R);
        const int page = __builtin_amdgcn_readlane(ptv, min(kperm(kcopy * KROWS_PER_KB) / kPage, last_page));
        const uint32_t off = (uint32_t)((((page * H + head) * kPage + key % kPage) * HD + 8 * (slot ^ kswz<HD>(R))) * 2);
        lds_dma16(kbase + kcopy * 1024, off, rk, 0);
      } else {
        const int vcopy = c * VC + (sub - KC);  // 1 KB of V^T pages
        const int pg = vcopy / (VPAGE / 1024);
        const int unit = (vcopy % (VPAGE / 1024)) * 64 + lane;  // 16-byte unit of the page
        const int f = unit >> 1, h = (unit & 1) ^ ((f >> 3) & 1);
        const int page = __builtin_amdgcn_readlane(ptv, min(pg, last_page));
        const uint32_t off = (uint32_t)((((page * H + head) * HD + f) * kPage + 8 * h) * 2);
        lds_dma16(vbase + vcopy * 1024, off, rv, 0);
      }
    }
  }
  // phase 1: the tiles whose keys lie in the first h1 chunks start as soon as
  // those chunks have landed, while the rest are still being copied
  const int h1 = min(nch, kMaxChunks / 2);
  const int nq = (L + 15) / 16;
  const int q1 = min(nq, 2 * h1);  // tiles 0 .. q1-1 need chunks < h1
  switch ((nch - h1) * (CP / 8)) {  // this wave's copies of the later chunks may stay in flight
    case 0: WAIT_VMCNT(0); break;
    case 1: WAIT_VMCNT(1); break;
    case 2: WAIT_VMCNT(2); break;
    case 3: WAIT_VMCNT(3); break;
    case 4: WAIT_VMCNT(4); break;
    case 5: WAIT_VMCNT(5); break;
    case 6: WAIT_VMCNT(6); break;
    case 7: WAIT_VMCNT(7); break;
    case 8: WAIT_VMCNT(8); break;
    case 9: WAIT_VMCNT(9); break;
    default: WAIT_VMCNT(10); break;
  }
  __syncthreads();
  // query tiles below the first needed row are skipped (their keys are still loaded: later rows see them)
  const int qlo = a.env_q0 ? min(max(a.env_q0[env], 0), L - 1) / 16 : 0;
  if (qlo < q1) attn_tiles<HD>(a, klds, vlds, qlo, q1, L, row0, head, wave, lane);
  if (q1 < nq) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    attn_tiles<HD>(a, klds, vlds, max(qlo, q1), nq, L, row0, head, wave, lane);
  }
}

template <int HD>
__global__ __launch_bounds__(256) void attn_decode_kernel(DecodeAttnArgs a) {
  constexpr int LPK = HD / 8;          // lanes per key row
  constexpr int KPP = 256 / LPK;       // keys per pass
  constexpr int G = 256 / HD;          // feature groups in P*V
  constexpr int HALF = HD / 2;
  __shared__ float sc[kMaxKeys];
  __shared__ float qs[HD], kn[HD], vn[HD];  // this token's rotated q, k and its v (bf16 values)
  __shared__ float red[4];
  __shared__ float op[G][HD];
  __shared__ int ptl[kMaxPages];  // the environment's page table
  const int head = blockIdx.x, b = blockIdx.y;
  const int H = a.n_heads, tid = threadIdx.x;
  const int n = a.env_prefix[b] + a.step;  // keys 0 .. n-1; key n-1 is this step's token
  const int pos = n - 1;
  const int32_t* pt = a.page_table + b * a.max_pages;
  if (tid < a.max_pages) ptl[tid] = pt[tid];

  // ---- q, k, v of the token for this head: one thread per rotary pair of
  // q and k (columns permuted per head as for the prefill GEMM's epilogue:
  // pair (32 blk + c, HALF + 32 blk + c) sits in columns 64 blk + c and
  // 64 blk + c + 32 of the head) and per pair of v features (e, e + HALF)
  if (tid < 3 * HALF) {
    const int region = tid / HALF, e = tid % HALF;
    const int N = 3 * a.d;
    int col1, col2;
    if (region < 2) {
      col1 = region * a.d + head * HD + 64 * (e / 32) + e % 32;
      col2 = col1 + 32;
    } else {
      col1 = 2 * a.d + head * HD + e;
      col2 = col1 + HALF;
    }
    const float x1 = skinny_sum(a.part, a.plan, a.B, N, b, col1);
    const float x2 = skinny_sum(a.part, a.plan, a.B, N, b, col2);
    const int page = pt[pos / kPage], slot = pos % kPage;
    if (region == 2) {
      const bf16_t v1 = f2bf(x1), v2 = f2bf(x2);
      bf16_t* vb = a.kv.v + ((size_t)page * H + head) * HD * kPage + slot;
      vb[(size_t)e * kPage] = v1;
      vb[(size_t)(e + HALF) * kPage] = v2;
      vn[e] = bf2f(v1);
      vn[e + HALF] = bf2f(v2);
    } else {
      const float2 cs = a.rope[pos * HALF + e];
      const bf16_t r1 = f2bf(x1 * cs.x - x2 * cs.y), r2 = f2bf(x1 * cs.y + x2 * cs.x);
      if (region == 0) {
        qs[e] = bf2f(r1);
        qs[e + HALF] = bf2f(r2);
      } else {
        bf16_t* kr = a.kv.k + (((size_t)page * H + head) * kPage + slot) * HD;
        kr[e] = r1;
        kr[e + HALF] = r2;
        kn[e] = bf2f(r1);
        kn[e + HALF] = bf2f(r2);
      }
    }
  }
  __syncthreads();

  const int part = tid % LPK;
  float qv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) qv[j] = qs[part * 8 + j];
  // scores: one key row per LPK lanes
  for (int base = 0; base < n; base += KPP) {
    const int key = base + tid / LPK;
    float acc = 0.f;
    if (key < n) {
      float kf[8];
      if (key < pos) {
        const bf16_t* kp = a.kv.k + (((size_t)ptl[key / kPage] * H + head) * kPage + key % kPage) * HD + part * 8;
        unpack8(*reinterpret_cast<const uint4*>(kp), kf);
      } else {  // this step's token
#pragma unroll
        for (int j = 0; j < 8; ++j) kf[j] = kn[part * 8 + j];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) acc += qv[j] * kf[j];
    }
#pragma unroll
    for (int o = LPK / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kWave);
    if (part == 0 && key < n) sc[key] = acc * a.scale;
  }
  __syncthreads();

  float m = -INFINITY;
  for (int t = tid; t < n; t += 256) m = fmaxf(m, sc[t]);
  m = wave_max(m);
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float s = 0.f;
  for (int t = tid; t < n; t += 256) {
    const float p = expf(sc[t] - m);
    sc[t] = p;
    s += p;
  }
  s = wave_sum(s);
  if ((tid & 63) == 0) red[tid >> 6] = s;
  __syncthreads();
  s = red[0] + red[1] + red[2] + red[3];

  const int i = tid % HD, grp = tid / HD;
  const float vnew = vn[i];
  float acc = 0.f;
  for (int pg = grp; pg * kPage < n; pg += G) {
    const bf16_t* vp = a.kv.v + (((size_t)ptl[pg] * H + head) * HD + i) * kPage;
    float vf[16];
    unpack8(*reinterpret_cast<const uint4*>(vp), vf);
    unpack8(*reinterpret_cast<const uint4*>(vp + 8), vf + 8);
    const int lim = min(kPage, n - pg * kPage);
#pragma unroll
    for (int j = 0; j < kPage; ++j)
      if (j < lim) acc += sc[pg * kPage + j] * (pg * kPage + j == pos ? vnew : vf[j]);  // the token's v from LDS
  }
  op[grp][i] = acc;
  __syncthreads();
  if (grp == 0) {
    float t = 0.f;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) t += op[gg][i];
    a.o[frag_index(b, head * HD + i, a.d)] = f2bf(t / s);  // frag layout: A operand of the O projection
  }
}

// ------------------------------------------------------------------ sampler
// One wave per row over A <= 256 bins (4 per lane).  Gumbel-max: the sampled
// bin maximises z/T + g (lowest bin on exact ties); log-probability and
// entropy are those of softmax(z/T).
__global__ __launch_bounds__(256) void sampler_kernel(SamplerArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows) return;
  const float* z = a.z + (size_t)row * a.A;
  float zv[4], zt[4];
  float m = -INFINITY;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int j = lane + 64 * t;
    zv[t] = j < a.A ? z[j] : 0.f;
    zt[t] = j < a.A ? zv[t] / a.temperature : -INFINITY;
    m = fmaxf(m, zt[t]);
  }
  m = wave_max(m);
  float se = 0.f, sz = 0.f;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (lane + 64 * t < a.A) {
      const float e = expf(zt[t] - m);
      se += e;
      sz += e * (zt[t] - m);
    }
  }
  se = wave_sum(se);
  sz = wave_sum(sz);
  const float lse = m + logf(se);
  const float ent = logf(se) - sz / se;

  int out;    // index into [B, n_actions] outputs
  int kbin;   // scored bin
  if (a.gumbel) {
    const int b = row, i = a.step;
    const float* gp = a.gumbel + ((size_t)b * a.n_actions + i) * a.A;
    float best = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = lane + 64 * t;
      if (j < a.A) {
        float s = zt[t] + gp[j];
        if (s != s) s = -INFINITY;
        if (s > best || (s == best && j < bi)) { best = s; bi = j; }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o, kWave);
      const int oi = __shfl_xor(bi, o, kWave);
      if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    if (bi >= a.A) bi = 0;  // every score was NaN
    kbin = bi;
    out = b * a.n_actions + i;
    if (lane == 0) {
      a.tokens[out] = a.action_begin + kbin;
      a.next_tok[b] = a.action_begin + kbin;
    }
  } else {
    out = row;
    kbin = a.given[row] - a.action_begin;
    if (kbin < 0 || kbin >= a.A) {
      if (lane == 0) atomicOr(a.flags, 2u);
      kbin = -1;
    }
  }
  // z/T at the chosen bin, read from the lane that holds it
  const int src_lane = kbin < 0 ? 0 : (kbin & 63), src_t = kbin < 0 ? 0 : (kbin >> 6);
  float mine = zt[0];
#pragma unroll
  for (int t = 1; t < 4; ++t)
    if (t == src_t) mine = zt[t];
  const float ztk = __shfl(mine, src_lane, kWave);
  if (lane == 0) {
    a.logp[out] = kbin < 0 ? __builtin_nanf("") : ztk - lse;
    if (a.entropy) a.entropy[out] = ent;
  }
  if (a.logits_out) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = lane + 64 * t;
      if (j < a.A) a.logits_out[(size_t)out * a.A + j] = zv[t];
    }
  }
}

}  // namespace

hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.n_env <= 0) return hipSuccess;
  const dim3 grid(a.n_env, a.n_heads), block(512);
  if (a.head_dim == 128) hipLaunchKernelGGL(attn_prefill_kernel<128>, grid, block, 0, s, a);
  else if (a.head_dim == 64) hipLaunchKernelGGL(attn_prefill_kernel<64>, grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_decode(const DecodeAttnArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  const dim3 grid(a.n_heads, a.B), block(256);
  if (a.head_dim == 128) hipLaunchKernelGGL(attn_decode_kernel<128>, grid, block, 0, s, a);
  else if (a.head_dim == 64) hipLaunchKernelGGL(attn_decode_kernel<64>, grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_sampler(const SamplerArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.A > 256) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sampler_kernel, dim3((a.rows + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace vla
