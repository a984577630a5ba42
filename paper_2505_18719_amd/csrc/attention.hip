// Causal attention over the paged KV cache on gfx950.
//
// Prefill: one 256-thread workgroup per (64-query block of one environment,
// head); each wave owns 16 queries.  K and V^T are staged through LDS one
// 32-key chunk at a time (double-buffered, one copy per workgroup), scores
// are computed transposed so that P stays in registers in the layout the
// P*V MFMA consumes, and a whole score row (<= 320 keys, the longest sequence
// of one environment) stays in registers, so the softmax is exact.
//
// Decode: one workgroup per (environment, head) and one query; scores and
// P*V in fp32 on the vector ALUs, streaming K rows and transposed V pages with
// 16-byte loads.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int kMaxKeyTiles = 20;  // 320 keys
constexpr int kMaxChunks = kMaxKeyTiles / 2;  // 32-key chunks

// One 32-key chunk of one head staged in LDS.  K rows keep the page layout
// (key-major, HD contiguous) with a 16-byte pad per row; V^T rows (one per
// feature, 16 keys of one page) get a 16-byte pad too.  The pads put the 16
// rows read by one MFMA operand load on distinct bank groups.
template <int HD>
struct AttnChunk {
  static constexpr int KROW = HD * 2 + 16;       // bytes per key row
  static constexpr int VROW = 48;                // bytes per feature row (16 keys + pad)
  static constexpr int KBYTES = 32 * KROW;
  static constexpr int VBYTES = 2 * HD * VROW;
};

// Copy chunk c (pages 2c, 2c+1 of this environment) of head `head` from the
// page pool into registers: each thread moves 16-byte pieces of both pages of
// K and of V^T (coalesced: a page of one head is contiguous).
template <int HD>
struct ChunkRegs {
  static constexpr int PER = (2 * 16 * HD * 2) / (256 * 16);  // 16-byte pieces per thread per tensor
  uint4 k[PER], v[PER];
};

template <int HD>
__device__ __forceinline__ void chunk_load(ChunkRegs<HD>& r, const bf16_t* kpool, const bf16_t* vpool,
                                           const int32_t* pt, int c, int H, int head, bool kv_k, bool kv_v) {
  constexpr int PIECES_PER_PAGE = 16 * HD * 2 / 16;
#pragma unroll
  for (int i = 0; i < ChunkRegs<HD>::PER; ++i) {
    const int piece = threadIdx.x + 256 * i;
    const int pl = piece / PIECES_PER_PAGE, off = piece % PIECES_PER_PAGE;
    const size_t base = ((size_t)pt[2 * c + pl] * H + head) * (16 * HD);
    if (kv_k) r.k[i] = *reinterpret_cast<const uint4*>(kpool + base + off * 8);
    if (kv_v) r.v[i] = *reinterpret_cast<const uint4*>(vpool + base + off * 8);
  }
}

template <int HD>
__device__ __forceinline__ void chunk_store(const ChunkRegs<HD>& r, char* kl, char* vl, bool kv_k, bool kv_v) {
  constexpr int PIECES_PER_PAGE = 16 * HD * 2 / 16;
#pragma unroll
  for (int i = 0; i < ChunkRegs<HD>::PER; ++i) {
    const int piece = threadIdx.x + 256 * i;
    const int pl = piece / PIECES_PER_PAGE, off = piece % PIECES_PER_PAGE;
    if (kv_k) {  // K page: [slot][HD]
      const int slot = off / (HD / 8), j = off % (HD / 8);
      *reinterpret_cast<uint4*>(kl + (pl * 16 + slot) * AttnChunk<HD>::KROW + j * 16) = r.k[i];
    }
    if (kv_v) {  // V^T page: [HD][16 slots]
      const int f = off / 2, half = off % 2;
      *reinterpret_cast<uint4*>(vl + (pl * HD + f) * AttnChunk<HD>::VROW + half * 16) = r.v[i];
    }
  }
}

// Prefill attention, one workgroup per (64-query block of one environment,
// head), 16 queries per wave.  Scores are computed transposed, S^T = K Q^T,
// with the keys of each 32-key chunk assigned to MFMA rows so that the lane
// group g ends up holding keys 8g .. 8g+7 of the chunk for its query: exactly
// the B-operand fragment of P^T in O^T = V^T P^T.  P therefore never leaves
// registers; it enters the MFMA as P_hi + P_lo (two bf16 products, ~16
// significant bits).  The whole score row of a query (<= 320 keys) is kept,
// so the softmax is exact (true maximum, no online rescaling).
template <int HD>
__global__ __launch_bounds__(256) void attn_prefill_kernel(PrefillAttnArgs a) {
  using C = AttnChunk<HD>;
  __shared__ __attribute__((aligned(16))) char klds[2][C::KBYTES];
  __shared__ __attribute__((aligned(16))) char vlds[2][C::VBYTES];
  const int item = blockIdx.x, head = blockIdx.y;
  const int env = a.qblocks[2 * item], q0 = a.qblocks[2 * item + 1];
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int H = a.n_heads;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const int qw = q0 + wave * 16;                 // first query of this wave
  const int kend = min(L, q0 + 64);
  const int nch = (kend + 31) / 32;
  const int32_t* pt = a.page_table + env * a.max_pages;

  constexpr int KS = HD / 32;
  uint4 qf[KS];  // B operand: query r16, features 32 ks + 8g .. +8
  {
    const bf16_t* qp = a.q + (size_t)(row0 + min(qw + r16, L - 1)) * a.d + head * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const uint4*>(qp + ks * 32);
  }
  // MFMA row i of tile t (0: A, 1: B) of a chunk is key 8*(i/4) + 4t + i%4
  const int krowA = 8 * (r16 >> 2) + (r16 & 3);

  // ---- pass 1: scores
  f32x4 sc[kMaxKeyTiles];
#pragma unroll
  for (int t = 0; t < kMaxKeyTiles; ++t) sc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  ChunkRegs<HD> cr;
  chunk_load<HD>(cr, a.kv.k, a.kv.v, pt, 0, H, head, true, false);
  chunk_store<HD>(cr, klds[0], nullptr, true, false);
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    if (c < nch) {
      if (c + 1 < nch) chunk_load<HD>(cr, a.kv.k, a.kv.v, pt, c + 1, H, head, true, false);
      const char* kl = klds[c & 1];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const char* kr = kl + (krowA + 4 * t) * C::KROW + 16 * g;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          sc[2 * c + t] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(kr + ks * 64)), as_bf16x8(qf[ks]),
                                 sc[2 * c + t]);
      }
      if (c + 1 < nch) chunk_store<HD>(cr, klds[(c + 1) & 1], nullptr, true, false);
      __syncthreads();
    }
  }

  // lane holds S(query qw + r16, key 32c + 8g + 4t + r) in sc[2c + t][r]
  const int qpos = qw + r16;
  float mx = -INFINITY;
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c)
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 32 * c + 8 * g + 4 * t + r;
        const bool ok = c < nch && key <= qpos && key < L;
        const float v = ok ? sc[2 * c + t][r] * a.scale : -INFINITY;
        sc[2 * c + t][r] = v;
        mx = fmaxf(mx, v);
      }
  mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
  mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
  float sum = 0.f;
#pragma unroll
  for (int t = 0; t < kMaxKeyTiles; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = sc[t][r] == -INFINITY ? 0.f : expf(sc[t][r] - mx);
      sc[t][r] = p;
      sum += p;
    }
  sum += __shfl_xor(sum, 16, kWave);
  sum += __shfl_xor(sum, 32, kWave);

  // ---- pass 2: O^T = V^T P^T
  constexpr int NB = HD / 16;
  f32x4 o[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  chunk_load<HD>(cr, a.kv.k, a.kv.v, pt, 0, H, head, false, true);
  chunk_store<HD>(cr, nullptr, vlds[0], false, true);
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kMaxChunks; ++c) {
    if (c < nch) {
      if (c + 1 < nch) chunk_load<HD>(cr, a.kv.k, a.kv.v, pt, c + 1, H, head, false, true);
      bf16x8 phi, plo;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = sc[2 * c + t][r];
          const __bf16 h = (__bf16)p;
          phi[4 * t + r] = h;
          plo[4 * t + r] = (__bf16)(p - (float)h);
        }
      // A operand: V^T row (feature nb*16 + r16), keys 8g .. 8g+7 of the chunk
      const char* vl = vlds[c & 1] + (g >> 1) * HD * C::VROW + (g & 1) * 16;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint4 vv = *reinterpret_cast<const uint4*>(vl + (nb * 16 + r16) * C::VROW);
        o[nb] = mfma16(as_bf16x8(vv), phi, o[nb]);
        o[nb] = mfma16(as_bf16x8(vv), plo, o[nb]);
      }
      if (c + 1 < nch) chunk_store<HD>(cr, nullptr, vlds[(c + 1) & 1], false, true);
      __syncthreads();
    }
  }

  // o[nb][r] = O(query qw + r16, feature nb*16 + 4g + r)
  if (qpos < L) {
    const float inv = 1.f / sum;
    // frag layout (the O projection's A operand): 4 consecutive features stay contiguous
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      *reinterpret_cast<uint2*>(a.o + frag_index(row0 + qpos, head * HD + nb * 16 + 4 * g, a.d)) =
          make_uint2(pack2bf(o[nb][0] * inv, o[nb][1] * inv), pack2bf(o[nb][2] * inv, o[nb][3] * inv));
  }
}

template <int HD>
__global__ __launch_bounds__(256) void attn_decode_kernel(DecodeAttnArgs a) {
  constexpr int LPK = HD / 8;          // lanes per key row
  constexpr int KPP = 256 / LPK;       // keys per pass
  constexpr int G = 256 / HD;          // feature groups in P*V
  __shared__ float sc[kMaxKeyTiles * 16];
  __shared__ float qs[HD];
  __shared__ float red[4];
  __shared__ float op[G][HD];
  const int head = blockIdx.x, b = blockIdx.y;
  const int H = a.n_heads, tid = threadIdx.x;
  const int n = a.env_prefix[b] + a.step;  // keys 0 .. n-1
  const int32_t* pt = a.page_table + b * a.max_pages;
  if (tid < HD) qs[tid] = bf2f(a.q[(size_t)b * a.d + head * HD + tid]);
  __syncthreads();

  const int part = tid % LPK;
  float qv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) qv[j] = qs[part * 8 + j];
  for (int base = 0; base < n; base += KPP) {
    const int key = base + tid / LPK;
    float acc = 0.f;
    if (key < n) {
      const int page = pt[key / kPage];
      const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + key % kPage) * HD + part * 8;
      float kf[8];
      unpack8(*reinterpret_cast<const uint4*>(kp), kf);
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
  float acc = 0.f;
  for (int pg = grp; pg * kPage < n; pg += G) {
    const int page = pt[pg];
    const bf16_t* vp = a.kv.v + (((size_t)page * H + head) * HD + i) * kPage;
    float vf[16];
    unpack8(*reinterpret_cast<const uint4*>(vp), vf);
    unpack8(*reinterpret_cast<const uint4*>(vp + 8), vf + 8);
    const int lim = min(kPage, n - pg * kPage);
#pragma unroll
    for (int j = 0; j < kPage; ++j)
      if (j < lim) acc += sc[pg * kPage + j] * vf[j];
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
  const int nrows = a.gumbel ? a.rows : a.rows;
  if (row >= nrows) return;
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
  if (a.n_qblocks <= 0) return hipSuccess;
  const dim3 grid(a.n_qblocks, a.n_heads), block(256);
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
