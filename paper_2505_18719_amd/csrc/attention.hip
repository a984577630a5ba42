// Causal attention over the paged KV cache on gfx950.
//
// Prefill: one 256-thread workgroup per (64-query block of one environment,
// head); each wave owns 16 queries.  Scores S = Q K^T / sqrt(hd) come from
// v_mfma_f32_16x16x32_bf16 with the key rows read straight from their pages;
// a whole score row (<= 320 keys, the longest sequence of one environment)
// stays in registers, so the softmax is exact (true row maximum, no online
// rescaling).  P goes through LDS into the MFMA A-operand layout and P*V runs
// as two bf16 MFMAs (P = P_hi + P_lo) against the transposed V pages, which
// keeps P at ~16 significant bits.
//
// Decode: one workgroup per (environment, head) and one query; scores and
// P*V in fp32 on the vector ALUs, streaming K rows and transposed V pages with
// 16-byte loads.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int kMaxKeyTiles = 20;  // 320 keys
constexpr int kPRow = kMaxKeyTiles * 16 + 4;

template <int HD>
__global__ __launch_bounds__(256) void attn_prefill_kernel(PrefillAttnArgs a) {
  __shared__ float pl[4][16][kPRow];
  const int item = blockIdx.x, head = blockIdx.y;
  const int env = a.qblocks[2 * item], q0 = a.qblocks[2 * item + 1];
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int H = a.n_heads;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const int qw = q0 + wave * 16;
  const int kend = min(L, q0 + 64);
  const int nkt = (kend + 15) / 16;
  const int32_t* pt = a.page_table + env * a.max_pages;

  constexpr int KS = HD / 32;
  uint4 qf[KS];
  {
    const int qrow = min(qw + r16, L - 1);
    const bf16_t* qp = a.q + (size_t)(row0 + qrow) * a.d + head * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const uint4*>(qp + ks * 32);
  }

  f32x4 sc[kMaxKeyTiles];
#pragma unroll
  for (int kt = 0; kt < kMaxKeyTiles; ++kt) {
    sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (kt < nkt) {
      const int page = pt[kt];
      const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + r16) * HD + 8 * g;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sc[kt] = mfma16(as_bf16x8(qf[ks]), as_bf16x8(*reinterpret_cast<const uint4*>(kp + ks * 32)), sc[kt]);
    }
  }

  // lane holds queries qw + 4g + r (r < 4) against key kt*16 + r16
  float mx[4], sum[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) mx[r] = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < kMaxKeyTiles; ++kt) {
    if (kt < nkt) {
      const int key = kt * 16 + r16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qpos = qw + 4 * g + r;
        const float v = (key <= qpos && key < L) ? sc[kt][r] * a.scale : -INFINITY;
        sc[kt][r] = v;
        mx[r] = fmaxf(mx[r], v);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    mx[r] = group16_max(mx[r]);
    sum[r] = 0.f;
  }
#pragma unroll
  for (int kt = 0; kt < kMaxKeyTiles; ++kt) {
    if (kt < nkt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = (sc[kt][r] == -INFINITY) ? 0.f : expf(sc[kt][r] - mx[r]);
        sum[r] += p;
        pl[wave][4 * g + r][kt * 16 + r16] = p;
      }
    }
  }
  if (nkt & 1) {  // zero the unused half of the last 32-key chunk
#pragma unroll
    for (int r = 0; r < 4; ++r) pl[wave][4 * g + r][nkt * 16 + r16] = 0.f;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) sum[r] = group16_sum(sum[r]);
  __syncthreads();

  constexpr int NB = HD / 16;
  f32x4 o[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nch = (nkt + 1) / 2;
  for (int ch = 0; ch < nch; ++ch) {
    const float* pr = &pl[wave][r16][ch * 32 + 8 * g];
    bf16x8 phi, plo;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = pr[j];
      const __bf16 h = (__bf16)p;
      phi[j] = h;
      plo[j] = (__bf16)(p - (float)h);
    }
    const int tile = 2 * ch + (g >> 1);
    const bool valid = tile < nkt;
    const bf16_t* vp = a.kv.v + ((size_t)(valid ? pt[tile] : 0) * H + head) * HD * kPage + 8 * (g & 1);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const uint4 vv = valid ? *reinterpret_cast<const uint4*>(vp + (size_t)(nb * 16 + r16) * kPage)
                             : make_uint4(0, 0, 0, 0);
      o[nb] = mfma16(phi, as_bf16x8(vv), o[nb]);
      o[nb] = mfma16(plo, as_bf16x8(vv), o[nb]);
    }
  }

#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qpos = qw + 4 * g + r;
    if (qpos >= L) continue;
    const float inv = 1.f / sum[r];
    bf16_t* op = a.o + (size_t)(row0 + qpos) * a.d + head * HD + r16;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) op[nb * 16] = f2bf(o[nb][r] * inv);
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
    a.o[(size_t)b * a.d + head * HD + i] = f2bf(t / s);
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
