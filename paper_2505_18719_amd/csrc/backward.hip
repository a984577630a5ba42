// Backward of the teacher-forced pass (the PPO update's gradient through the
// decoder, Sec. 3.3 "Learning Phase"): layout conversions for the backward
// GEMMs, RMSNorm and SwiGLU backward, and the causal attention backward with
// the inverse rotary embedding.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

// dst (bf16 frag [R, kdst]) = x (fp32 row-major, row stride ld) for columns < n; the
// other columns up to kdst and the rows of the last 16-row block past R are zero.
__global__ void to_frag_kernel(const float* __restrict__ x, int ld, int R, int n, int kdst, bf16_t* __restrict__ dst) {
  const int kc = kdst / 8;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int Rp = (R + 15) & ~15;
  if (i >= (size_t)Rp * kc) return;
  const int r = (int)(i / kc), k = (int)(i % kc) * 8;
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (r < R && k + e < n) ? x[(size_t)r * ld + k + e] : 0.f;
  uint4 o;
  o.x = pack2bf(v[0], v[1]);
  o.y = pack2bf(v[2], v[3]);
  o.z = pack2bf(v[4], v[5]);
  o.w = pack2bf(v[6], v[7]);
  *reinterpret_cast<uint4*>(dst + frag_index(r, k, kdst)) = o;
}

// dst[k, r] = src[r, k] into a bf16 frag matrix [K rows, Kd] (Kd >= R, multiple of 32;
// columns R .. Kd and the rows of the last 16-row block past K zero).  The source is
// fp32 row-major (row stride ld) or a bf16 frag matrix of frag width ld.  One
// 64 x 64 tile per 256-thread workgroup through LDS.
template <bool SRC_F32>
__global__ __launch_bounds__(256) void transpose_frag_kernel(const void* __restrict__ src, int ld, int R, int K,
                                                             int Kd, bf16_t* __restrict__ dst) {
  __shared__ float t[64][65];
  const int r0 = blockIdx.x * 64, k0 = blockIdx.y * 64, tid = threadIdx.x;
  // load: thread reads 8 consecutive k of one source row (two rows per thread)
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = tid / 8 + 32 * h, kk = (tid % 8) * 8;
    const int r = r0 + rr, k = k0 + kk;
    float v[8];
    if (r < R && k + 8 <= K) {  // 8 consecutive k: one 16-byte frag chunk, or two float4
      if (SRC_F32) {
        const float* p = static_cast<const float*>(src) + (size_t)r * ld + k;
        const float4 a0 = *reinterpret_cast<const float4*>(p), a1 = *reinterpret_cast<const float4*>(p + 4);
        v[0] = a0.x; v[1] = a0.y; v[2] = a0.z; v[3] = a0.w; v[4] = a1.x; v[5] = a1.y; v[6] = a1.z; v[7] = a1.w;
      } else {
        unpack8(*reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(src) + frag_index(r, k, ld)), v);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] = 0.f;
        if (r < R && k + e < K) {
          if (SRC_F32) v[e] = static_cast<const float*>(src)[(size_t)r * ld + k + e];
          else v[e] = bf2f(static_cast<const bf16_t*>(src)[frag_index(r, k + e, ld)]);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) t[rr][kk + e] = v[e];
  }
  __syncthreads();
  // store: thread writes 8 consecutive destination columns (source rows) of one destination row
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int kk = tid / 8 + 32 * h, rr = (tid % 8) * 8;
    const int k = k0 + kk, r = r0 + rr;
    const int Kp = (K + 15) & ~15;
    if (k >= Kp || r >= Kd) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (k < K) ? t[rr + e][kk] : 0.f;
    uint4 o;
    o.x = pack2bf(v[0], v[1]);
    o.y = pack2bf(v[2], v[3]);
    o.z = pack2bf(v[4], v[5]);
    o.w = pack2bf(v[6], v[7]);
    *reinterpret_cast<uint4*>(dst + frag_index(k, r, Kd)) = o;
  }
}

// RMSNorm backward of y = x r g, r = (mean(x^2) + eps)^(-1/2), for one row per
// workgroup: dx = dres + r (g dy) - x r^3 (sum x g dy) / d.  dres may be null;
// dx_frag (bf16 frag, K = d) may be null.  The row stays in registers: thread t
// takes features 8 (t + 256 j) .. + 8, j < kRmsBwdSteps (d <= 8192, d % 8 == 0).
constexpr int kRmsBwdSteps = 4;
__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a0 = *reinterpret_cast<const float4*>(p), a1 = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a0.x; v[1] = a0.y; v[2] = a0.z; v[3] = a0.w; v[4] = a1.x; v[5] = a1.y; v[6] = a1.z; v[7] = a1.w;
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                                          float eps, const float* __restrict__ dy,
                                                          const float* __restrict__ dres, float* __restrict__ dx,
                                                          bf16_t* __restrict__ dx_frag, int d) {
  __shared__ float red[2][4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const size_t base = (size_t)row * d;
  float xv[kRmsBwdSteps][8], gv[kRmsBwdSteps][8], dv[kRmsBwdSteps][8];
  float ss = 0.f, dot = 0.f;
#pragma unroll
  for (int j = 0; j < kRmsBwdSteps; ++j) {
    const int k = 8 * (tid + 256 * j);
    if (k < d) {
      load8(x + base + k, xv[j]);
      load8(g + k, gv[j]);
      load8(dy + base + k, dv[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ss += xv[j][e] * xv[j][e];
        dot += xv[j][e] * gv[j][e] * dv[j][e];
      }
    }
  }
  ss = wave_sum(ss);
  dot = wave_sum(dot);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = ss;
    red[1][tid >> 6] = dot;
  }
  __syncthreads();
  ss = red[0][0] + red[0][1] + red[0][2] + red[0][3];
  dot = red[1][0] + red[1][1] + red[1][2] + red[1][3];
  const float r = 1.f / sqrtf(ss / d + eps);
  const float c = r * r * r * dot / d;
#pragma unroll
  for (int j = 0; j < kRmsBwdSteps; ++j) {
    const int k = 8 * (tid + 256 * j);
    if (k >= d) continue;
    float rv[8], v[8];
    if (dres) load8(dres + base + k, rv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (dres ? rv[e] : 0.f) + r * gv[j][e] * dv[j][e] - xv[j][e] * c;
    store8(dx + base + k, v);
    if (dx_frag)
      *reinterpret_cast<uint4*>(dx_frag + frag_index(row, k, d)) =
          make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
  }
}

// SwiGLU backward for h = silu(g) up, with g, up the fp32 gate/up pre-activations
// in the packed interleaved order (columns 64 (j / 32) + j % 32 and +32 of cgu) and
// dh fp32 [M, F] (row stride ldh): writes d[g; up] as bf16 frag in that same order
// (K = 2 Fp) and the forward h = bf16(silu(g) up) as bf16 frag (K = Fp).  A wave
// takes one 16-row x 32-feature block, lane (r, u) rows 16 mb + r and features
// 32 jb + 8 u .. + 8, so each of its three stores is one contiguous 1 KB frag
// block; rows >= M of the last block are written as zeros.
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const float* __restrict__ cgu, int ldc,
                                                         const float* __restrict__ dh, int ldh, int M, int F, int Fp,
                                                         bf16_t* __restrict__ dgu, bf16_t* __restrict__ h) {
  const int nj = Fp / 32;
  const size_t w = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= (size_t)((M + 15) / 16) * nj) return;
  const int mb = (int)(w / nj), jb = (int)(w % nj), lane = threadIdx.x & 63;
  const int m = 16 * mb + (lane & 15), j0 = 32 * jb + 8 * (lane >> 4);
  const int cg = 64 * jb + 8 * (lane >> 4);
  float dgv[8], duv[8], hv[8], gv[8], uv[8], dv[8];
  const float* cr = cgu + (size_t)m * ldc + cg;
  if (m < M && j0 + 8 <= F) {
    load8(cr, gv);
    load8(cr + 32, uv);
    load8(dh + (size_t)m * ldh + j0, dv);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool in = m < M && j0 + e < F;
      gv[e] = in ? cr[e] : 0.f;
      uv[e] = in ? cr[32 + e] : 0.f;
      dv[e] = in ? dh[(size_t)m * ldh + j0 + e] : 0.f;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float gg = gv[e], up = uv[e];
    const float s = 1.f / (1.f + expf(-gg));
    const float d = dv[e];
    dgv[e] = d * up * s * (1.f + gg * (1.f - s));
    duv[e] = d * gg * s;
    hv[e] = gg / (1.f + expf(-gg)) * up;  // the forward epilogue's expression
  }
  uint4 o;
  o.x = pack2bf(dgv[0], dgv[1]); o.y = pack2bf(dgv[2], dgv[3]); o.z = pack2bf(dgv[4], dgv[5]); o.w = pack2bf(dgv[6], dgv[7]);
  *reinterpret_cast<uint4*>(dgu + frag_index(m, cg, 2 * Fp)) = o;
  o.x = pack2bf(duv[0], duv[1]); o.y = pack2bf(duv[2], duv[3]); o.z = pack2bf(duv[4], duv[5]); o.w = pack2bf(duv[6], duv[7]);
  *reinterpret_cast<uint4*>(dgu + frag_index(m, cg + 32, 2 * Fp)) = o;
  o.x = pack2bf(hv[0], hv[1]); o.y = pack2bf(hv[2], hv[3]); o.z = pack2bf(hv[4], hv[5]); o.w = pack2bf(hv[6], hv[7]);
  *reinterpret_cast<uint4*>(h + frag_index(m, j0, Fp)) = o;
}

// ---- causal attention backward on the matrix cores -----------------------------
// With P = softmax(scale q k^T) (causal) recovered from the forward's log-sum-exp
// per query row (P = exp(scale q.k - lse)), dP = dO V^T, D_t = dO_t . O_t and
// dS = P (dP - D):  dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO.
// Two passes, each one 512-thread workgroup (8 waves) per (environment, head),
// <= 320 rows, every product a 16x16x32 bf16 MFMA with fp32 accumulation:
//   pass 1 (queries): a wave takes 16-query tiles; per 32-key chunk it forms
//     S^T = K Q^T and dP^T = V dO^T, keys on the MFMA rows in the order that
//     leaves lane group g holding keys 8g .. 8g+7 of the chunk, so dS^T is
//     already the B operand of dQ^T += K^T dS^T.  V (key-major) and K^T (16-key
//     pages) are transposed into LDS once; K rows stream from the cache.  Also
//     writes D and dO rounded to bf16 (row-major) for pass 2.
//   pass 2 (keys): a wave takes 16-key tiles; per 32-query chunk it forms
//     S = Q K^T and dP = dO V^T with queries on the MFMA rows in the same
//     order, so P and dS are the B operands of dV^T += dO^T P and
//     dK^T += Q^T dS.  Q^T and dO^T (16-query pages) are transposed into LDS
//     once; Q and dO rows stream from memory.
// P and dS enter their products as hi + lo bf16 pairs (~16 significant bits);
// q, k, v and dO are the bf16 operands of the forward.  q and k are the rotated
// values the forward attended with: their gradients go back through the inverse
// rotation and are written as bf16 into the [q; k; v] gradient in the packed
// weight's column order (frag layout, K = 3 d).
constexpr int kAbKeys = 320;  // longest sequence (one environment)
constexpr int kAbPages = kAbKeys / kPage;
constexpr int kAbWaves = 8;

// packed column of natural feature f of a rotated head (q, k): pairs (i, i + HD/2) of each
// 32-feature block sit 32 columns apart in 64-column groups
template <int HD>
__device__ __forceinline__ int qk_packed_col(int f) {
  constexpr int half = HD / 2;
  return f < half ? 64 * (f >> 5) + (f & 31) : 64 * ((f - half) >> 5) + 32 + ((f - half) & 31);
}
// Row order of a key- (query-) major MFMA operand: row i of 16-row tile t of 32-row chunk c
// is sequence row 32 c + 8 (i / 4) + 4 t + i % 4, so C rows 4 g + r of tiles t = 0, 1 are
// rows 8 g .. 8 g + 7 of the chunk in lane group g.  ab_slot inverts it.
__device__ __forceinline__ int ab_row(int R) { return 32 * (R >> 5) + 8 * ((R & 15) >> 2) + 4 * ((R >> 4) & 1) + (R & 3); }
__device__ __forceinline__ int ab_slot(int k) {
  const int w = k & 31;
  return 32 * (k >> 5) + 16 * ((w >> 2) & 1) + 4 * (w >> 3) + (w & 3);
}
// 16-byte feature chunk j of LDS row R of a row-major tile is stored at chunk j ^ ab_swz(R)
template <int HD>
__device__ __forceinline__ int ab_swz(int R) {
  return HD == 128 ? (R & 15) : ((R >> 1) & 7);
}
// byte offset of (feature f, rows 8h .. 8h + 7 of a 16-row page) in a paged transposed tile:
// half h of feature f sits at 16-byte unit 2 f + (h ^ ((f >> 3) & 1)) of its page
template <int HD>
__device__ __forceinline__ int ab_page_off(int page, int f, int h) {
  return page * (HD * kPage * 2) + 16 * (2 * f + (h ^ ((f >> 3) & 1)));
}
// transpose of an 8 x 8 bf16 block: out[b] element a = in[a] element b
__device__ __forceinline__ void transpose8(const uint4* in, uint4* out) {
  uint32_t w[32], o[32];
#pragma unroll
  for (int a = 0; a < 8; ++a) {
    w[4 * a] = in[a].x; w[4 * a + 1] = in[a].y; w[4 * a + 2] = in[a].z; w[4 * a + 3] = in[a].w;
  }
#pragma unroll
  for (int b = 0; b < 8; ++b)
#pragma unroll
    for (int ap = 0; ap < 4; ++ap) {
      const uint32_t lo = w[8 * ap + b / 2], hi = w[8 * ap + 4 + b / 2];
      o[4 * b + ap] = (b & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
#pragma unroll
  for (int b = 0; b < 8; ++b) out[b] = make_uint4(o[4 * b], o[4 * b + 1], o[4 * b + 2], o[4 * b + 3]);
}
// element i of hi, lo = v as a hi + lo pair of bf16
__device__ __forceinline__ void split_bf16(float v, bf16x8& hi, bf16x8& lo, int i) {
  const __bf16 h = (__bf16)v;
  hi[i] = h;
  lo[i] = (__bf16)(v - (float)h);
}
// Store a q or k gradient held transposed (acc[nb][r] = gradient of feature 16 nb + 4 g + r,
// times 1 / mul) for sequence position pos through the inverse rotation: pair i = (i, i + HD/2)
// sits in blocks nb and nb + NB/2 of the same lane.
template <int HD>
__device__ __forceinline__ void ab_store_rot(const AttnBwdArgs& a, size_t row, int pos, int head, int region,
                                             const f32x4* acc, float mul, int g) {
  constexpr int NB = HD / 16, half = HD / 2;
  const float2* cs = a.rope + (size_t)pos * half;
  const int base = region * a.d + head * HD, K3 = 3 * a.d;
#pragma unroll
  for (int nb = 0; nb < NB / 2; ++nb) {
    float lo[4], hi[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float2 c = cs[16 * nb + 4 * g + r];
      const float g1 = mul * acc[nb][r], g2 = mul * acc[nb + NB / 2][r];
      lo[r] = g1 * c.x + g2 * c.y;
      hi[r] = -g1 * c.y + g2 * c.x;
    }
    *reinterpret_cast<uint2*>(a.dqkv + frag_index(row, base + qk_packed_col<HD>(16 * nb + 4 * g), K3)) =
        make_uint2(pack2bf(lo[0], lo[1]), pack2bf(lo[2], lo[3]));
    *reinterpret_cast<uint2*>(a.dqkv + frag_index(row, base + qk_packed_col<HD>(16 * nb + 4 * g + half), K3)) =
        make_uint2(pack2bf(hi[0], hi[1]), pack2bf(hi[2], hi[3]));
  }
}

// pass 1, one 16-query tile: queries 16 qt .. 16 qt + 15, keys in chunks 0 .. qt / 2
template <int HD>
__device__ __forceinline__ void ab_dq_tile(const AttnBwdArgs& a, const char* vlds, const char* ktlds, int ptv, int qt,
                                           int L, int row0, int head, int lane) {
  constexpr int KROW = HD * 2, KS = HD / 32, NB = HD / 16;
  const int r16 = lane & 15, g = lane >> 4, H = a.n_heads;
  const int q = qt * 16 + r16;
  const size_t row = (size_t)(row0 + min(q, L - 1));
  // B operands: query q, features 32 ks + 8 g .. + 8
  uint4 qf[KS], df[KS];
  float dd = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const size_t at = row * a.d + head * HD + 32 * ks + 8 * g;
    qf[ks] = *reinterpret_cast<const uint4*>(a.q + at);
    const float4 x0 = *reinterpret_cast<const float4*>(a.dout + at), x1 = *reinterpret_cast<const float4*>(a.dout + at + 4);
    df[ks] = make_uint4(pack2bf(x0.x, x0.y), pack2bf(x0.z, x0.w), pack2bf(x1.x, x1.y), pack2bf(x1.z, x1.w));
    float o8[8], d8[8];
    unpack8(*reinterpret_cast<const uint4*>(a.o + frag_index(row, head * HD + 32 * ks + 8 * g, a.d)), o8);
    unpack8(df[ks], d8);
#pragma unroll
    for (int e = 0; e < 8; ++e) dd += d8[e] * o8[e];
    if (q < L) *reinterpret_cast<uint4*>(a.do16 + at) = df[ks];
  }
  dd += __shfl_xor(dd, 16, kWave);
  dd += __shfl_xor(dd, 32, kWave);  // D_q = dO_q . O_q (dO as its bf16 operand)
  float* st = a.stats + (row * H + head) * 2;
  const float lse = st[0];
  if (q < L && g == 0) st[1] = dd;

  f32x4 dq[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) dq[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int ncq = qt / 2 + 1;
  for (int c = 0; c < ncq; ++c) {
    f32x4 s[2], dp[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      // A operand row r16 of tile t: key 32 c + 8 (r16 / 4) + 4 t + r16 % 4 (clamped into the sequence)
      const int key = min(ab_row(32 * c + 16 * t + r16), L - 1);
      const int page = __shfl(ptv, key / kPage, kWave);
      const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + key % kPage) * HD + 8 * g;
      const char* vr = vlds + (32 * c + 16 * t + r16) * KROW;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s[t] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(kp + 32 * ks)), as_bf16x8(qf[ks]), s[t]);
        dp[t] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(vr + 16 * ((4 * ks + g) ^ ab_swz<HD>(r16)))),
                       as_bf16x8(df[ks]), dp[t]);
      }
    }
    // lane: query q, keys 32 c + 8 g + 4 t + r -> dS^T as the B operand (hi + lo)
    bf16x8 shi, slo;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 32 * c + 8 * g + 4 * t + r;
        const float p = expf(a.scale * s[t][r] - lse);
        const float ds = key <= q ? p * (dp[t][r] - dd) : 0.f;
        split_bf16(ds, shi, slo, 4 * t + r);
      }
    // dQ^T += K^T dS^T: A operand = K^T rows 16 nb + r16, keys 32 c + 8 g .. + 8
    const char* kt0 = ktlds + ab_page_off<HD>(2 * c + (g >> 1), r16, g & 1);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const bf16x8 kv = as_bf16x8(*reinterpret_cast<const uint4*>(kt0 + nb * 512));
      dq[nb] = mfma16(kv, shi, dq[nb]);
      dq[nb] = mfma16(kv, slo, dq[nb]);
    }
  }
  if (q < L) ab_store_rot<HD>(a, row, q, head, 0, dq, a.scale, g);
}

template <int HD>
__global__ __launch_bounds__(64 * kAbWaves, 1) void attn_bwd_dq_kernel(AttnBwdArgs a) {
  constexpr int KROW = HD * 2, VPAGE = HD * kPage * 2, HC = HD / 8;
  __shared__ __attribute__((aligned(1024))) char lds[kAbKeys * KROW + kAbPages * VPAGE];
  char* const vlds = lds;                     // V, key-major rows in ab_row order
  char* const ktlds = lds + kAbKeys * KROW;   // K^T, 16-key pages
  const int env = blockIdx.x, head = blockIdx.y, H = a.n_heads;
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nch = (L + 31) / 32;
  const int32_t* pt = a.page_table + env * a.max_pages;
  // fill: task (8-key group kg, feature chunk fc); keys >= L are zero
  for (int i = threadIdx.x; i < nch * 4 * HC; i += 64 * kAbWaves) {
    const int kg = i / HC, fc = i % HC, k0 = 8 * kg;
    uint4 vin[8], kin[8], vout[8], kout[8];
    if (k0 < L) {
      const int page = pt[kg >> 1], h = kg & 1;
      const bf16_t* vp = a.kv.v + (((size_t)page * H + head) * HD + 8 * fc) * kPage + 8 * h;
      const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + 8 * h) * HD + 8 * fc;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        vin[e] = *reinterpret_cast<const uint4*>(vp + e * kPage);            // feature 8 fc + e, keys k0 ..
        kin[e] = k0 + e < L ? *reinterpret_cast<const uint4*>(kp + e * HD)  // key k0 + e, features 8 fc ..
                            : make_uint4(0, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) vin[e] = kin[e] = make_uint4(0, 0, 0, 0);
    }
    transpose8(vin, vout);  // vout[b]: key k0 + b, features 8 fc ..
    transpose8(kin, kout);  // kout[e]: feature 8 fc + e, keys k0 ..
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int R = ab_slot(k0 + b);
      *reinterpret_cast<uint4*>(vlds + R * KROW + 16 * (fc ^ ab_swz<HD>(R))) =
          k0 + b < L ? vout[b] : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(ktlds + ab_page_off<HD>(kg >> 1, 8 * fc + b, kg & 1)) = kout[b];
    }
  }
  // the environment's page table, one entry per lane (<= 20 pages)
  const int ptv = pt[min(lane, a.max_pages - 1)];
  __syncthreads();
  const int nq = (L + 15) / 16;
  for (int p0 = 0; p0 < nq; p0 += kAbWaves) {  // most expensive tiles first, snake order
    const int p = p0 + (((p0 / kAbWaves) & 1) ? kAbWaves - 1 - wave : wave);
    if (p < nq) ab_dq_tile<HD>(a, vlds, ktlds, ptv, nq - 1 - p, L, row0, head, lane);
  }
}

// pass 2, one 16-key tile: keys 16 kt .. 16 kt + 15, queries in chunks kt / 2 .. nch - 1
template <int HD>
__device__ __forceinline__ void ab_dkv_tile(const AttnBwdArgs& a, const char* qtl, const char* otl, const int32_t* pt,
                                            int kt, int L, int nch, int row0, int head, int lane) {
  constexpr int KS = HD / 32, NB = HD / 16;
  const int r16 = lane & 15, g = lane >> 4, H = a.n_heads;
  const int key = kt * 16 + r16, kc = min(key, L - 1);
  // B operands: key `key`, features 32 ks + 8 g .. + 8
  uint4 kf[KS], vf[KS];
  {
    const int page = pt[kc / kPage], slot = kc % kPage;
    const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + slot) * HD + 8 * g;
    const bf16_t* vp = a.kv.v + (((size_t)page * H + head) * HD + 8 * g) * kPage + slot;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kf[ks] = *reinterpret_cast<const uint4*>(kp + 32 * ks);
      bf16_t v8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = vp[(32 * ks + e) * kPage];
      vf[ks] = make_uint4(v8[0] | (uint32_t(v8[1]) << 16), v8[2] | (uint32_t(v8[3]) << 16),
                          v8[4] | (uint32_t(v8[5]) << 16), v8[6] | (uint32_t(v8[7]) << 16));
    }
  }
  f32x4 dk[NB], dv[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) dk[nb] = dv[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c = kt / 2; c < nch; ++c) {
    f32x4 s[2], dp[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      // A operand row r16 of tile t: query 32 c + 8 (r16 / 4) + 4 t + r16 % 4 (clamped)
      const int qi = min(ab_row(32 * c + 16 * t + r16), L - 1);
      const size_t at = (size_t)(row0 + qi) * a.d + head * HD + 8 * g;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s[t] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(a.q + at + 32 * ks)), as_bf16x8(kf[ks]), s[t]);
        dp[t] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(a.do16 + at + 32 * ks)), as_bf16x8(vf[ks]), dp[t]);
      }
    }
    // lane: key `key`, queries 32 c + 8 g + 4 t + r -> P and dS as B operands (hi + lo)
    bf16x8 phi, plo, shi, slo;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qq = 32 * c + 8 * g + 4 * t + r;
        const float2 ld = *reinterpret_cast<const float2*>(a.stats + ((size_t)(row0 + min(qq, L - 1)) * H + head) * 2);
        const bool live = qq >= key && qq < L;
        const float p = live ? expf(a.scale * s[t][r] - ld.x) : 0.f;
        const float ds = live ? p * (dp[t][r] - ld.y) : 0.f;
        split_bf16(p, phi, plo, 4 * t + r);
        split_bf16(ds, shi, slo, 4 * t + r);
      }
    // dV^T += dO^T P, dK^T += Q^T dS: A operands = rows 16 nb + r16 of the transposed tiles,
    // queries 32 c + 8 g .. + 8
    const int off = ab_page_off<HD>(2 * c + (g >> 1), r16, g & 1);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const bf16x8 ov = as_bf16x8(*reinterpret_cast<const uint4*>(otl + off + nb * 512));
      const bf16x8 qv = as_bf16x8(*reinterpret_cast<const uint4*>(qtl + off + nb * 512));
      dv[nb] = mfma16(ov, phi, dv[nb]);
      dv[nb] = mfma16(ov, plo, dv[nb]);
      dk[nb] = mfma16(qv, shi, dk[nb]);
      dk[nb] = mfma16(qv, slo, dk[nb]);
    }
  }
  if (key < L) {
    const size_t row = (size_t)(row0 + key);
    const int K3 = 3 * a.d;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      *reinterpret_cast<uint2*>(a.dqkv + frag_index(row, 2 * a.d + head * HD + 16 * nb + 4 * g, K3)) =
          make_uint2(pack2bf(dv[nb][0], dv[nb][1]), pack2bf(dv[nb][2], dv[nb][3]));
    ab_store_rot<HD>(a, row, key, head, 1, dk, a.scale, g);
  }
}

template <int HD>
__global__ __launch_bounds__(64 * kAbWaves, 1) void attn_bwd_dkv_kernel(AttnBwdArgs a) {
  constexpr int VPAGE = HD * kPage * 2, HC = HD / 8;
  __shared__ __attribute__((aligned(1024))) char lds[2 * kAbPages * VPAGE];
  char* const qtl = lds;                   // Q^T, 16-query pages
  char* const otl = lds + kAbPages * VPAGE;  // dO^T (bf16), 16-query pages
  const int env = blockIdx.x, head = blockIdx.y;
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nch = (L + 31) / 32;
  // fill: task (8-query group kg, feature chunk fc); queries >= L are zero
  for (int i = threadIdx.x; i < nch * 4 * HC; i += 64 * kAbWaves) {
    const int kg = i / HC, fc = i % HC, t0 = 8 * kg;
    uint4 qin[8], oin[8], qout[8], oout[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const size_t at = (size_t)(row0 + t0 + e) * a.d + head * HD + 8 * fc;
      const bool in = t0 + e < L;
      qin[e] = in ? *reinterpret_cast<const uint4*>(a.q + at) : make_uint4(0, 0, 0, 0);
      oin[e] = in ? *reinterpret_cast<const uint4*>(a.do16 + at) : make_uint4(0, 0, 0, 0);
    }
    transpose8(qin, qout);
    transpose8(oin, oout);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int off = ab_page_off<HD>(kg >> 1, 8 * fc + b, kg & 1);
      *reinterpret_cast<uint4*>(qtl + off) = qout[b];
      *reinterpret_cast<uint4*>(otl + off) = oout[b];
    }
  }
  __syncthreads();
  const int nq = (L + 15) / 16;
  const int32_t* pt = a.page_table + env * a.max_pages;
  for (int p0 = 0; p0 < nq; p0 += kAbWaves) {  // most expensive (earliest) key tiles first, snake order
    const int p = p0 + (((p0 / kAbWaves) & 1) ? kAbWaves - 1 - wave : wave);
    if (p < nq) ab_dkv_tile<HD>(a, qtl, otl, pt, p, L, nch, row0, head, lane);
  }
}

// ---- LoRA gradients ---------------------------------------
// LoRA gradients (W = W0 + s B A): with T1 = X A^T and T2 = dY B over the M rows,
// dL/dB = s dY^T T1 and dL/dA = s T2^T X, the rank-r reductions of dL/dW = dY^T X
// taken without forming it.  Output o of a projection sits at column o0 + o of the
// packed output order of `mode`; grad_row maps it to the natural row, or -1 for a
// padding row or the other half of [gate; up].
__device__ __forceinline__ int grad_row(const LoraGradArgs& a, int o) {
  int part;
  const int j = pack_src_row(a.mode, o, a.head_dim, a.out, part);
  return (j >= 0 && (a.mode != kPackGateUp || part == a.part)) ? j : -1;
}

// B^T of one projection as a skinny-GEMM operand: dst (bf16 frag [rows, K]) row c,
// column o0 + o = B[grad_row(o), c] for o < n_cols and c < r, zero elsewhere.
__global__ void pack_bt_kernel(LoraGradArgs a, int K, int rows, bf16_t* __restrict__ dst) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * (K / 8)) return;
  const int c = i / (K / 8), k0 = (i % (K / 8)) * 8;
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int o = k0 + e - a.o0;
    const int nr = (c < a.r && o >= 0 && o < a.n_cols) ? grad_row(a, o) : -1;
    v[e] = nr >= 0 ? bf2f(a.b[(size_t)nr * a.r + c]) : 0.f;
  }
  uint4 q;
  q.x = pack2bf(v[0], v[1]); q.y = pack2bf(v[2], v[3]); q.z = pack2bf(v[4], v[5]); q.w = pack2bf(v[6], v[7]);
  *reinterpret_cast<uint4*>(dst + frag_index(c, k0, K)) = q;
}

// scale and place a [64, ldc] product: dB[grad_row(o), c] = s C[c, o] (o < n_cols), or
// dA[c, i] = s C[c, i] (i < in)
__global__ void lora_finalize_kernel(LoraGradArgs a, const float* __restrict__ C, int ldc, bool to_b) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int n = to_b ? a.n_cols : a.in;
  if (e >= a.r * n) return;
  const int c = e / n, o = e % n;
  const float v = a.scale * C[(size_t)c * ldc + o];
  if (to_b) {
    const int nr = grad_row(a, o);
    if (nr >= 0) a.db[(size_t)nr * a.r + c] = v;
  } else {
    a.da[(size_t)c * a.in + o] = v;
  }
}

// dst[rows[i]] = src[i] (scatter) or dst[i] = src[rows[i]] (gather), fp32 rows of d
template <bool SCATTER>
__global__ void move_rows_kernel(const float* __restrict__ src, const int32_t* __restrict__ rows, int d,
                                 float* __restrict__ dst) {
  const int i = blockIdx.x, r = rows[i];
  for (int k = threadIdx.x; k < d; k += 256) {
    if (SCATTER) dst[(size_t)r * d + k] = src[(size_t)i * d + k];
    else dst[(size_t)i * d + k] = src[(size_t)r * d + k];
  }
}

}  // namespace

hipError_t launch_pack_bt(const LoraGradArgs& a, int K, int rows, bf16_t* dst, hipStream_t s) {
  if (K % 32 != 0 || a.r < 1 || a.r > 64 || rows % 16 != 0 || rows < a.r || rows > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_bt_kernel, dim3((rows * (K / 8) + 255) / 256), dim3(256), 0, s, a, K, rows, dst);
  return hipGetLastError();
}

hipError_t launch_lora_finalize(const LoraGradArgs& a, const float* C, int ldc, bool to_b, hipStream_t s) {
  const int n = to_b ? a.n_cols : a.in;
  if (a.r < 1 || a.r > 64 || n <= 0 || n > ldc) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lora_finalize_kernel, dim3((a.r * n + 255) / 256), dim3(256), 0, s, a, C, ldc, to_b);
  return hipGetLastError();
}

hipError_t launch_move_rows(const float* src, const int32_t* rows, int R, int d, float* dst, bool scatter,
                            hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (scatter) hipLaunchKernelGGL(move_rows_kernel<true>, dim3(R), dim3(256), 0, s, src, rows, d, dst);
  else hipLaunchKernelGGL(move_rows_kernel<false>, dim3(R), dim3(256), 0, s, src, rows, d, dst);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const AttnBwdArgs& a, hipStream_t s) {
  if (a.n_env <= 0) return hipSuccess;
  if (a.max_pages < 1 || a.max_pages > 64 || !a.do16) return hipErrorInvalidValue;
  const dim3 grid(a.n_env, a.n_heads), block(64 * kAbWaves);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<128>, grid, block, 0, s, a);
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<128>, grid, block, 0, s, a);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<64>, grid, block, 0, s, a);
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<64>, grid, block, 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_to_frag(const float* x, int ld, int R, int n, int kdst, bf16_t* dst, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (kdst % 32 != 0 || n > kdst) return hipErrorInvalidValue;
  const size_t work = (size_t)((R + 15) & ~15) * (kdst / 8);
  hipLaunchKernelGGL(to_frag_kernel, dim3((unsigned)((work + 255) / 256)), dim3(256), 0, s, x, ld, R, n, kdst, dst);
  return hipGetLastError();
}

hipError_t launch_transpose_frag(const void* src, bool src_f32, int ld, int R, int K, int Kd, bf16_t* dst,
                                 hipStream_t s) {
  if (R <= 0 || K <= 0) return hipSuccess;
  if (Kd % 32 != 0 || Kd < R) return hipErrorInvalidValue;
  // tiles cover rows up to Kd (zero columns) and destination rows up to K rounded to 16
  const dim3 grid((Kd + 63) / 64, (((K + 15) & ~15) + 63) / 64);
  if (src_f32) hipLaunchKernelGGL(transpose_frag_kernel<true>, grid, dim3(256), 0, s, src, ld, R, K, Kd, dst);
  else hipLaunchKernelGGL(transpose_frag_kernel<false>, grid, dim3(256), 0, s, src, ld, R, K, Kd, dst);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(const float* x, const float* g, float eps, const float* dy, const float* dres,
                              float* dx, bf16_t* dx_frag, int M, int d, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (d % 8 != 0 || d > 8 * 256 * kRmsBwdSteps) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(M), dim3(256), 0, s, x, g, eps, dy, dres, dx, dx_frag, d);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(const float* cgu, int ldc, const float* dh, int ldh, int M, int F, int Fp, bf16_t* dgu,
                             bf16_t* h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (Fp % 32 != 0 || F > Fp || !cgu || !h || !dh || !dgu) return hipErrorInvalidValue;
  const size_t waves = (size_t)((M + 15) / 16) * (Fp / 32);
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, cgu, ldc, dh, ldh, M, F,
                     Fp, dgu, h);
  return hipGetLastError();
}

}  // namespace vla
