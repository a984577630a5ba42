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
    const int r = r0 + rr;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = k0 + kk + e;
      float v = 0.f;
      if (r < R && k < K) {
        if (SRC_F32) v = static_cast<const float*>(src)[(size_t)r * ld + k];
        else v = bf2f(static_cast<const bf16_t*>(src)[frag_index(r, k, ld)]);
      }
      t[rr][kk + e] = v;
    }
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
// dx_frag (bf16 frag, K = d) may be null.
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                                          float eps, const float* __restrict__ dy,
                                                          const float* __restrict__ dres, float* __restrict__ dx,
                                                          bf16_t* __restrict__ dx_frag, int d) {
  __shared__ float red[2][4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* xr = x + (size_t)row * d;
  const float* dyr = dy + (size_t)row * d;
  float ss = 0.f, dot = 0.f;
  for (int k = tid; k < d; k += 256) {
    const float xv = xr[k];
    ss += xv * xv;
    dot += xv * g[k] * dyr[k];
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
  for (int k = 8 * tid; k < d; k += 8 * 256) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const size_t i = (size_t)row * d + k + e;
      v[e] = (dres ? dres[i] : 0.f) + r * g[k + e] * dy[i] - xr[k + e] * c;
      dx[i] = v[e];
    }
    if (dx_frag) {
      uint4 o;
      o.x = pack2bf(v[0], v[1]);
      o.y = pack2bf(v[2], v[3]);
      o.z = pack2bf(v[4], v[5]);
      o.w = pack2bf(v[6], v[7]);
      *reinterpret_cast<uint4*>(dx_frag + frag_index(row, k, d)) = o;
    }
  }
}

// SwiGLU backward for h = silu(g) up, with g, up the fp32 gate/up pre-activations
// in the packed interleaved order (columns 64 (j / 32) + j % 32 and +32 of cgu) and
// dh fp32 [M, F] (row stride ldh): writes d[g; up] as bf16 frag in that same order
// (K = 2 Fp) and the forward h = bf16(silu(g) up) as bf16 frag (K = Fp).
__global__ void swiglu_bwd_kernel(const float* __restrict__ cgu, int ldc, const float* __restrict__ dh, int ldh,
                                  int M, int F, int Fp, bf16_t* __restrict__ dgu, bf16_t* __restrict__ h) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int fc = Fp / 8;  // 8-feature chunks per row
  if (i >= (size_t)M * fc) return;
  const int m = (int)(i / fc), j0 = (int)(i % fc) * 8;  // features j0 .. j0 + 7 (one 32-block)
  const int cg = 64 * (j0 / 32) + j0 % 32;
  float dgv[8], duv[8], hv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int j = j0 + e;
    if (j < F) {
      const float gg = cgu[(size_t)m * ldc + cg + e], up = cgu[(size_t)m * ldc + cg + 32 + e];
      const float s = 1.f / (1.f + expf(-gg));
      const float d = dh[(size_t)m * ldh + j];
      dgv[e] = d * up * s * (1.f + gg * (1.f - s));
      duv[e] = d * gg * s;
      hv[e] = gg / (1.f + expf(-gg)) * up;  // the forward epilogue's expression
    } else {
      dgv[e] = duv[e] = hv[e] = 0.f;
    }
  }
  uint4 o;
  o.x = pack2bf(dgv[0], dgv[1]); o.y = pack2bf(dgv[2], dgv[3]); o.z = pack2bf(dgv[4], dgv[5]); o.w = pack2bf(dgv[6], dgv[7]);
  *reinterpret_cast<uint4*>(dgu + frag_index(m, cg, 2 * Fp)) = o;
  o.x = pack2bf(duv[0], duv[1]); o.y = pack2bf(duv[2], duv[3]); o.z = pack2bf(duv[4], duv[5]); o.w = pack2bf(duv[6], duv[7]);
  *reinterpret_cast<uint4*>(dgu + frag_index(m, cg + 32, 2 * Fp)) = o;
  o.x = pack2bf(hv[0], hv[1]); o.y = pack2bf(hv[2], hv[3]); o.z = pack2bf(hv[4], hv[5]); o.w = pack2bf(hv[6], hv[7]);
  *reinterpret_cast<uint4*>(h + frag_index(m, j0, Fp)) = o;
}

// ---- causal attention backward ------------------------------------------------
// Per (environment, head) workgroup of 16 waves.  With P = softmax(scale q k^T)
// (causal) given by the forward's log-sum-exp per query row (P = exp(scale
// q.k - lse)), dP = dO V^T, D_t = dO_t . O_t and dS = P (dP - D):
//   pass 1 (queries): D_t, and dq_t = scale sum_j dS_tj k_j;
//   pass 2 (keys):    dk_j = scale sum_t dS_tj q_t, dv_j = sum_t P_tj dO_t.
// A wave takes one row (query or key) at a time; its lanes hold 8 features
// each, HD / 8 lanes per row of the other side, 512 / HD of those rows per step,
// and reduce their partial dot products with shuffles.  q and k are the
// rotated values the forward attended with; the gradients go back through the
// inverse rotation at each row's position and are written as bf16 into the
// [q; k; v] gradient in the packed weight's column order (frag layout, K = 3 d).
constexpr int kBwdKeys = 320;  // longest sequence (one environment)
constexpr int kBwdWaves = 16;

template <int HD>
__device__ __forceinline__ int bwd_swz(int row) { return row & (HD / 8 - 1); }
// packed column of natural feature f of a rotated head (q, k): pairs (i, i + HD/2) of each
// 32-feature block sit 32 columns apart in 64-column groups
template <int HD>
__device__ __forceinline__ int qk_packed_col(int f) {
  constexpr int half = HD / 2;
  return f < half ? 64 * (f >> 5) + (f & 31) : 64 * ((f - half) >> 5) + 32 + ((f - half) & 31);
}
// 16-byte chunk c of row `row` of a [kBwdKeys, HD] bf16 LDS tile (chunks swizzled per row)
template <int HD>
__device__ __forceinline__ void lds_chunk(const bf16_t* t, int row, int c, float* f8) {
  unpack8(*reinterpret_cast<const uint4*>(t + (row * (HD / 8) + (c ^ bwd_swz<HD>(row))) * 8), f8);
}
template <int LPK>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = LPK / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// sum over the 64 / LPK row groups of a wave (lanes with the same feature chunk)
template <int LPK>
__device__ __forceinline__ float across_groups(float v) {
#pragma unroll
  for (int o = LPK; o < 64; o <<= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
// write features 8c .. 8c + 7 of a q or k gradient back through the rotation; the
// pair partner of chunk c is chunk c ^ (HD / 16), held by lane ^ (HD / 16)
template <int HD>
__device__ __forceinline__ void bwd_store_rot8(const AttnBwdArgs& a, int row, int pos, int head, int region, int c,
                                               const float* g) {
  constexpr int half = HD / 2, hc = HD / 16;
  float out[8];
  const bool first = c < hc;  // features below half
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float other = __shfl_xor(g[e], hc, kWave);
    const int i = (first ? 8 * c : 8 * c - half) + e;  // rotary pair index
    const float2 cs = a.rope[pos * half + i];
    // (g1, g2) of pair i: g1 belongs to feature i, g2 to i + half
    const float g1 = first ? g[e] : other, g2 = first ? other : g[e];
    out[e] = first ? g1 * cs.x + g2 * cs.y : -g1 * cs.y + g2 * cs.x;
  }
  const int base = region * a.d + head * HD, K3 = 3 * a.d;
#pragma unroll
  for (int e = 0; e < 8; ++e) a.dqkv[frag_index(row, base + qk_packed_col<HD>(8 * c + e), K3)] = f2bf(out[e]);
}

template <int HD>
__global__ __launch_bounds__(64 * kBwdWaves, 1) void attn_bwd_q_kernel(AttnBwdArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t ks[kBwdKeys * HD];
  __shared__ __attribute__((aligned(16))) bf16_t vs[kBwdKeys * HD];
  constexpr int LPK = HD / 8, RPS = 64 / LPK;  // lanes per key row, key rows per step
  const int env = blockIdx.x, head = blockIdx.y, H = a.n_heads;
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % LPK, grp = lane / LPK;  // feature chunk, key slot of the step
  const int32_t* pt = a.page_table + env * a.max_pages;
  // K rows (key-major in the cache) and V (feature-major pages) into key-major LDS
  for (int i = tid; i < L * (HD / 8); i += 64 * kBwdWaves) {
    const int j = i / (HD / 8), cc = i % (HD / 8);
    const int page = pt[j / kPage], slot = j % kPage;
    const bf16_t* kp = a.kv.k + (((size_t)page * H + head) * kPage + slot) * HD + 8 * cc;
    *reinterpret_cast<uint4*>(ks + (j * (HD / 8) + (cc ^ bwd_swz<HD>(j))) * 8) = *reinterpret_cast<const uint4*>(kp);
    const bf16_t* vp = a.kv.v + (((size_t)page * H + head) * HD + 8 * cc) * kPage + slot;
    bf16_t v8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v8[e] = vp[e * kPage];
    uint4 o;
    o.x = v8[0] | (uint32_t(v8[1]) << 16); o.y = v8[2] | (uint32_t(v8[3]) << 16);
    o.z = v8[4] | (uint32_t(v8[5]) << 16); o.w = v8[6] | (uint32_t(v8[7]) << 16);
    *reinterpret_cast<uint4*>(vs + (j * (HD / 8) + (cc ^ bwd_swz<HD>(j))) * 8) = o;
  }
  __syncthreads();
  for (int t = wave; t < L; t += kBwdWaves) {
    const int row = row0 + t;
    float q8[8], do8[8], o8[8];
    unpack8(*reinterpret_cast<const uint4*>(a.q + (size_t)row * a.d + head * HD + 8 * c), q8);
    unpack8(*reinterpret_cast<const uint4*>(a.o + frag_index(row, head * HD + 8 * c, a.d)), o8);
    const float* dp = a.dout + (size_t)row * a.d + head * HD + 8 * c;
    float dd = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      do8[e] = bf2f(f2bf(dp[e]));  // dO as the bf16 operand it is in pass 2
      dd += do8[e] * o8[e];
    }
    dd = group_sum<LPK>(dd);  // D_t = dO_t . O_t
    float* st = a.stats + ((size_t)row * H + head) * 2;
    const float lse = st[0];
    if (lane == 0) st[1] = dd;
    float dq[8] = {};
    for (int j0 = 0; j0 <= t; j0 += RPS) {
      const int j = j0 + grp;
      const int jj = min(j, t);  // rows past t read a valid row and contribute 0
      float k8[8], v8[8];
      lds_chunk<HD>(ks, jj, c, k8);
      lds_chunk<HD>(vs, jj, c, v8);
      float sp = 0.f, dpv = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sp += q8[e] * k8[e];
        dpv += do8[e] * v8[e];
      }
      sp = group_sum<LPK>(sp);
      dpv = group_sum<LPK>(dpv);
      const float p = j <= t ? expf(a.scale * sp - lse) : 0.f;
      const float ds = p * (dpv - dd);
#pragma unroll
      for (int e = 0; e < 8; ++e) dq[e] += ds * k8[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) dq[e] = a.scale * across_groups<LPK>(dq[e]);
    if (grp == 0) bwd_store_rot8<HD>(a, row, t, head, 0, c, dq);
  }
}

template <int HD>
__global__ __launch_bounds__(64 * kBwdWaves, 1) void attn_bwd_kv_kernel(AttnBwdArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t qs[kBwdKeys * HD];
  __shared__ __attribute__((aligned(16))) bf16_t os[kBwdKeys * HD];  // dO rounded to bf16
  constexpr int LPK = HD / 8, RPS = 64 / LPK;
  const int env = blockIdx.x, head = blockIdx.y, H = a.n_heads;
  const int L = a.env_len[env], row0 = a.env_row0[env];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % LPK, grp = lane / LPK;
  const int32_t* pt = a.page_table + env * a.max_pages;
  for (int i = tid; i < L * (HD / 8); i += 64 * kBwdWaves) {
    const int t = i / (HD / 8), cc = i % (HD / 8);
    const int at = (t * (HD / 8) + (cc ^ bwd_swz<HD>(t))) * 8;
    *reinterpret_cast<uint4*>(qs + at) =
        *reinterpret_cast<const uint4*>(a.q + (size_t)(row0 + t) * a.d + head * HD + 8 * cc);
    const float* dp = a.dout + (size_t)(row0 + t) * a.d + head * HD + 8 * cc;
    const float4 x0 = *reinterpret_cast<const float4*>(dp), x1 = *reinterpret_cast<const float4*>(dp + 4);
    uint4 o;
    o.x = pack2bf(x0.x, x0.y); o.y = pack2bf(x0.z, x0.w); o.z = pack2bf(x1.x, x1.y); o.w = pack2bf(x1.z, x1.w);
    *reinterpret_cast<uint4*>(os + at) = o;
  }
  __syncthreads();
  for (int j = wave; j < L; j += kBwdWaves) {
    const int page = pt[j / kPage], slot = j % kPage;
    float k8[8], v8[8];
    unpack8(*reinterpret_cast<const uint4*>(a.kv.k + (((size_t)page * H + head) * kPage + slot) * HD + 8 * c), k8);
    const bf16_t* vp = a.kv.v + (((size_t)page * H + head) * HD + 8 * c) * kPage + slot;
#pragma unroll
    for (int e = 0; e < 8; ++e) v8[e] = bf2f(vp[e * kPage]);
    float dk[8] = {}, dv[8] = {};
    for (int t0 = j; t0 < L; t0 += RPS) {
      const int t = t0 + grp;
      const int tt = min(t, L - 1);
      float q8[8], o8[8];
      lds_chunk<HD>(qs, tt, c, q8);
      lds_chunk<HD>(os, tt, c, o8);
      float sp = 0.f, dpv = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sp += q8[e] * k8[e];
        dpv += o8[e] * v8[e];
      }
      sp = group_sum<LPK>(sp);
      dpv = group_sum<LPK>(dpv);
      const float* st = a.stats + ((size_t)(row0 + tt) * H + head) * 2;
      const float p = t < L ? expf(a.scale * sp - st[0]) : 0.f;
      const float ds = p * (dpv - st[1]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        dk[e] += ds * q8[e];
        dv[e] += p * o8[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dk[e] = a.scale * across_groups<LPK>(dk[e]);
      dv[e] = across_groups<LPK>(dv[e]);
    }
    if (grp == 0) {
      const int row = row0 + j, K3 = 3 * a.d;
#pragma unroll
      for (int e = 0; e < 8; ++e) a.dqkv[frag_index(row, 2 * a.d + head * HD + 8 * c + e, K3)] = f2bf(dv[e]);
      bwd_store_rot8<HD>(a, row, j, head, 1, c, dk);
    }
  }
}

// ---- LoRA gradients from a weight gradient ---------------------------------------
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

// B^T of one projection as a skinny-GEMM operand: dst (bf16 frag [64 rows, K]) row c,
// column o0 + o = B[grad_row(o), c] for o < n_cols and c < r, zero elsewhere.
__global__ void pack_bt_kernel(LoraGradArgs a, int K, bf16_t* __restrict__ dst) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= 64 * (K / 8)) return;
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

hipError_t launch_pack_bt(const LoraGradArgs& a, int K, bf16_t* dst, hipStream_t s) {
  if (K % 32 != 0 || a.r < 1 || a.r > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_bt_kernel, dim3((64 * (K / 8) + 255) / 256), dim3(256), 0, s, a, K, dst);
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
  const dim3 grid(a.n_env, a.n_heads), block(64 * kBwdWaves);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(attn_bwd_q_kernel<128>, grid, block, 0, s, a);
    hipLaunchKernelGGL(attn_bwd_kv_kernel<128>, grid, block, 0, s, a);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL(attn_bwd_q_kernel<64>, grid, block, 0, s, a);
    hipLaunchKernelGGL(attn_bwd_kv_kernel<64>, grid, block, 0, s, a);
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
  if (d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(M), dim3(256), 0, s, x, g, eps, dy, dres, dx, dx_frag, d);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(const float* cgu, int ldc, const float* dh, int ldh, int M, int F, int Fp, bf16_t* dgu,
                             bf16_t* h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (Fp % 32 != 0 || F > Fp) return hipErrorInvalidValue;
  const size_t work = (size_t)M * (Fp / 8);
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((work + 255) / 256)), dim3(256), 0, s, cgu, ldc, dh, ldh, M,
                     F, Fp, dgu, h);
  return hipGetLastError();
}

}  // namespace vla
