// Memory-bound kernels of the VLA rollout path on gfx950: input assembly,
// RMSNorm (one wave per row, fp32 statistics), the consumers of the decode
// GEMM's split-K partials (residual add + RMSNorm, SwiGLU, RoPE + KV append,
// logits), and one-time weight repacking.  All loads and stores are 16-byte
// vectors where the layout allows.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

// ------------------------------------------------------------------ embed
// x^0 rows of each environment: n_visual projected visual embeddings, then the
// embedding rows of its prompt ids, then (teacher-forced pass) its actions.
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  const int row = blockIdx.x;
  const int env = a.row_env[row], pos = a.row_pos[row];
  const bf16_t* src;
  if (pos < a.n_visual) {
    src = a.vis + ((size_t)env * a.n_visual + pos) * a.d;
  } else {
    int id;
    if (pos < a.env_prefix[env]) id = a.prompt_ids[a.env_prompt_off[env] + pos - a.n_visual];
    else id = a.actions[env * a.n_actions + pos - a.env_prefix[env]];
    if (id < 0 || id >= a.vocab) {
      if (threadIdx.x == 0) atomicOr(a.flags, 1u);
      src = nullptr;
    } else {
      src = a.emb + (size_t)id * a.d;
    }
  }
  float* dst = a.x + (size_t)row * a.d;
  for (int c = threadIdx.x * 8; c < a.d; c += 256 * 8) {
    float f[8];
    if (src) unpack8(*reinterpret_cast<const uint4*>(src + c), f);
    else
#pragma unroll
      for (int i = 0; i < 8; ++i) f[i] = 0.f;
    reinterpret_cast<float4*>(dst + c)[0] = make_float4(f[0], f[1], f[2], f[3]);
    reinterpret_cast<float4*>(dst + c)[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
}

// ------------------------------------------------------------------ RMSNorm
// One wave per row: u = bf16(x * rsqrt(mean(x^2) + eps) * g), row-major (row stride ldu).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x, int ldx,
                                                      const int32_t* __restrict__ rows,
                                                      const float* __restrict__ g, float eps,
                                                      bf16_t* __restrict__ u, int ldu, int M, int d) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= M) return;
  const int src = rows ? rows[i] : i;
  const float* xr = x + (size_t)src * ldx;
  float ss = 0.f;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float r = rsqrtf(ss / (float)d + eps);
  bf16_t* ur = u + (size_t)i * ldu;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    const float4 w = *reinterpret_cast<const float4*>(g + c);
    uint2 o;
    o.x = pack2bf(v.x * r * w.x, v.y * r * w.y);
    o.y = pack2bf(v.z * r * w.z, v.w * r * w.w);
    *reinterpret_cast<uint2*>(ur + c) = o;
  }
}

// RMSNorm into frag layout.  A workgroup of RPW waves normalises RPW rows of
// one 16-row frag block (RPW = 16: the whole block; 8: one half), one wave per
// row: the wave reads its row once into registers (NJ float4 per lane, 1 KB
// per load instruction), reduces the mean square, and writes the scaled bf16
// row into LDS, row-major with a 16-byte pad per row; the workgroup then reads
// LDS in frag order (the pad puts the 8 rows of one 16-lane read phase on
// distinct banks) and writes each 1 KB block as one contiguous store per 64
// (or 32) lanes.  Rows past M are written as zeros.
template <int NJ, int RPW>
__global__ __launch_bounds__(64 * RPW) void rmsnorm_frag_kernel(const float* __restrict__ x, int ldx,
                                                                const int32_t* __restrict__ rows,
                                                                const float* __restrict__ g, float eps,
                                                                bf16_t* __restrict__ u, int M, int d) {
  extern __shared__ uint4 norm_lds[];
  char* ls = reinterpret_cast<char*>(norm_lds);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * RPW, nj = d / 256;
  const int lrow = 2 * d + 16;  // LDS bytes per row
  char* lr = ls + wave * lrow + 8 * lane;
  if (r0 + wave < M) {  // wave-uniform
    const int i = r0 + wave;
    const float* xr = x + (size_t)(rows ? rows[i] : i) * ldx + 4 * lane;
    float4 v[NJ];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < nj) v[j] = *reinterpret_cast<const float4*>(xr + 256 * j);
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < nj) ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
    ss = wave_sum(ss);
    const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < nj) {
        const float4 gv = *reinterpret_cast<const float4*>(g + 4 * lane + 256 * j);
        *reinterpret_cast<uint2*>(lr + 512 * j) =
            make_uint2(pack2bf(v[j].x * r * gv.x, v[j].y * r * gv.y), pack2bf(v[j].z * r * gv.z, v[j].w * r * gv.w));
      }
  } else {
    for (int j = 0; j < nj; ++j) *reinterpret_cast<uint2*>(lr + 512 * j) = make_uint2(0, 0);
  }
  __syncthreads();
  // block kb of the 16-row block: lane l = row % 16 + 16 (k % 32 / 8) holds 16 bytes
  constexpr int LPB = 4 * RPW;  // lanes of a block this workgroup writes
  const int idx = threadIdx.x % LPB, rr = idx % RPW, q = idx / RPW;
  const int ro = r0 & 15, l = ro + rr + 16 * q;
  bf16_t* ub = u + frag_index(r0 & ~15, 0, d) + 8 * l;
  const char* src = ls + rr * lrow + 16 * q;
  for (int kb = threadIdx.x / LPB; kb < d / 32; kb += 16)
    *reinterpret_cast<uint4*>(ub + (size_t)kb * 512) = *reinterpret_cast<const uint4*>(src + 64 * kb);
}

// Block-wide sum over 256 threads.
__device__ __forceinline__ float block_sum256(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return sh[0] + sh[1] + sh[2] + sh[3];
}

constexpr int kMaxPerThread = 32;  // d <= 8192

__global__ __launch_bounds__(256) void embed_token_norm_kernel(const int32_t* tok, const bf16_t* emb, float* x,
                                                               bf16_t* u, const float* g, float eps, int d,
                                                               int vocab, uint32_t* flags) {
  __shared__ float sh[4];
  const int b = blockIdx.x;
  int id = tok[b];
  const bool ok = id >= 0 && id < vocab;
  if (!ok && threadIdx.x == 0) atomicOr(flags, 1u);
  float v[kMaxPerThread];
  float ss = 0.f;
  const int n = (d / 4 + 255) / 256;  // groups of 4 columns per thread
#pragma unroll
  for (int t = 0; t < kMaxPerThread / 4; ++t) {
    if (t >= n) break;
    const int c = 4 * (threadIdx.x + 256 * t);
    if (c >= d) {
      v[4 * t] = v[4 * t + 1] = v[4 * t + 2] = v[4 * t + 3] = 0.f;
      continue;
    }
    const uint2 e = ok ? *reinterpret_cast<const uint2*>(emb + (size_t)id * d + c) : make_uint2(0, 0);
    v[4 * t] = __uint_as_float(e.x << 16);
    v[4 * t + 1] = __uint_as_float(e.x & 0xffff0000u);
    v[4 * t + 2] = __uint_as_float(e.y << 16);
    v[4 * t + 3] = __uint_as_float(e.y & 0xffff0000u);
    ss += v[4 * t] * v[4 * t] + v[4 * t + 1] * v[4 * t + 1] + v[4 * t + 2] * v[4 * t + 2] +
          v[4 * t + 3] * v[4 * t + 3];
  }
  ss = block_sum256(ss, sh);
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int t = 0; t < kMaxPerThread / 4; ++t) {
    if (t >= n) break;
    const int c = 4 * (threadIdx.x + 256 * t);
    if (c >= d) break;
    const float4 gv = *reinterpret_cast<const float4*>(g + c);
    *reinterpret_cast<float4*>(x + (size_t)b * d + c) = make_float4(v[4 * t], v[4 * t + 1], v[4 * t + 2], v[4 * t + 3]);
    *reinterpret_cast<uint2*>(u + frag_index(b, c, d)) =
        make_uint2(pack2bf(v[4 * t] * r * gv.x, v[4 * t + 1] * r * gv.y),
                   pack2bf(v[4 * t + 2] * r * gv.z, v[4 * t + 3] * r * gv.w));
  }
}


// One 1024-thread workgroup per row: 4 consecutive columns per thread and
// pass (two passes cover d <= 8192), every partial slot's float4 in flight together.
__global__ __launch_bounds__(1024) void reduce_residual_norm_kernel(const float* __restrict__ part, SkinnyPlan p,
                                                                    float* __restrict__ x, bf16_t* __restrict__ u,
                                                                    const float* __restrict__ g, float eps, int M,
                                                                    int d) {
  __shared__ float sh[16];
  const int m = blockIdx.x;
  float4 v[2];
  float ss = 0.f;
#pragma unroll
  for (int t = 0; t < 2; ++t) {  // d <= 8192
    const int c = 4 * (threadIdx.x + 1024 * t);
    if (c >= d) break;
    const float4 a = sum_slots4(part + (size_t)m * d + c, (size_t)M * d, skinny_slots(p, c >> 6),
                                *reinterpret_cast<const float4*>(x + (size_t)m * d + c));
    v[t] = a;
    ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) ss += sh[w];
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int c = 4 * (threadIdx.x + 1024 * t);
    if (c >= d) break;
    const float4 gv = *reinterpret_cast<const float4*>(g + c);
    *reinterpret_cast<float4*>(x + (size_t)m * d + c) = v[t];
    *reinterpret_cast<uint2*>(u + frag_index(m, c, d)) =
        make_uint2(pack2bf(v[t].x * r * gv.x, v[t].y * r * gv.y), pack2bf(v[t].z * r * gv.z, v[t].w * r * gv.w));
  }
}

__global__ __launch_bounds__(256) void reduce_sum_kernel(const float* __restrict__ part, SkinnyPlan p,
                                                         float* __restrict__ z, int M, int N) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)M * N) return;
  const int m = (int)(i / N), n = (int)(i % N);
  z[i] = skinny_sum(part, p, M, p.tiles * 64, m, n);
}

__global__ __launch_bounds__(256) void reduce_swiglu_kernel(const float* __restrict__ part, SkinnyPlan p,
                                                            bf16_t* __restrict__ h, int ldh, int M, int F) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;  // group of 4 consecutive j
  if (i >= (size_t)M * (F / 4)) return;
  const int m = (int)(i / (F / 4)), j = 4 * (int)(i % (F / 4));
  const int N = p.tiles * 64;
  const int cg = 64 * (j >> 5) + (j & 31);  // gate columns cg .. cg+3, up columns 32 further (one 64-column tile)
  const int ns = skinny_slots(p, cg >> 6);
  const float* pr = part + (size_t)m * N + cg;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  const float4 gs = sum_slots4(pr, (size_t)M * N, ns, z), us = sum_slots4(pr + 32, (size_t)M * N, ns, z);
  auto sw = [](float a, float b) { return a / (1.f + expf(-a)) * b; };
  *reinterpret_cast<uint2*>(h + frag_index(m, j, ldh)) =
      make_uint2(pack2bf(sw(gs.x, us.x), sw(gs.y, us.y)), pack2bf(sw(gs.z, us.z), sw(gs.w, us.w)));
}

// ------------------------------------------------------------------ repacking
// One 16-byte chunk (8 K elements) of destination row r per thread, written in
// frag layout.  The source row (or a zero row) follows the packing mode:
//  kPackRows:   source row r, rows >= src_rows zero, K elements >= src_cols zero
//  kPackQk:     q/k rows of each head reordered so that each 64-row block holds
//               rotary pairs 32 rows apart: block b = rows [32b, 32b+32) then
//               [half+32b, half+32b+32)
//  kPackGateUp: [gate; up] interleaved in blocks of 32 rows, zero rows past src_rows
__global__ __launch_bounds__(256) void pack_frag_kernel(PackArgs a) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int kc = a.K / 8;
  if (i >= (size_t)a.rows * kc) return;
  const int r = (int)(i / kc), k = (int)(i % kc) * 8;
  int part;
  const int j = pack_src_row(a.mode, r, a.head_dim, a.src_rows, part);
  const bf16_t* src = j < 0 ? nullptr : (part ? a.src2 : a.src) + (size_t)j * a.src_ld;
  bf16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (src && k + e < a.src_cols) ? src[k + e] : (bf16_t)0;
  uint4 o;
  o.x = v[0] | (uint32_t(v[1]) << 16);
  o.y = v[2] | (uint32_t(v[3]) << 16);
  o.z = v[4] | (uint32_t(v[5]) << 16);
  o.w = v[6] | (uint32_t(v[7]) << 16);
  *reinterpret_cast<uint4*>(a.dst + frag_index(r, k, a.K)) = o;
}

// a[r, i] = lo_i + (k + 1/2) (hi_i - lo_i) / bins for bin k = tokens[r, i] - action_begin,
// NaN outside the bins; one thread per element.
__global__ void extract_actions_kernel(const int32_t* __restrict__ tokens, int n_elems, int n_dims, int action_begin,
                                       int bins, const float* __restrict__ lo, const float* __restrict__ hi,
                                       float* __restrict__ out) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n_elems) return;
  const int dim = i % n_dims;
  const int k = tokens[i] - action_begin;
  const float l = lo[dim];
  out[i] = (k >= 0 && k < bins) ? l + ((float)k + 0.5f) * (hi[dim] - l) / (float)bins : __builtin_nanf("");
}

// Row i of the compact buffers takes row rows[i]: the fp32 residual row and the
// bf16 frag-layout row (8 elements = 16 bytes per thread step).
__global__ void gather_rows_kernel(const float* __restrict__ x, const bf16_t* __restrict__ o,
                                   const int32_t* __restrict__ rows, int d, float* __restrict__ xc,
                                   bf16_t* __restrict__ oc) {
  const int i = blockIdx.x, r = rows[i];
  for (int k = 8 * threadIdx.x; k < d; k += 8 * 256) {
    const float4* xs = reinterpret_cast<const float4*>(x + (size_t)r * d + k);
    float4* xd = reinterpret_cast<float4*>(xc + (size_t)i * d + k);
    xd[0] = xs[0];
    xd[1] = xs[1];
    *reinterpret_cast<uint4*>(oc + frag_index(i, k, d)) = *reinterpret_cast<const uint4*>(o + frag_index(r, k, d));
  }
}

__global__ void bf16_to_f32_kernel(float* dst, const bf16_t* src, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = bf2f(src[i]);
}

__global__ void fill_zero_kernel(uint4* dst, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
    dst[i] = make_uint4(0, 0, 0, 0);
}

}  // namespace

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_kernel, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

namespace {
template <int NJ, int RPW>
hipError_t launch_norm_frag(const float* x, int ldx, const int32_t* rows, const float* g, float eps, bf16_t* u,
                            int M, int d, hipStream_t s) {
  const size_t lds = (size_t)RPW * (2 * d + 16);
  static bool attr_set = false;  // dynamic LDS above 64 KB must be allowed once per kernel
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&rmsnorm_frag_kernel<NJ, RPW>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)(RPW * (2 * 256 * NJ + 16)));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((rmsnorm_frag_kernel<NJ, RPW>), dim3((M + RPW - 1) / RPW), dim3(64 * RPW), lds, s, x, ldx, rows,
                     g, eps, u, M, d);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_rmsnorm(const float* x, int ldx, const int32_t* rows, const float* g, float eps, bf16_t* u,
                          int ldu, int M, int d, hipStream_t s, bool frag) {
  if (M <= 0) return hipSuccess;
  if (d % 4 != 0 || (frag && d % 32 != 0)) return hipErrorInvalidValue;
  if (frag) {
    if (d % 256 != 0 || d > 8192) return hipErrorInvalidValue;
    if (d <= 4096) return launch_norm_frag<16, 8>(x, ldx, rows, g, eps, u, M, d, s);
    return launch_norm_frag<32, 8>(x, ldx, rows, g, eps, u, M, d, s);
  }
    hipLaunchKernelGGL(rmsnorm_kernel, dim3((M + 3) / 4), dim3(256), 0, s, x, ldx, rows, g, eps, u, ldu, M, d);
  return hipGetLastError();
}

hipError_t launch_embed_token_norm(const int32_t* tok, const bf16_t* emb, float* x, bf16_t* u, const float* g,
                                   float eps, int B, int d, int vocab, uint32_t* flags, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (d > 256 * kMaxPerThread || d % 32 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_token_norm_kernel, dim3(B), dim3(256), 0, s, tok, emb, x, u, g, eps, d, vocab, flags);
  return hipGetLastError();
}

hipError_t launch_reduce_residual_norm(const float* part, const SkinnyPlan& p, float* x, bf16_t* u, const float* g,
                                       float eps, int M, int d, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (d > 8192 || d % 64 != 0 || p.tiles * 64 != d) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_residual_norm_kernel, dim3(M), dim3(1024), 0, s, part, p, x, u, g, eps, M, d);
  return hipGetLastError();
}

hipError_t launch_reduce_sum(const float* part, const SkinnyPlan& p, float* z, int M, int N, hipStream_t s) {
  const size_t n = (size_t)M * N;
  if (n == 0) return hipSuccess;
  if (N > p.tiles * 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part, p, z, M, N);
  return hipGetLastError();
}

hipError_t launch_reduce_swiglu(const float* part, const SkinnyPlan& p, bf16_t* h, int ldh, int M, int F,
                                hipStream_t s) {
  const size_t n = (size_t)M * (F / 4);
  if (n == 0) return hipSuccess;
  if (2 * F > p.tiles * 64 || F % 32 != 0 || ldh < F) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_swiglu_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part, p, h, ldh, M, F);
  return hipGetLastError();
}

// LoRA merge, one 256-thread workgroup per 64 rows x 64 K columns.  Rows are
// the projection's own rows in packed order: for the interleaved [gate; up]
// weight only the 32-row halves of `part`, so no workgroup computes rows it
// does not write.  The update B A of the tile is a 64 x 64 x rank product on
// MFMA: wave w takes rows 16 w .. 16 w + 15, its A operand the 16 B rows of
// their source rows (contiguous 16-byte reads), its B operand the adapter's A
// factor staged transposed in LDS.  The original weights are loaded first;
// each wave stages its fp32 update in its own LDS rows (no workgroup barrier
// after the staging of A), adds two 8-element chunks per lane to the original
// weights, rounds to bf16 and writes them in frag layout.  (Measured: wider
// tiles that reuse the staged A over 128 or 256 columns are slower, 7.7 and
// 12.1 ms against 6.9 ms for every projection of the 7B shape at rank 32:
// fewer workgroups fit on a CU to cover the loads' latency.)
constexpr int kMergeCols = 64;

// Rows of the projection a merge computes (for [gate; up], the part's half of the packed rows).
__host__ __device__ inline int merge_rows(const MergeArgs& a) { return a.mode == kPackGateUp ? a.rows / 2 : a.rows; }

// Tile (rows 64 rb .., columns kMergeCols cb ..) of one merge.
__device__ __forceinline__ void merge_tile(const MergeArgs& a, int rb, int cb) {
  __shared__ __attribute__((aligned(16))) bf16_t at[kMergeCols][72];  // A^T: [column][rank], padded rows
  __shared__ float dws[4][16][68];                                     // per wave: the block's update of its rows
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c0 = cb * kMergeCols;
  const int nblk = min(kMergeCols, a.K - c0) / 64;  // K % 64 == 0
  const int RK = (a.rank + 31) / 32 * 32;
  const bool gu = a.mode == kPackGateUp;
  const int nrows = merge_rows(a);
  // packed row of the projection's row l
  auto prow = [&](int l) { return gu ? 64 * (l >> 5) + 32 * a.part + (l & 31) : l; };
  // this lane's two 8-column chunks of each block: row 16 wave + e / 8, columns 8 (e % 8), e = lane + 64 t
  int crow[2], csrc[2];
  bool cin[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int l = rb * 64 + 16 * wave + (lane + 64 * t) / 8;
    cin[t] = l < nrows;
    crow[t] = prow(l);
    int pt;
    csrc[t] = cin[t] ? pack_src_row(a.mode, crow[t], a.head_dim, a.src_rows, pt) : -1;
  }
  uint4 w0v[kMergeCols / 64][2];
#pragma unroll
  for (int cb = 0; cb < kMergeCols / 64; ++cb)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int col = c0 + 64 * cb + 8 * ((lane + 64 * t) % 8);
      w0v[cb][t] = make_uint4(0, 0, 0, 0);  // zero rows and columns of the packed layout
      if (cb < nblk && csrc[t] >= 0 && col < a.src_cols)  // src_cols % 8 == 0: a chunk is wholly in or out
        w0v[cb][t] = *reinterpret_cast<const uint4*>(a.w0 + (size_t)csrc[t] * a.src_ld + col);
    }
  // this lane's A-operand row (row 16 wave + lane % 16) of B, both rank halves
  const int lb = rb * 64 + 16 * wave + (lane & 15);
  int part;
  const int j = lb < nrows ? pack_src_row(a.mode, prow(lb), a.head_dim, a.src_rows, part) : -1;
  uint4 bv[2];
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) {
    const int k = 32 * kc + 8 * (lane >> 4);
    bv[kc] = make_uint4(0, 0, 0, 0);
    if (kc < RK / 32 && j >= 0 && k < a.rank) bv[kc] = *reinterpret_cast<const uint4*>(a.b + (size_t)j * a.rank + k);
  }
  // A^T of the tile's columns, zero past the rank and past the source columns: 8 columns of one rank row per
  // 16-byte load
  for (int e = tid; e < RK * (kMergeCols / 8); e += 256) {
    const int kr = e / (kMergeCols / 8), c = 8 * (e % (kMergeCols / 8));
    uint4 v = make_uint4(0, 0, 0, 0);
    if (kr < a.rank && c0 + c < a.src_cols) v = *reinterpret_cast<const uint4*>(a.a + (size_t)kr * a.src_cols + c0 + c);
    const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int x = 0; x < 8; ++x) at[c + x][kr] = (bf16_t)(vv[x >> 1] >> (16 * (x & 1)));
  }
  __syncthreads();
  float(*dw)[68] = dws[wave];
#pragma unroll
  for (int cb = 0; cb < kMergeCols / 64; ++cb) {
    if (cb >= nblk) break;
    f32x4 acc[4];
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) acc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      if (kc < RK / 32) {
        const int k = 32 * kc + 8 * (lane >> 4);
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
          const uint4 av = *reinterpret_cast<const uint4*>(&at[64 * cb + 16 * jb + (lane & 15)][k]);
          acc[jb] = mfma16(as_bf16x8(bv[kc]), as_bf16x8(av), acc[jb]);
        }
      }
    }
    // acc[jb][r]: update of row 16 wave + 4 (lane / 16) + r, column 64 cb + 16 jb + lane % 16
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
#pragma unroll
      for (int r = 0; r < 4; ++r) dw[4 * (lane >> 4) + r][16 * jb + (lane & 15)] = acc[jb][r];
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the wave's own staging rows are written
    // add the scaled update to the original weights, round to bf16, write in frag layout
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (!cin[t]) continue;
      const int e = lane + 64 * t, rr = e / 8, cc = 8 * (e % 8), col = c0 + 64 * cb + cc;
      float w[8];
      unpack8(w0v[cb][t], w);
      if (csrc[t] >= 0 && col < a.src_cols) {
#pragma unroll
        for (int x = 0; x < 8; ++x) w[x] += a.scale * dw[rr][cc + x];
      }
      *reinterpret_cast<uint4*>(a.dst + frag_index(crow[t], col, a.K)) =
          make_uint4(pack2bf(w[0], w[1]), pack2bf(w[2], w[3]), pack2bf(w[4], w[5]), pack2bf(w[6], w[7]));
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // this block's staging reads are done before the next block's writes
  }
}

// One workgroup per tile of each item, the items' tiles one after the other (row blocks fastest).
__global__ __launch_bounds__(256) void lora_merge_kernel(MergeBatch b) {
  int i = 0;
  while (i + 1 < b.n && (int)blockIdx.x >= b.wg0[i + 1]) ++i;
  const MergeArgs& a = b.item[i];
  const int local = (int)blockIdx.x - b.wg0[i], nrb = (merge_rows(a) + 63) / 64;
  merge_tile(a, local % nrb, local / nrb);
}

static bool merge_ok(const MergeArgs& a) {
  return a.K % 64 == 0 && a.rank >= 8 && a.rank <= 64 && a.rank % 8 == 0 && a.src_ld % 8 == 0 && a.src_cols % 8 == 0 &&
         (a.mode != kPackGateUp || (a.part >= 0 && a.part <= 1 && a.rows % 64 == 0));
}

hipError_t launch_lora_merge_batch(MergeBatch b, hipStream_t s) {
  if (b.n < 1 || b.n > kMergeBatchMax) return hipErrorInvalidValue;
  int wg = 0;
  for (int i = 0; i < b.n; ++i) {
    if (b.item[i].rows < 0 || !merge_ok(b.item[i])) return hipErrorInvalidValue;
    b.wg0[i] = wg;
    wg += (merge_rows(b.item[i]) + 63) / 64 * ((b.item[i].K + kMergeCols - 1) / kMergeCols);
  }
  b.wg0[b.n] = wg;
  if (wg == 0) return hipSuccess;
  hipLaunchKernelGGL(lora_merge_kernel, dim3(wg), dim3(256), 0, s, b);
  return hipGetLastError();
}

hipError_t launch_lora_merge(const MergeArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  MergeBatch b{};
  b.item[0] = a;
  b.n = 1;
  return launch_lora_merge_batch(b, s);
}

// One wave per row: 16-byte chunks of 8 consecutive K elements (contiguous in
// frag layout), lane l taking chunks l, l + 64, ..., then a butterfly sum.
__global__ __launch_bounds__(256) void value_head_kernel(const bf16_t* __restrict__ u, int R, int d,
                                                         const bf16_t* __restrict__ head, float* __restrict__ values) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= R) return;
  float acc = 0.f;
  for (int c = lane; c < d / 8; c += 64) {
    float uf[8], hf[8];
    unpack8(*reinterpret_cast<const uint4*>(u + frag_index(r, 8 * c, d)), uf);
    unpack8(*reinterpret_cast<const uint4*>(head + 8 * c), hf);
#pragma unroll
    for (int x = 0; x < 8; ++x) acc += uf[x] * hf[x];
  }
  acc = wave_sum(acc);
  if (lane == 0) values[r] = acc;
}

hipError_t launch_value_head(const bf16_t* u, int R, int d, const bf16_t* head, float* values, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(value_head_kernel, dim3((R + 3) / 4), dim3(256), 0, s, u, R, d, head, values);
  return hipGetLastError();
}

hipError_t launch_pack_frag(const PackArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.K % 32 != 0 || a.src_cols > a.K || !a.dst || !a.src || (a.mode == kPackGateUp && !a.src2))
    return hipErrorInvalidValue;
  const size_t n = (size_t)a.rows * (a.K / 8);
  hipLaunchKernelGGL(pack_frag_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bf16_to_f32(float* dst, const bf16_t* src, int n, hipStream_t s) {
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, src, n);
  return hipGetLastError();
}

hipError_t launch_extract_actions(const int32_t* tokens, int n, int n_dims, int action_begin, int bins,
                                  const float* lo, const float* hi, float* actions, hipStream_t s) {
  const int n_elems = n * n_dims;
  if (n_elems <= 0) return hipSuccess;
  hipLaunchKernelGGL(extract_actions_kernel, dim3((n_elems + 255) / 256), dim3(256), 0, s, tokens, n_elems, n_dims,
                     action_begin, bins, lo, hi, actions);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const float* x, const bf16_t* o, const int32_t* rows, int R, int d, float* xc,
                              bf16_t* oc, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (d % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(R), dim3(256), 0, s, x, o, rows, d, xc, oc);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (bytes % 16 != 0) return hipErrorInvalidValue;
  const size_t n16 = bytes / 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<uint4*>(dst), n16);
  return hipGetLastError();
}

}  // namespace vla
