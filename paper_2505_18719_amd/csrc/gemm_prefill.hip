// Prefill GEMM on gfx950 MFMA: C = A * W^T, A [M, K] bf16, W [N, K] bf16,
// fp32 accumulation, with fused epilogues (residual add, SwiGLU, RoPE + paged
// KV append).
//
// Tiling: a 256-thread workgroup (4 wave64s, one per SIMD) owns a 256 x 256
// output tile; each wave owns 128 x 128 of it as 4 x 4 blocks of
// v_mfma_f32_32x32x16_bf16 (256 fp32 accumulators per lane, held in AGPRs),
// which halves the LDS operand traffic per MFMA compared with 128 x 64 wave
// tiles.  K advances in steps of 64 through two 64 KB LDS stages.
//
// The kernel is bound by how fast L2 delivers the A and W tiles to the CU
// (128 flops per delivered byte at this tile size): the operand tiles are
// brought in with plain 16-byte buffer loads into VGPRs, two K steps ahead,
// and written to LDS one step ahead, so about 1.5 steps of loads are in flight
// per CU; each wave load instruction reads 8 whole 128-byte rows.  Loads, LDS
// writes, operand reads and MFMAs are interleaved one memory instruction per
// MFMA in a pinned order.  16-byte chunks are XOR-swizzled by row so that the
// MFMA operand reads (ds_read_b128, 32 rows x one chunk column) and the LDS
// writes spread over the banks.  Workgroup ids are remapped so that the tiles
// one XCD runs are contiguous in a grouped (8 tile-rows) order, which keeps A
// panels and W panels resident in that XCD's L2.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;        // 4 waves, 2 x 2, each owning 128 x 128 of the tile
constexpr int CH = BK / 8;     // 16-byte chunks per tile row (128-byte rows)
constexpr int GROUP_M = 8;


__device__ __forceinline__ void map_tile(int pid, int G, int tiles_m, int tiles_n, int& tm, int& tn) {
  // XCD-aware remap: the hardware deals workgroups round-robin to 8 XCDs.
  const int per = G / 8;
  int L = pid;
  if (pid < per * 8) L = (pid & 7) * per + (pid >> 3);
  const int group = GROUP_M * tiles_n;
  const int g = L / group;
  const int first_m = g * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int r = L - g * group;
  tm = first_m + r % gm;
  tn = r / gm;
}

// Physical position of logical 16-byte chunk c of tile row r is c ^ swz(r).
// An operand read takes one chunk column of 16 consecutive rows per 16 lanes;
// two 128-byte rows share a 256-byte bank row, so the chunk index must take 8
// distinct values over the 8 rows of each parity: then the 16 reads hit 16
// distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// nothing may be scheduled across this point
#define PIN() __builtin_amdgcn_sched_barrier(0)

// Orders of the 16 MFMAs of one k-step over the 4 x 4 blocks of the wave
// tile (row block i, column block j) and of the 8 operand reads that feed them
// (o = 0 for A, 1 for W; block index).  Order 0 ("triangular") lets each MFMA
// wait only for fragments read well before it; order 1 is row-major, so that
// its first 8 MFMAs need only the first 6 reads (the k-step that straddles the
// barrier).
__device__ constexpr int kMfmaI[2][16] = {{0, 0, 1, 1, 0, 1, 2, 2, 2, 0, 1, 2, 3, 3, 3, 3},
                                          {0, 0, 0, 0, 1, 1, 1, 1, 2, 2, 2, 2, 3, 3, 3, 3}};
__device__ constexpr int kMfmaJ[2][16] = {{0, 1, 0, 1, 2, 2, 0, 1, 2, 3, 3, 3, 0, 1, 2, 3},
                                          {0, 1, 2, 3, 0, 1, 2, 3, 0, 1, 2, 3, 0, 1, 2, 3}};
__device__ constexpr int kReadO[2][8] = {{0, 1, 0, 1, 0, 1, 0, 1}, {0, 0, 1, 1, 1, 1, 0, 0}};
__device__ constexpr int kReadB[2][8] = {{0, 0, 1, 1, 2, 2, 3, 3}, {0, 1, 0, 1, 2, 3, 2, 3}};

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 as_uint4(u32x4_t v) { return make_uint4(v.x, v.y, v.z, v.w); }

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs a, int tiles_m, int tiles_n) {
  __shared__ uint4 lds[2][2][BM * CH];  // [stage][A / W][256 rows x 8 chunks]

  int tm, tn;
  map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Loads: per K step each thread brings 8 16-byte chunks of the A tile and 8
  // of the W tile into VGPRs and later writes them to LDS at physical chunk
  // c ^ swz(row).  A (row-major): chunk j is row 32 j + tid / 8, K chunk
  // tid % 8, so each wave instruction reads 8 whole 128-byte rows.  W (frag
  // layout, see frag_index): wave w's chunk j is lane l's 16 bytes of 1 KB
  // block (16-row block 2 j + w / 2, K block w % 2) of the step, i.e. row
  // 16 (2 j + w / 2) + l % 16, K chunk 4 (w % 2) + l / 16: each wave
  // instruction reads one contiguous 1 KB block.
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  uint32_t voffA[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
    voffA[j] = (uint32_t)((min(m0 + j * 32 + (tid >> 3), M - 1) * a.lda + (tid & 7) * 8) * 2);
  // W rows past N (whole 16-row blocks, N % 64 == 0) are clamped to the last block
  const int wv = tid >> 6, wl = tid & 63;
  const int KB = K / 32;
  uint32_t voffW[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
    voffW[j] = (uint32_t)((min((n0 >> 4) + 2 * j + (wv >> 1), N / 16 - 1) * KB + (wv & 1)) * 1024 + wl * 16);
  // uint4 index of this thread's chunk in the A tile (chunk j: + 256 j) and in the W tile (chunk j: + 256 j)
  const int widx = (tid >> 3) * CH + ((tid & 7) ^ ((tid >> 4) & 7));
  const int wrow = (wv >> 1) * 16 + (wl & 15);
  const int widx_w = wrow * CH + (((wv & 1) * 4 + (wl >> 4)) ^ swz(wrow));

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // fragment rows wm*128 + 32 i + l31 (A) and wn*128 + 32 i + l31 (W): all share swz = swz(l31)
  const int l31 = lane & 31;
  const int roff[2] = {(wm * 128 + l31) * CH, BM * CH + (wn * 128 + l31) * CH};
  const int rswz = swz(l31);
  uint4* ring = &lds[0][0][0];
  bf16x8 fr[2][2][4];
  uint4 rg[2][16];  // register stages: [parity][A chunks 0-7, W chunks 0-7]
  auto read = [&](int ord, int r, int st, int q) {
    const int o = kReadO[ord][r], i = kReadB[ord][r];
    const int c = (2 * q + (lane >> 5)) ^ rswz;
    fr[q & 1][o][i] = as_bf16x8(ring[st * (2 * BM * CH) + roff[o] + i * 32 * CH + c]);
  };
  auto mfma = [&](int ord, int t, int q) {
    const int i = kMfmaI[ord][t], j = kMfmaJ[ord][t];
    acc[i][j] = mfma32(fr[q & 1][0][i], fr[q & 1][1][j], acc[i][j]);
  };
  const int nk = K / BK;
  // load chunk c (0..15: A 0-7, W 8-15) of K step ks into register stage p
  auto gload = [&](int p, int c, int ks) {
    const int j = c & 7;
    if (c < 8)
      rg[p][c] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsA, voffA[j], ks * BK * 2, 0));
    else
      rg[p][c] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsW, voffW[j], ks * BK * 32, 0));
  };
  auto lwrite = [&](int p, int c, int st) {
    const int j = c & 7;
    if (c < 8)
      ring[st * (2 * BM * CH) + j * 256 + widx] = rg[p][c];
    else
      ring[st * (2 * BM * CH) + BM * CH + j * 256 + widx_w] = rg[p][c];
  };

  // Pipeline: step s's tiles are loaded into register stage s % 2 during step
  // s - 2, written to LDS stage s % 2 during the second half of step s - 1,
  // and consumed in step s.  One step of a wave is 64 MFMAs with one memory
  // instruction after each:
  //   k-step 0: + the 8 operand reads of k-step 1, + loads 0-7 of step kt+2
  //   k-step 1: + the 8 operand reads of k-step 2, + loads 8-15 of step kt+2
  //   k-step 2: + the 8 operand reads of k-step 3 (row-major order), + LDS writes 0-7 of step kt+1
  //   k-step 3: MFMAs 0-7 + LDS writes 8-15 of step kt+1, barrier,
  //             MFMAs 8-15 + the 8 operand reads of k-step 0 of step kt+1
  // The order is pinned.  LDS stage (kt+1) % 2 was last read in step kt-1,
  // before that step's barrier.
  auto step = [&](int kt, int P) {
    const int cur = P, nxt = P ^ 1;
    const int k2 = min(kt + 2, nk - 1);
    PIN();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        mfma(0, t, q);
        read(0, t, cur, q + 1);
        PIN();
      }
#pragma unroll
      for (int t = 8; t < 16; ++t) {
        mfma(0, t, q);
        gload(P, 8 * q + t - 8, k2);
        PIN();
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      mfma(0, t, 2);
      read(1, t, cur, 3);
      PIN();
    }
#pragma unroll
    for (int t = 8; t < 16; ++t) {
      mfma(0, t, 2);
      lwrite(nxt, t - 8, nxt);
      PIN();
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      mfma(1, t, 3);
      lwrite(nxt, t + 8, nxt);
      PIN();
    }
    __syncthreads();
    PIN();
#pragma unroll
    for (int t = 8; t < 16; ++t) {
      mfma(1, t, 3);
      read(0, t - 8, nxt, 0);
      PIN();
    }
  };

#pragma unroll
  for (int c = 0; c < 16; ++c) gload(0, c, 0);
#pragma unroll
  for (int c = 0; c < 16; ++c) gload(1, c, min(1, nk - 1));
#pragma unroll
  for (int c = 0; c < 16; ++c) lwrite(0, c, 0);
  __syncthreads();
  PIN();
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    read(0, r, 0, 0);
    PIN();
  }
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(kt, 0);
    step(kt + 1, 1);
  }
  if (kt < nk) step(kt, 0);
  __syncthreads();

  // ---------------------------------------------------------------- epilogue
  // The LDS stages are free after the last barrier; each wave stages its
  // 128 x 128 accumulator tile through its own 32 KB of them, 64 columns at a
  // time, and then writes the epilogue's outputs with contiguous stores.
  // acc[i][j][r] holds row i*32 + 8*(r/4) + 4*lhi + r%4 and column j*32 + l31
  // of the wave tile; in LDS the float4 chunk q of row rl sits at q ^ (rl%16).
  float* st = reinterpret_cast<float*>(&lds[0][0][0]) + wave * (128 * 64);
  const int lhi = lane >> 5;
  const int wrow0 = m0 + wm * 128;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c0 = n0 + wn * 128 + h * 64;   // first column of this 64-column group
    if (c0 >= N) break;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = i * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
          const int cl = jj * 32 + l31;
          st[rl * 64 + (((cl >> 2) ^ (rl & 15)) << 2) + (cl & 3)] = acc[i][2 * h + jj][r];
        }
    __builtin_amdgcn_s_waitcnt(0);
    if constexpr (EPI == kEpiStoreF32 || EPI == kEpiResidual) {
      const int q = lane & 15;
      for (int it = 0; it < 32; ++it) {
        const int rl = it * 4 + (lane >> 4);
        const int row = wrow0 + rl;
        const float4 v = *reinterpret_cast<const float4*>(st + rl * 64 + ((q ^ (rl & 15)) << 2));
        if (row < M) {
          float4* p = reinterpret_cast<float4*>(a.C + (size_t)row * a.ldc + c0 + 4 * q);
          if constexpr (EPI == kEpiResidual) {
            const float4 o = *p;
            *p = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
          } else {
            *p = v;
          }
        }
      }
    } else {
      // pair epilogues: chunk q (< 8) of the group pairs with chunk q + 8
      const int q = lane & 7;
      for (int it = 0; it < 16; ++it) {
        const int rl = it * 8 + (lane >> 3);
        const int row = wrow0 + rl;
        const float4 v1 = *reinterpret_cast<const float4*>(st + rl * 64 + ((q ^ (rl & 15)) << 2));
        const float4 v2 = *reinterpret_cast<const float4*>(st + rl * 64 + (((q + 8) ^ (rl & 15)) << 2));
        if (row >= M) continue;
        const float x1[4] = {v1.x, v1.y, v1.z, v1.w}, x2[4] = {v2.x, v2.y, v2.z, v2.w};
        if constexpr (EPI == kEpiSwiGlu) {
          // columns [c0, c0+32) are gate rows, [c0+32, c0+64) the matching up rows
          float o[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) o[t] = x1[t] / (1.f + expf(-x1[t])) * x2[t];
          *reinterpret_cast<uint2*>(a.H + (size_t)row * a.ldh + c0 / 2 + 4 * q) =
              make_uint2(pack2bf(o[0], o[1]), pack2bf(o[2], o[3]));
        } else {  // kEpiQkvRope
          const int d = a.d_model, hd = a.head_dim, H = a.n_heads, half = hd / 2;
          const int region = c0 / d;
          const int cc0 = c0 - region * d;
          const int head = cc0 / hd;
          const int blk = (cc0 % hd) / 64;
          const int pos = a.meta.row_pos[row];
          if (region < 2) {
            // q and k rows were permuted per head so that columns c and c+32 of
            // this 64-column group are the rotary pair (32*blk + c, half + 32*blk + c)
            const int ai = 32 * blk + 4 * q;
            float o1[4], o2[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const float2 cs = a.rope[pos * half + ai + t];
              o1[t] = x1[t] * cs.x - x2[t] * cs.y;
              o2[t] = x1[t] * cs.y + x2[t] * cs.x;
            }
            bf16_t* dst;
            if (region == 0) {
              dst = a.q + (size_t)row * a.ldq + head * hd;
            } else {
              const int env = a.meta.row_env[row];
              const int page = a.meta.page_table[env * a.meta.max_pages + pos / kPage];
              dst = a.kv.k + (((size_t)page * H + head) * kPage + pos % kPage) * hd;
            }
            *reinterpret_cast<uint2*>(dst + ai) = make_uint2(pack2bf(o1[0], o1[1]), pack2bf(o1[2], o1[3]));
            *reinterpret_cast<uint2*>(dst + half + ai) = make_uint2(pack2bf(o2[0], o2[1]), pack2bf(o2[2], o2[3]));
          } else {
            const int env = a.meta.row_env[row];
            const int page = a.meta.page_table[env * a.meta.max_pages + pos / kPage];
            bf16_t* vb = a.kv.v + ((size_t)page * H + head) * hd * kPage + pos % kPage;
            const int i1 = cc0 % hd + 4 * q;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              vb[(size_t)(i1 + t) * kPage] = f2bf(x1[t]);
              vb[(size_t)(i1 + t + 32) * kPage] = f2bf(x2[t]);
            }
          }
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, GemmEpilogue epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.K % BK != 0 || a.N % 64 != 0 || a.lda % 8 != 0 || (long long)a.N * a.K * 2 >= (1ll << 31))
    return hipErrorInvalidValue;
  const int tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  const dim3 grid(tm * tn), block(NT);
  switch (epi) {
    case kEpiStoreF32: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiStoreF32>, grid, block, 0, s, a, tm, tn); break;
    case kEpiResidual: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiResidual>, grid, block, 0, s, a, tm, tn); break;
    case kEpiSwiGlu: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiSwiGlu>, grid, block, 0, s, a, tm, tn); break;
    case kEpiQkvRope: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiQkvRope>, grid, block, 0, s, a, tm, tn); break;
  }
  return hipGetLastError();
}

}  // namespace vla
