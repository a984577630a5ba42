// Prefill GEMM on gfx950 MFMA: C = A * W^T, A [M, K] bf16, W [N, K] bf16,
// fp32 accumulation, with fused epilogues (residual add, SwiGLU, RoPE + paged
// KV append).
//
// Tiling: a 256-thread workgroup (4 wave64s, one per SIMD) owns a 256 x 256
// output tile; each wave owns 128 x 128 of it as 4 x 4 blocks of
// v_mfma_f32_32x32x16_bf16 (256 fp32 accumulators per lane, held in AGPRs),
// which halves the LDS operand traffic per MFMA compared with 128 x 64 wave
// tiles.
//
// The kernel is bound by how fast the A and W tiles reach LDS (128 flops per
// delivered byte at this tile size), and a copy's round trip is long when its
// lines miss L2, so the copies run four K steps of 32 ahead through a ring of
// five 32 KB LDS stages (all 160 KB of LDS).  Both operands are in frag layout
// (see frag_index), so a K step of either tile is sixteen 1 KB blocks and
// every copy is one block moved whole by buffer_load ... lds (no VGPR round
// trip, one contiguous 1 KB read per wave instruction).  An MFMA operand read
// then takes 32 rows of a block pair as contiguous 256-byte runs, which is
// free of LDS bank conflicts without any swizzle.  Copies, operand reads and
// MFMAs are interleaved one memory instruction per MFMA in a pinned order.
// Workgroup ids are remapped so that the tiles one XCD runs are contiguous in
// a grouped (8 tile-rows) order, which keeps A panels and W panels resident
// in that XCD's L2.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int NT = 256;        // 4 waves, 2 x 2, each owning 128 x 128 of the tile
constexpr int NSTAGE = 5;      // LDS ring of K steps: A 16 KB + W 16 KB each
constexpr int AHEAD = 4;       // K steps whose copies are in flight ahead of the one consumed
constexpr int STAGE_U4 = 2 * 16 * 64;  // uint4 per stage: 2 operands x 16 blocks x 64 lanes
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

typedef __attribute__((address_space(3))) void lds_ptr_t;

// s_waitcnt with vmcnt <= n (n < 64) and the other counters unconstrained.
#define WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) >> 4) << 14) | (0xF << 8) | (0x7 << 4) | ((n) & 15))

// 16 bytes per lane from a buffer straight into LDS (buffer_load_dwordx4 ... lds):
// lane i writes bytes [16 i, 16 i + 16) after the wave-uniform LDS byte address
// m0.  Issued through inline assembly so that the compiler does not treat it
// as an LDS store (it would wait for every copy in flight before any later LDS
// read); the kernel waits for the copies it consumes itself.
__device__ __forceinline__ void dma16(uint32_t m0, uint32_t voff, __amdgpu_buffer_rsrc_t rsrc, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory");
}

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs a, int tiles_m, int tiles_n) {
  // [stage][A 16 blocks | W 16 blocks][64 lanes]: block b of an operand is its
  // 16-row block b of the tile over the stage's 32 K
  __shared__ uint4 lds[NSTAGE][STAGE_U4];

  int tm, tn;
  map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int KB = frag_kb(K);  // blocks per 16-row block (frag layout)
  const int last_rb_a = (M + 15) / 16 - 1, last_rb_w = N / 16 - 1;

  // Copies: wave w moves blocks 8 w .. 8 w + 7 of the step's 32 (A blocks
  // 0-15, W blocks 16-31).  Row blocks past the matrix are clamped to its last
  // one (their rows only feed outputs that are not stored).
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  // waves 0, 1 copy A blocks 0-15, waves 2, 3 W blocks 0-15 (wave-uniform choice, no branch)
  const bool copies_a = wave < 2;
  const __amdgpu_buffer_rsrc_t rsC = copies_a ? rsA : rsW;
  const int rb0 = copies_a ? (m0 >> 4) : (n0 >> 4), rb_last = copies_a ? last_rb_a : last_rb_w;
  const uint32_t voff = lane * 16;
  const uint32_t lds_base = (uint32_t)(uintptr_t)((lds_ptr_t*)&lds[0][0]);
  auto copy = [&](int j, int st, int ks) {
    const int b = wave * 8 + j;  // A block b, or W block b - 16
    dma16(lds_base + (st * STAGE_U4 + b * 64) * 16, voff, rsC, (min(rb0 + (b & 15), rb_last) * KB + ks) * 1024);
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Operand fragments of MFMA k-step q (0, 1) for lane (l31, lhi): row
  // 128 wm + 32 i + l31 of A (128 wn + ... of W) is row l31 % 16 of the
  // operand's block 8 wm + 2 i + l31 / 16, and K 16 q + 8 lhi is its column
  // group 2 q + lhi: the lane's 16 bytes sit at block lane (l31 % 16) + 16 (2 q + lhi).
  const int l31 = lane & 31, lhi = lane >> 5;
  const int fa = (wm * 8 + (l31 >> 4)) * 64 + (l31 & 15) + 16 * lhi;
  const int fw = 16 * 64 + (wn * 8 + (l31 >> 4)) * 64 + (l31 & 15) + 16 * lhi;
  const uint4* ring = &lds[0][0];
  bf16x8 fr[2][2][4];  // [k-step][A / W][block]
  auto read = [&](int ord, int r, int st, int q) {
    const int o = kReadO[ord][r], i = kReadB[ord][r];
    fr[q][o][i] = as_bf16x8(ring[st * STAGE_U4 + (o ? fw : fa) + i * 128 + 32 * q]);
  };
  auto mfma = [&](int ord, int t, int q) {
    const int i = kMfmaI[ord][t], j = kMfmaJ[ord][t];
    acc[i][j] = mfma32(fr[q][0][i], fr[q][1][j], acc[i][j]);
  };

  // Pipeline over K steps of 32 (two MFMA k-steps of 16).  One step of a wave
  // is 32 MFMAs with one memory instruction after 24 of them:
  //   k-step 0: MFMAs 0-7 + the 8 operand reads of k-step 1 (row-major order),
  //             MFMAs 8-15 + the 8 copies of step kt+AHEAD
  //   k-step 1: MFMAs 0-7 (row blocks 0, 1), wait for this wave's copies of
  //             step kt+1, barrier, MFMAs 8-15 + the 8 operand reads of
  //             k-step 0 of step kt+1
  // The order is pinned (the scheduler would otherwise hoist the barrier and
  // its LDS wait above the MFMAs that are meant to hide them).  The stage
  // filled in step kt was last read in step kt-1, before that step's barrier.
  // Loads complete in order: with the copies of AHEAD-1 later steps allowed
  // to stay in flight, the wait covers exactly the copies of step kt+1.
  const int nk = K / BK;
#pragma unroll
  for (int st = 0; st < AHEAD; ++st)
#pragma unroll
    for (int j = 0; j < 8; ++j) copy(j, st, min(st, nk - 1));
  WAIT_VMCNT(8 * (AHEAD - 1));
  __syncthreads();
  PIN();
#pragma unroll
  for (int r = 0; r < 8; ++r) {  // same order as in the loop, so the loop's waits hold on entry
    read(0, r, 0, 0);
    PIN();
  }
  int cur = 0, fill = AHEAD;  // ring stages of steps kt and kt + AHEAD
  for (int kt = 0; kt < nk; ++kt) {
    const int nxt = cur + 1 == NSTAGE ? 0 : cur + 1;
    const int kfill = min(kt + AHEAD, nk - 1);  // past the end the last step is re-copied
    PIN();
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      mfma(0, t, 0);
      read(1, t, cur, 1);
      PIN();
    }
#pragma unroll
    for (int t = 8; t < 16; ++t) {
      mfma(0, t, 0);
      copy(t - 8, fill, kfill);
      PIN();
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      mfma(1, t, 1);
      PIN();
    }
    WAIT_VMCNT(8 * (AHEAD - 1));   // this wave's copies of step kt+1 have landed
    __syncthreads();               // ... and everyone's
    PIN();
#pragma unroll
    for (int t = 8; t < 16; ++t) {
      mfma(1, t, 1);
      read(0, t - 8, nxt, 0);
      PIN();
    }
    cur = nxt;
    fill = fill + 1 == NSTAGE ? 0 : fill + 1;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // ---------------------------------------------------------------- epilogue
  // The LDS stages are free after the last barrier; each wave stages its
  // 128 x 128 accumulator tile through its own 32 KB of them, 64 columns at a
  // time, and then writes the epilogue's outputs with contiguous stores.
  // acc[i][j][r] holds row i*32 + 8*(r/4) + 4*lhi + r%4 and column j*32 + l31
  // of the wave tile; in LDS the float4 chunk q of row rl sits at q ^ (rl%16).
  float* st = reinterpret_cast<float*>(&lds[0][0]) + wave * (128 * 64);
  // (l31, lhi as in the main loop)
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
          *reinterpret_cast<uint2*>(a.H + frag_index(row, c0 / 2 + 4 * q, a.ldh)) =  // frag layout, K = ldh
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
  // frag-layout operands, 32-bit byte offsets into them
  if (a.K % BK != 0 || a.N % 64 != 0 || (long long)frag_elems(a.M, a.K) * 2 >= (1ll << 31) ||
      (long long)frag_elems(a.N, a.K) * 2 >= (1ll << 31))
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
