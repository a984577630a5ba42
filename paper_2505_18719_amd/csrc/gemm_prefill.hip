// Prefill GEMM on gfx950 MFMA: C = A * W^T, A [M, K] bf16, W [N, K] bf16,
// fp32 accumulation, with fused epilogues (residual add, SwiGLU, RoPE + paged
// KV append).
//
// Tiling: a 256-thread workgroup (4 wave64s, one per SIMD) owns a 256 x 256
// output tile; each wave owns 128 x 128 of it as 4 x 4 blocks of
// v_mfma_f32_32x32x16_bf16 (256 fp32 accumulators per lane, held in AGPRs),
// which halves the LDS operand traffic per MFMA compared with 128 x 64 wave
// tiles.  K advances in steps of 32 through a ring of four 32 KB LDS stages
// filled by direct global -> LDS loads (global_load_lds_dwordx4, no VGPR round
// trip) issued three steps ahead, one copy instruction between MFMAs, so the
// copies neither stall the MFMA issue in a burst nor have to land within one
// step.  16-byte chunks are XOR-swizzled by row so that the MFMA operand
// reads (ds_read_b128, 32 rows x one chunk column) spread over the LDS banks.  Workgroup ids are
// remapped so that the tiles one XCD runs are contiguous in a grouped (8
// tile-rows) order, which keeps A panels and W panels resident in that XCD's L2.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int NT = 256;        // 4 waves, 2 x 2, each owning 128 x 128 of the tile
constexpr int CH = BK / 8;     // 16-byte chunks per tile row (64-byte rows)
constexpr int NSTAGE = 4;      // LDS ring of K steps (4 x 32 KB)
constexpr int AHEAD = 3;       // K steps in flight ahead of the one being consumed
constexpr int GROUP_M = 8;

typedef __attribute__((address_space(3))) void lds_ptr_t;
typedef __attribute__((address_space(1))) const void gbl_ptr_t;

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
// A 32-row operand read (one chunk column of 64-byte rows) then hits distinct
// bank groups for every 8 consecutive rows and for every 16 consecutive rows,
// i.e. it is conflict free whether the LDS serves 8 or 16 lanes per cycle.
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane i of the wave writes bytes [16 i, 16 i + 16) after the wave-uniform LDS
// address in M0.  Issued through inline assembly so that the compiler does
// not treat the copy as an LDS store: it would otherwise wait for every copy
// in flight (vmcnt(0)) before any later LDS read, serialising the copies that
// run ahead; the kernel instead waits explicitly for the stage it consumes.
__device__ __forceinline__ void g2lds16(const bf16_t* g, uint4* lds_wave_base) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)((lds_ptr_t*)lds_wave_base));
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(m0), "v"(g) : "memory", "m0");
}

// Each wave copies 4 blocks of 16 rows x 64 bytes of the A tile and of the W
// tile per K step.  Lane i of a block covers row 16b + i/4 and stores physical
// chunk i%4, which holds logical K chunk (i%4) ^ swz(row).
struct Loader {
  const bf16_t* a;
  const bf16_t* w;
  int aoff[4], woff[4];  // element offsets of this lane's rows (rows clamped to M-1 / N-1)
};

__device__ __forceinline__ void issue_tile(const Loader& ld, int k0, uint4* sa, uint4* sw, int wave) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int blk = wave * 4 + j;
    g2lds16(ld.a + ld.aoff[j] + k0, sa + blk * 64);
    g2lds16(ld.w + ld.woff[j] + k0, sw + blk * 64);
  }
}

__device__ __forceinline__ void load_frags(const uint4* sa, const uint4* sw, int ks, int wm, int wn, int lane,
                                           bf16x8 (&af)[4], bf16x8 (&bw)[4]) {
  const int l31 = lane & 31, c = 2 * ks + (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wm * 128 + i * 32 + l31;
    af[i] = as_bf16x8(sa[row * CH + (c ^ swz(row))]);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = wn * 128 + j * 32 + l31;
    bw[j] = as_bf16x8(sw[row * CH + (c ^ swz(row))]);
  }
}

__device__ __forceinline__ void mfma_rows(const bf16x8 (&af)[4], const bf16x8 (&bw)[4], f32x16 (&acc)[4][4],
                                          int i0, int i1) {
#pragma unroll
  for (int i = i0; i < i1; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(af[i], bw[j], acc[i][j]);
}

// s_waitcnt with vmcnt <= n (n < 64) and the other counters unconstrained.
#define WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) >> 4) << 14) | (0xF << 8) | (0x7 << 4) | ((n) & 15))

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs a, int tiles_m, int tiles_n) {
  __shared__ uint4 lds[NSTAGE][2][BM * CH];  // [stage][A / W][256 rows x 4 chunks]

  int tm, tn;
  map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  Loader ld;
  ld.a = a.A;
  ld.w = a.W;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = (wave * 4 + j) * 16 + (lane >> 2);
    const int chunk = (lane & 3) ^ swz(row);
    ld.aoff[j] = min(m0 + row, M - 1) * a.lda + chunk * 8;
    ld.woff[j] = min(n0 + row, N - 1) * K + chunk * 8;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Pipeline over K steps of 32 (two MFMA k-steps of 16).  Copies run AHEAD
  // steps ahead through the 4-stage ring, one copy instruction between MFMAs;
  // a step only waits for its own stage (the later copies stay in flight).
  // The barrier that hands the next stage over sits inside the second k-step:
  // the first operand fragments of the next stage are read while its last 8
  // MFMAs run.  Each wave issues 8 copies per step.
  const int nk = K / BK;
  bf16x8 fa[2][4], fb[2][4];
#pragma unroll
  for (int st = 0; st < AHEAD; ++st) issue_tile(ld, min(st, nk - 1) * BK, lds[st][0], lds[st][1], wave);
  WAIT_VMCNT(8 * (AHEAD - 1));
  __syncthreads();
  load_frags(lds[0][0], lds[0][1], 0, wm, wn, lane, fa[0], fb[0]);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & (NSTAGE - 1);
    const int nxt = (kt + 1) & (NSTAGE - 1);
    const int fill = (kt + AHEAD) & (NSTAGE - 1);
    // the stage being filled was read in step kt - 1, before the last barrier;
    // past the end the last step is re-copied, keeping the count per step fixed
    issue_tile(ld, min(kt + AHEAD, nk - 1) * BK, lds[fill][0], lds[fill][1], wave);
    load_frags(lds[cur][0], lds[cur][1], 1, wm, wn, lane, fa[1], fb[1]);
    mfma_rows(fa[0], fb[0], acc, 0, 4);
    mfma_rows(fa[1], fb[1], acc, 0, 2);
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 24, 0);
    WAIT_VMCNT(8 * (AHEAD - 1));   // this wave's copies of step kt+1 have landed
    __syncthreads();               // ... and everyone's
    load_frags(lds[nxt][0], lds[nxt][1], 0, wm, wn, lane, fa[0], fb[0]);
    mfma_rows(fa[1], fb[1], acc, 2, 4);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // ---------------------------------------------------------------- epilogue
  // The LDS stages are free after the last barrier; each wave stages its
  // 128 x 128 accumulator tile through its own 32 KB of them, 64 columns at a
  // time, and then writes the epilogue's outputs with contiguous stores.
  // acc[i][j][r] holds row i*32 + 8*(r/4) + 4*lhi + r%4 and column j*32 + l31
  // of the wave tile; in LDS the float4 chunk q of row rl sits at q ^ (rl%16).
  float* st = reinterpret_cast<float*>(&lds[0][0][0]) + wave * (128 * 64);
  const int l31 = lane & 31, lhi = lane >> 5;
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
  if (a.K % BK != 0 || a.N % 64 != 0 || a.lda % 8 != 0) return hipErrorInvalidValue;
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
