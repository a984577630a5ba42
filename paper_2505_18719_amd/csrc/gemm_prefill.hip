// Prefill GEMM on gfx950 MFMA: C = A * W^T, A [M, K] bf16, W [N, K] bf16,
// fp32 accumulation, with fused epilogues (residual add, SwiGLU, RoPE + paged
// KV append).
//
// Tiling: a 512-thread workgroup (8 wave64s, 2 per SIMD) owns a 256 x 256
// output tile; each wave owns 128 x 64 of it as 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16.  K advances in steps of 64 through a two-stage
// LDS ring (2 x 64 KB) whose 16-byte chunks are XOR-swizzled by row so that
// the MFMA operand reads (ds_read_b128, 32 rows x one chunk column) are
// bank-conflict free.  Workgroup ids are remapped so that the tiles one XCD
// runs are contiguous in a grouped (8 tile-rows) order, which keeps A panels
// and W panels resident in that XCD's L2.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 512;
constexpr int CH = BK / 8;  // 16-byte chunks per tile row
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

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs a, int tiles_m, int tiles_n) {
  __shared__ uint4 lds[2][2][BM * CH];

  int tm, tn;
  map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;

  // global -> LDS assignment: 4 passes of 64 rows, 8 threads per 128-byte row
  const int lrow = tid >> 3, lchunk = tid & 7;
  const bf16_t* ag[4];
  const bf16_t* wg[4];
  int so[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int r = p * 64 + lrow;
    ag[p] = a.A + (size_t)min(m0 + r, M - 1) * a.lda + lchunk * 8;
    wg[p] = a.W + (size_t)min(n0 + r, N - 1) * K + lchunk * 8;
    so[p] = r * CH + (lchunk ^ (r & 7));
  }

  uint4 ra[4], rb[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    ra[p] = *reinterpret_cast<const uint4*>(ag[p]);
    rb[p] = *reinterpret_cast<const uint4*>(wg[p]);
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    lds[0][0][so[p]] = ra[p];
    lds[0][1][so[p]] = rb[p];
  }
  __syncthreads();

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = K / BK;
  const int l31 = lane & 31, lhi = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int koff = (kt + 1) * BK;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        ra[p] = *reinterpret_cast<const uint4*>(ag[p] + koff);
        rb[p] = *reinterpret_cast<const uint4*>(wg[p] + koff);
      }
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = 2 * ks + lhi;
      bf16x8 af[4], bw[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + i * 32 + l31;
        af[i] = as_bf16x8(lds[cur][0][row * CH + (c ^ (row & 7))]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wn * 64 + j * 32 + l31;
        bw[j] = as_bf16x8(lds[cur][1][row * CH + (c ^ (row & 7))]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(af[i], bw[j], acc[i][j]);
    }
    if (more) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        lds[cur ^ 1][0][so[p]] = ra[p];
        lds[cur ^ 1][1][so[p]] = rb[p];
      }
    }
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][r] holds row wm*128 + i*32 + 8*(r/4) + 4*lhi + r%4 and column
  // wn*64 + j*32 + l31 of the tile.
  const int c0 = n0 + wn * 64;
  if (c0 >= N) return;
  if constexpr (EPI == kEpiStoreF32 || EPI == kEpiResidual) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = c0 + j * 32 + l31;
          if (col >= N) continue;
          float* p = a.C + (size_t)row * a.ldc + col;
          if constexpr (EPI == kEpiResidual) *p += acc[i][j][r];
          else *p = acc[i][j][r];
        }
      }
  } else if constexpr (EPI == kEpiSwiGlu) {
    // columns [c0, c0+32) are gate rows, [c0+32, c0+64) the matching up rows
    const int jj = c0 / 2 + l31;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        if (row >= M) continue;
        const float g = acc[i][0][r], u = acc[i][1][r];
        a.H[(size_t)row * a.ldh + jj] = f2bf(g / (1.f + expf(-g)) * u);
      }
  } else {  // kEpiQkvRope
    const int d = a.d_model, hd = a.head_dim, H = a.n_heads, half = hd / 2;
    const int region = c0 / d;
    const int cc0 = c0 - region * d;
    const int head = cc0 / hd;
    const int blk = (cc0 % hd) / 64;
    // q and k rows were permuted per head so that columns c and c+32 of this
    // 64-column block are the rotary pair (32*blk + c, half + 32*blk + c).
    const int ai = 32 * blk + l31;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        if (row >= M) continue;
        const int pos = a.meta.row_pos[row];
        const float x1 = acc[i][0][r], x2 = acc[i][1][r];
        if (region == 0) {
          const float2 cs = a.rope[pos * half + ai];
          bf16_t* qr = a.q + (size_t)row * a.ldq + head * hd;
          qr[ai] = f2bf(x1 * cs.x - x2 * cs.y);
          qr[half + ai] = f2bf(x1 * cs.y + x2 * cs.x);
        } else {
          const int env = a.meta.row_env[row];
          const int page = a.meta.page_table[env * a.meta.max_pages + pos / kPage];
          const int slot = pos % kPage;
          if (region == 1) {
            const float2 cs = a.rope[pos * half + ai];
            bf16_t* kr = a.kv.k + (((size_t)page * H + head) * kPage + slot) * hd;
            kr[ai] = f2bf(x1 * cs.x - x2 * cs.y);
            kr[half + ai] = f2bf(x1 * cs.y + x2 * cs.x);
          } else {
            const int i1 = cc0 % hd + l31;
            bf16_t* vb = a.kv.v + ((size_t)page * H + head) * hd * kPage + slot;
            vb[(size_t)i1 * kPage] = f2bf(x1);
            vb[(size_t)(i1 + 32) * kPage] = f2bf(x2);
          }
        }
      }
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
