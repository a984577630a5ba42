// Decode-time skinny GEMM on gfx950: C = A * W^T for M <= 128 rows (one per
// environment), A [M, K] bf16, W [N, K] bf16, fp32 accumulation.
//
// Decode streams every weight once per step, so the kernel is shaped for HBM
// bandwidth: a 256-thread workgroup owns 64 output columns (four
// v_mfma_f32_16x16x32_bf16 column blocks) and one K slice; its four waves
// take interleaved 32-wide k-steps of that slice, so together they read each
// weight row as one contiguous stream, and they combine their partial tiles
// through LDS at the end.  Each lane loads its weight fragment straight from
// global memory as 16-byte loads; several k-steps are in flight per wave.
// Each workgroup starts at a different point of its K range so that the
// workgroups running at the same time spread their activation reads over L2.  The activations (<= 128 x K bf16) are read through L2, where
// every workgroup of the GPU shares them; owning 64 columns amortises each
// activation fragment over four weight fragments.
//
// The K split is kept small (1-4 slices): with one slice the epilogue is
// applied in place (SwiGLU to bf16 h, or a plain fp32 store); with more, fp32
// partial sums go to a buffer that one consumer kernel reduces in a fixed
// order, so results are bitwise deterministic.
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int COLS = 64;      // output columns per workgroup
constexpr int NW = 4;         // waves per workgroup

template <int MB, int U, int EPI>
__global__ __launch_bounds__(64 * NW) void skinny_kernel(SkinnyArgs a, int kslice) {
  extern __shared__ float red[];  // [NW][MB*16][COLS]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * COLS;
  const int s = blockIdx.y;
  const int kb = s * kslice;
  const int ke = min(a.K, kb + kslice);
  const int r16 = lane & 15, g = lane >> 4;

  const bf16_t* wp[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) wp[nb] = a.W + (size_t)(n0 + nb * 16 + r16) * a.K + 8 * g;
  const bf16_t* ap[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) ap[mb] = a.A + (size_t)min(mb * 16 + r16, a.M - 1) * a.lda + 8 * g;

  f32x4 acc[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Wave w takes the k-steps kb + 32 * (NW * j + w), j < Tw, starting at a
  // workgroup-dependent rotation so that concurrently running workgroups read
  // different parts of the shared activations.  Batches of U k-steps are
  // double-buffered in registers: batch b+1 is in flight while the MFMAs of
  // batch b run.
  const int T = (ke - kb + 31) / 32;
  const int Tw = T > wave ? (T - wave + NW - 1) / NW : 0;
  const int rot = Tw > 0 ? (int)((blockIdx.x * 37u + blockIdx.y * 11u) % (unsigned)Tw) : 0;
  const int nbatch = Tw / U;
  uint4 wv[2][U][4], av[2][U][MB];
  auto kstep = [&](int j) {
    j += rot;
    j = j >= Tw ? j - Tw : j;
    return kb + 32 * (NW * j + wave);
  };
  auto load = [&](int b, uint4 (&w)[U][4], uint4 (&x)[U][MB]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kstep(b * U + u);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) w[u][nb] = *reinterpret_cast<const uint4*>(wp[nb] + k);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) x[u][mb] = *reinterpret_cast<const uint4*>(ap[mb] + k);
    }
  };
  auto math = [&](const uint4 (&w)[U][4], const uint4 (&x)[U][MB]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma16(as_bf16x8(x[u][mb]), as_bf16x8(w[u][nb]), acc[mb][nb]);
  };
  if (nbatch > 0) load(0, wv[0], av[0]);
  int b = 0;
  for (; b + 2 <= nbatch; b += 2) {
    load(b + 1, wv[1], av[1]);
    math(wv[0], av[0]);
    if (b + 2 < nbatch) load(b + 2, wv[0], av[0]);
    math(wv[1], av[1]);
  }
  if (b < nbatch) math(wv[0], av[0]);
  for (int j = nbatch * U; j < Tw; ++j) {
    const int k = kstep(j);
    uint4 w1[4], x1[MB];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) w1[nb] = *reinterpret_cast<const uint4*>(wp[nb] + k);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) x1[mb] = *reinterpret_cast<const uint4*>(ap[mb] + k);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma16(as_bf16x8(x1[mb]), as_bf16x8(w1[nb]), acc[mb][nb]);
  }

  // acc[mb][nb][r] is row mb*16 + 4g + r, column nb*16 + r16 of the tile
  constexpr int ROWS = MB * 16;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[(wave * ROWS + mb * 16 + 4 * g + r) * COLS + nb * 16 + r16] = acc[mb][nb][r];
  __syncthreads();

  if constexpr (EPI == kSkinnySwiGlu) {
    // columns [0, 32) of the tile are gate rows, [32, 64) the matching up rows
    for (int e = threadIdx.x; e < ROWS * 32; e += 64 * NW) {
      const int row = e / 32, c = e % 32;
      if (row >= a.M) break;
      float gs = 0.f, us = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        gs += red[(w * ROWS + row) * COLS + c];
        us += red[(w * ROWS + row) * COLS + c + 32];
      }
      a.h[(size_t)row * a.ldh + n0 / 2 + c] = f2bf(gs / (1.f + expf(-gs)) * us);
    }
  } else {
    float* out = a.part + (size_t)s * a.M * a.N + n0;
    for (int e = threadIdx.x; e < ROWS * COLS; e += 64 * NW) {
      const int row = e / COLS, c = e % COLS;
      if (row >= a.M) break;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += red[(w * ROWS + row) * COLS + c];
      out[(size_t)row * a.N + c] = v;
    }
  }
}

template <int MB, int U, int EPI>
hipError_t launch_one(const SkinnyArgs& a, int kslice, hipStream_t st) {
  const dim3 grid(a.N / COLS, a.splits), block(64 * NW);
  const size_t lds = (size_t)NW * MB * 16 * COLS * sizeof(float);
  static bool attr_set = false;  // dynamic LDS above 64 KB must be allowed once per kernel
  if (!attr_set && lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&skinny_kernel<MB, U, EPI>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((skinny_kernel<MB, U, EPI>), grid, block, lds, st, a, kslice);
  return hipGetLastError();
}

template <int MB, int U>
hipError_t launch_mb(const SkinnyArgs& a, int kslice, SkinnyEpilogue epi, hipStream_t st) {
  if (epi == kSkinnySwiGlu) return launch_one<MB, U, kSkinnySwiGlu>(a, kslice, st);
  return launch_one<MB, U, kSkinnyPartial>(a, kslice, st);
}

}  // namespace

int skinny_splits(int M, int N, int K, int max_splits) {
  (void)M;
  // enough workgroups for ~2 per CU without splitting K more than 4 ways
  const int blocks = N / COLS;
  int s = (512 + blocks - 1) / blocks;
  if (s > 4) s = 4;
  if (s > max_splits) s = max_splits;
  const int ksteps = K / 32;
  if (s > ksteps) s = ksteps;
  return s < 1 ? 1 : s;
}

hipError_t launch_skinny(const SkinnyArgs& a, hipStream_t st, SkinnyEpilogue epi) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.M > 128 || a.N % COLS != 0 || a.K % 32 != 0 || a.splits < 1 || a.lda % 8 != 0) return hipErrorInvalidValue;
  if (epi == kSkinnySwiGlu && a.splits != 1) return hipErrorInvalidValue;
  // K slice: a multiple of 32, splits * kslice >= K
  const int ksteps = a.K / 32;
  const int kslice = ((ksteps + a.splits - 1) / a.splits) * 32;
  const int mb = (a.M + 15) / 16;
  if (mb <= 1) return launch_mb<1, 4>(a, kslice, epi, st);
  if (mb <= 2) return launch_mb<2, 4>(a, kslice, epi, st);
  if (mb <= 4) return launch_mb<4, 2>(a, kslice, epi, st);
  return launch_mb<8, 1>(a, kslice, epi, st);
}

}  // namespace vla
