// Decode-time skinny GEMM on gfx950: part[s, m, n] = sum over K-slice s of
// A[m, k] * W[n, k] for M <= 128 (one row per environment).
//
// Decode is bound by streaming the weights from HBM once per step, so the
// kernel is shaped for that: every wave owns 16 output columns (one
// v_mfma_f32_16x16x32_bf16 column block) and one K slice; each lane loads its
// weight fragment straight from global memory as 16-byte loads (a wave reads
// 16 rows x 64 contiguous bytes per MFMA k-step), four k-steps are in flight
// per iteration, and the small activation matrix A (<= 128 x K bf16) is read
// through L2 where every wave of the GPU shares it.  K is split so that the
// grid holds about 8 waves per CU; the fp32 partial sums are combined,
// deterministically, by the consumer kernel (residual add + RMSNorm, SwiGLU,
// RoPE + KV append, or the logits reduction).
#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int WAVES = 4;      // waves per workgroup (4 column blocks)
constexpr int KU = 4;         // k-steps of 32 per iteration

template <int MB>
__global__ __launch_bounds__(64 * WAVES) void skinny_kernel(SkinnyArgs a, int kslice) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nblk = blockIdx.x * WAVES + wave;       // 16-column block
  const int n0 = nblk * 16;
  if (n0 >= a.N) return;
  const int s = blockIdx.y;
  const int kb = s * kslice;
  const int ke = min(a.K, kb + kslice);
  const int r16 = lane & 15, g = lane >> 4;

  const bf16_t* wp = a.W + (size_t)(n0 + r16) * a.K + 8 * g;
  const bf16_t* ap[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) ap[mb] = a.A + (size_t)min(mb * 16 + r16, a.M - 1) * a.lda + 8 * g;

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  int k = kb;
  for (; k + 32 * KU <= ke; k += 32 * KU) {
    uint4 wv[KU];
#pragma unroll
    for (int u = 0; u < KU; ++u) wv[u] = load_stream16(wp + k + 32 * u);
    uint4 av[KU][MB];
#pragma unroll
    for (int u = 0; u < KU; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) av[u][mb] = *reinterpret_cast<const uint4*>(ap[mb] + k + 32 * u);
#pragma unroll
    for (int u = 0; u < KU; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16(as_bf16x8(av[u][mb]), as_bf16x8(wv[u]), acc[mb]);
  }
  for (; k < ke; k += 32) {
    const uint4 wv = load_stream16(wp + k);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      acc[mb] = mfma16(as_bf16x8(*reinterpret_cast<const uint4*>(ap[mb] + k)), as_bf16x8(wv), acc[mb]);
  }

  // acc[mb][r] is row mb*16 + 4*g + r, column n0 + r16
  float* out = a.part + (size_t)s * a.M * a.N + n0 + r16;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = mb * 16 + 4 * g + r;
      if (row < a.M) out[(size_t)row * a.N] = acc[mb][r];
    }
}

}  // namespace

int skinny_splits(int M, int N, int K, int max_splits) {
  (void)M;
  const int blocks = (N / 16 + WAVES - 1) / WAVES;     // workgroups per split
  const int target = 256 * 8 / WAVES;                  // ~8 waves per CU
  int s = (target + blocks - 1) / blocks;
  const int ksteps = K / 32;
  s = s < 1 ? 1 : s;
  s = s > max_splits ? max_splits : s;
  s = s > ksteps ? ksteps : s;
  return s;
}

hipError_t launch_skinny(const SkinnyArgs& a, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.M > 128 || a.N % 64 != 0 || a.K % 32 != 0 || a.splits < 1 || a.lda % 8 != 0)
    return hipErrorInvalidValue;
  // K slice: a multiple of 32, splits * kslice >= K
  const int ksteps = a.K / 32;
  const int kslice = ((ksteps + a.splits - 1) / a.splits) * 32;
  const dim3 grid((a.N / 16 + WAVES - 1) / WAVES, a.splits), block(64 * WAVES);
  const int mb = (a.M + 15) / 16;
  if (mb <= 1) hipLaunchKernelGGL(skinny_kernel<1>, grid, block, 0, st, a, kslice);
  else if (mb <= 2) hipLaunchKernelGGL(skinny_kernel<2>, grid, block, 0, st, a, kslice);
  else if (mb <= 4) hipLaunchKernelGGL(skinny_kernel<4>, grid, block, 0, st, a, kslice);
  else hipLaunchKernelGGL(skinny_kernel<8>, grid, block, 0, st, a, kslice);
  return hipGetLastError();
}

}  // namespace vla
