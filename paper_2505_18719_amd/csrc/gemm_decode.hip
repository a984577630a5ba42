// Decode-time skinny GEMM on gfx950: C = A * W^T for M <= 128 rows (one per
// environment), A [M, K] bf16, W [N, K] bf16, fp32 accumulation.
//
// Decode streams every weight once per step, so the kernel is shaped for HBM
// bandwidth and for balance over the CUs:
//  - One persistent 256-thread workgroup per CU.  The work is cut into units
//    of 64 output columns x 256 K.  Whole column tiles are dealt out one per
//    workgroup per round; the tiles left over after the last full round are
//    split into their units, and each workgroup takes an equal contiguous run
//    of those (stream-K), so every workgroup streams the same weight bytes.
//  - Every tile segment a workgroup finishes is written as an fp32 partial
//    sum into a slot of a partial buffer; the consumer kernel adds a tile's
//    slots in slot order, so results are bitwise deterministic.  The slot of
//    a segment and a tile's slot count follow from the plan in closed form.
//  - Within a unit the four waves take one 64-wide K step each, as two
//    v_mfma_f32_16x16x32_bf16 k-steps.  Weights and activations are both in
//    frag layout, so every load instruction reads one contiguous 1 KB block
//    that leaves each lane holding its MFMA fragment (the number of memory
//    requests per byte is what bounds this kernel).  Loads run a ring of units
//    ahead of the MFMAs (about 96 KB of weights in flight per CU), pinned in
//    issue order.
//  - The activations (<= 128 x K bf16) are read through L2, where every
//    workgroup of the GPU shares them; owning 64 columns amortises each
//    activation fragment over four weight fragments.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int COLS = 64;   // output columns per tile
constexpr int NW = 4;      // waves per workgroup
constexpr int UNIT_K = 256;
#define PIN() __builtin_amdgcn_sched_barrier(0)

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 as_uint4(u32x4_t v) { return make_uint4(v.x, v.y, v.z, v.w); }

// Ring depth (units in flight) by the number of 16-row blocks of A.
template <int MB>
constexpr int ring_depth() { return MB <= 4 ? 3 : 2; }

template <int MB>
__global__ __launch_bounds__(64 * NW, 1) void skinny_kernel(SkinnyArgs a, SkinnyPlan p) {
  extern __shared__ float red[];  // [NW][MB*16][COLS]
  constexpr int D = ring_depth<MB>();
  constexpr int ROWS = MB * 16;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: keeps load offsets scalar
  const int r16 = lane & 15, g4 = lane >> 4;
  const int G = p.G, g = blockIdx.x, C = p.chunks;

  // this workgroup's units: whole tiles first, then its stream-K run
  const int n_dp = (p.dp_tiles / G) * C;
  const int U = (p.tiles - p.dp_tiles) * C;
  const int su0 = (int)(((long long)g * U) / G), su1 = (int)(((long long)(g + 1) * U) / G);
  const int total = n_dp + (su1 - su0);
  auto unit_tile = [&](int i, int& chunk) {
    if (i < n_dp) {
      chunk = i % C;
      return (i / C) * G + g;
    }
    const int su = su0 + i - n_dp;
    chunk = su % C;
    return p.dp_tiles + su / C;
  };

  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  // W and A are in frag layout: the fragment of block (row block, K block) is
  // 1 KB at ((row block) * frag_kb(K) + K block) * 1024, lane l's 16 bytes at 16 l
  const uint32_t loff = lane * 16;
  const int KB = frag_kb(a.K);  // blocks per 16-row block (frag layout)

  uint4 wr[D][4][2], ar[D][MB][2];
  // issue the loads of unit i (clamped: past the end the last unit is re-read) into a ring slot;
  // the wave takes K blocks 8 chunk + 2 wave + h, h = 0, 1
  auto load = [&](int i, uint4 (&w)[4][2], uint4 (&x)[MB][2]) {
    int chunk;
    const int tile = unit_tile(min(i, total - 1), chunk);
    const int kb = 8 * chunk + 2 * wave;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        w[nb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsW, loff, ((tile * 4 + nb) * KB + kb + h) * 1024, 0));
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        x[mb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsA, loff, (mb * KB + kb + h) * 1024, 0));
  };

  f32x4 acc[MB][4];
  auto zero = [&]() {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  zero();

  // Reduce the four waves' partial tiles through LDS and store the segment's
  // partial sum into its slot.  acc[mb][nb][r] is row mb*16 + 4*g4 + r,
  // column nb*16 + r16 of the tile.
  auto flush = [&](int tile) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[(wave * ROWS + mb * 16 + 4 * g4 + r) * COLS + nb * 16 + r16] = acc[mb][nb][r];
    __syncthreads();
    int slot = 0;
    if (tile >= p.dp_tiles) {
      const int t = tile - p.dp_tiles;
      slot = g - skinny_owner(t * C, U, G);
    }
    float* out = a.part + (size_t)slot * a.M * a.N + tile * COLS;
    for (int e = threadIdx.x; e < ROWS * COLS; e += 64 * NW) {
      const int row = e / COLS, c = e % COLS;
      if (row >= a.M) break;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += red[(w * ROWS + row) * COLS + c];
      out[(size_t)row * a.N + c] = v;
    }
    __syncthreads();
    zero();
  };

  // unit i: MFMAs on ring slot i % D, after issuing the loads of unit i + D - 1
  auto step = [&](int i, uint4 (&w)[4][2], uint4 (&x)[MB][2], uint4 (&wn)[4][2], uint4 (&xn)[MB][2]) {
    load(i + D - 1, wn, xn);  // unconditional, so the wait counts are the same on every path
    PIN();
    if (i < total) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma16(as_bf16x8(x[mb][h]), as_bf16x8(w[nb][h]), acc[mb][nb]);
      int c0, c1;
      const int t0 = unit_tile(i, c0);
      if (i + 1 >= total || unit_tile(i + 1, c1) != t0) flush(t0);
    }
    PIN();
  };

  if (total <= 0) return;
#pragma unroll
  for (int j = 0; j < D - 1; ++j) load(j, wr[j], ar[j]);
  for (int i = 0; i < total; i += D) {
    // ring slots rotate statically: unit i + j uses slot j, its loads go to slot (j + D - 1) % D
#pragma unroll
    for (int j = 0; j < D; ++j) step(i + j, wr[j], ar[j], wr[(j + D - 1) % D], ar[(j + D - 1) % D]);
  }
}

template <int MB>
hipError_t launch_mb(const SkinnyArgs& a, const SkinnyPlan& p, hipStream_t st) {
  const size_t lds = (size_t)NW * MB * 16 * COLS * sizeof(float);
  static bool attr_set = false;  // dynamic LDS above 64 KB must be allowed once per kernel
  if (!attr_set && lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&skinny_kernel<MB>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((skinny_kernel<MB>), dim3(p.G), dim3(64 * NW), lds, st, a, p);
  return hipGetLastError();
}

}  // namespace

SkinnyPlan skinny_plan(int N, int K, int workgroups, int max_slots) {
  SkinnyPlan p{};
  p.tiles = N / COLS;
  p.chunks = K / UNIT_K;
  for (int G = workgroups; G >= 1; --G) {
    p.G = G;
    p.dp_tiles = (p.tiles / G) * G;
    const int U = (p.tiles - p.dp_tiles) * p.chunks;
    if (U > 0 && U < G) continue;  // every workgroup of a stream-K run needs at least one unit
    p.slots = 1;
    for (int t = p.dp_tiles; t < p.tiles; ++t) p.slots = std::max(p.slots, skinny_slots(p, t));
    if (p.slots <= max_slots) break;
  }
  return p;
}

hipError_t launch_skinny(const SkinnyArgs& a, const SkinnyPlan& p, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.M > 128 || a.N % COLS != 0 || a.K % UNIT_K != 0 || p.tiles != a.N / COLS ||
      p.chunks != a.K / UNIT_K || p.G < 1 || (long long)frag_elems(a.N, a.K) * 2 >= (1ll << 31))
    return hipErrorInvalidValue;
  const int mb = (a.M + 15) / 16;
  if (mb <= 1) return launch_mb<1>(a, p, st);
  if (mb <= 2) return launch_mb<2>(a, p, st);
  if (mb <= 4) return launch_mb<4>(a, p, st);
  return launch_mb<8>(a, p, st);
}

}  // namespace vla
