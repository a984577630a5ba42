// Device side of the decode-time skinny GEMM (C = A W^T for M <= 128 rows),
// shared by the standalone kernel (gemm_decode.hip) and the persistent decode
// layer kernel (decode_layer.hip).
//
// Work is cut into units of 64 output columns x 256 of K; a workgroup of four
// waves takes its whole tiles first, then an equal contiguous stream-K run of
// the leftover tiles' units.  Each wave takes one 64-wide K step of a unit as
// two v_mfma_f32_16x16x32_bf16 k-steps; weights and activations are frag
// blocks (one contiguous 1 KB per load instruction).  A ring of units keeps
// loads in flight ahead of the MFMAs.  Every finished tile segment is reduced
// across the waves through LDS and stored as an fp32 partial into a slot that
// follows from the plan in closed form; consumers add a tile's slots in slot
// order (bitwise deterministic).
#pragma once

#include "common.h"
#include "kernels.h"

namespace vla {
namespace skinny {

constexpr int COLS = 64;   // output columns per tile
constexpr int NW = 4;      // waves per workgroup
constexpr int UNIT_K = 256;
#define SKINNY_PIN() __builtin_amdgcn_sched_barrier(0)

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 as_uint4(u32x4_t v) { return make_uint4(v.x, v.y, v.z, v.w); }

// Ring depths (units in flight) of the weights and of the activations.  The
// weights of the next unit are in flight while a unit's MFMAs run; a unit's
// activations (shared by an XCD's workgroups, so L2 hits) are loaded in the
// step that uses them.  Measured at 8 to 128 rows on the four projection
// shapes: deeper rings (2-5 units ahead, with the activations as deep as the
// weights) were 2-13 % slower per launch, since the extra loads only queue
// and the registers they take leave the accumulators shuffled between the two
// register files; at 8 row blocks the deeper rings also spilled.
template <int MB>
constexpr int ring_depth() { return 2; }
template <int MB>
constexpr int x_ring_depth() { return 1; }
constexpr int gcd_(int a, int b) { return b == 0 ? a : gcd_(b, a % b); }

// LDS bytes of the cross-wave reduction.
template <int MB>
constexpr size_t red_bytes() { return (size_t)NW * MB * 16 * COLS * sizeof(float); }

template <int MB>
struct Ring {
  uint4 w[ring_depth<MB>()][4][2];
  uint4 x[x_ring_depth<MB>()][MB][2];
};

// The units of workgroup g under plan p: whole tiles first, then its stream-K run.
struct Sched {
  int g, G, C, dp_tiles, n_dp, U, su0, total;
  __device__ __forceinline__ int unit_tile(int i, int& chunk) const {
    if (i < n_dp) {
      chunk = i % C;
      return (i / C) * G + g;
    }
    const int su = su0 + i - n_dp;
    chunk = su % C;
    return dp_tiles + su / C;
  }
};

__device__ __forceinline__ Sched make_sched(const SkinnyPlan& p, int g) {
  Sched s;
  s.g = g;
  s.G = p.G;
  s.C = p.chunks;
  s.dp_tiles = p.dp_tiles;
  s.n_dp = (p.dp_tiles / p.G) * p.chunks;
  s.U = (p.tiles - p.dp_tiles) * p.chunks;
  s.su0 = (int)(((long long)g * s.U) / p.G);
  const int su1 = (int)(((long long)(g + 1) * s.U) / p.G);
  s.total = g < p.G ? s.n_dp + (su1 - s.su0) : 0;
  return s;
}

// Weight / activation fragments of unit i (clamped: past the end the last unit
// is re-read) into ring slot (w, x); the wave takes K blocks 8 chunk + 2 wave + h.
template <int MB>
__device__ __forceinline__ void load_w(const Sched& sc, const SkinnyArgs& a, int i, int wave, uint4 (&w)[4][2]) {
  int chunk;
  const int tile = sc.unit_tile(min(i, sc.total - 1), chunk);
  const int kb = 8 * chunk + 2 * wave, KB = frag_kb(a.K);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  const uint32_t loff = (threadIdx.x & 63) * 16;
#pragma unroll
  for (int nb = 0; nb < 4; ++nb)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      w[nb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsW, loff, ((tile * 4 + nb) * KB + kb + h) * 1024, 0));
}

template <int MB>
__device__ __forceinline__ void load_x(const Sched& sc, const SkinnyArgs& a, int i, int wave, uint4 (&x)[MB][2]) {
  int chunk;
  (void)sc.unit_tile(min(i, sc.total - 1), chunk);
  const int kb = 8 * chunk + 2 * wave, KB = frag_kb(a.K);
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  const uint32_t loff = (threadIdx.x & 63) * 16;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      x[mb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsA, loff, (mb * KB + kb + h) * 1024, 0));
}

// Issue the weight loads of the first ring_depth - 1 units (e.g. before a grid
// barrier that the activations wait for).
template <int MB>
__device__ __forceinline__ void prefetch_w(const Sched& sc, const SkinnyArgs& a, Ring<MB>& r) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (sc.total <= 0) return;
#pragma unroll
  for (int j = 0; j < ring_depth<MB>() - 1; ++j) load_w<MB>(sc, a, j, wave, r.w[j]);
}

// All units of workgroup sc.g.  `red` is LDS of red_bytes<MB>().  With
// `prefetched`, the weights of the first ring_depth - 1 units were loaded by
// prefetch_w.  SC1: partial sums are written through to memory (sc1 stores), so
// that workgroups of other XCDs can read them after a grid barrier without a
// cache write-back.
template <int MB, bool SC1>
__device__ __forceinline__ void run(const Sched& sc, const SkinnyArgs& a, const SkinnyPlan& p, Ring<MB>& r,
                                    float* red, bool prefetched) {
  constexpr int D = ring_depth<MB>(), DX = x_ring_depth<MB>();
  constexpr int P = D * DX / gcd_(D, DX);  // the rings' common period
  constexpr int ROWS = MB * 16;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: keeps load offsets scalar
  const int r16 = lane & 15, g4 = lane >> 4;
  const int total = sc.total;
  if (total <= 0) return;

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
        for (int q = 0; q < 4; ++q) red[(wave * ROWS + mb * 16 + 4 * g4 + q) * COLS + nb * 16 + r16] = acc[mb][nb][q];
    __syncthreads();
    int slot = 0;
    if (tile >= p.dp_tiles) {
      const int t = tile - p.dp_tiles;
      slot = sc.g - skinny_owner(t * p.chunks, sc.U, p.G);
    }
    float* out = a.part + (size_t)slot * a.M * a.N + tile * COLS;
    for (int e = threadIdx.x; e < ROWS * COLS; e += 64 * NW) {
      const int row = e / COLS, c = e % COLS;
      if (row >= a.M) break;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += red[(w * ROWS + row) * COLS + c];
      if constexpr (SC1) __hip_atomic_store(out + (size_t)row * a.N + c, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else out[(size_t)row * a.N + c] = v;
    }
    __syncthreads();
    zero();
  };

  const int KB = frag_kb(a.K);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  const uint32_t loff = lane * 16;
  auto ldw = [&](int i, uint4 (&wv)[4][2]) {
    int chunk;
    const int tile = sc.unit_tile(min(i, total - 1), chunk);
    const int kb = 8 * chunk + 2 * wave;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        wv[nb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsW, loff, ((tile * 4 + nb) * KB + kb + h) * 1024, 0));
  };
  auto ldx = [&](int i, uint4 (&xv)[MB][2]) {
    int chunk;
    (void)sc.unit_tile(min(i, total - 1), chunk);
    const int kb = 8 * chunk + 2 * wave;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        xv[mb][h] = as_uint4(__builtin_amdgcn_raw_buffer_load_b128(rsA, loff, (mb * KB + kb + h) * 1024, 0));
  };
  // The weight loads of unit i + D - 1 and the activation loads of unit i + DX - 1 go out before the MFMAs
  // of unit i (ring slots i % D, i % DX); they are unconditional, so that the wait counts are the same on every
  // path, and the activations go out first, so that the wait for a unit's activations does not also wait for
  // later weights.
  if (!prefetched) {
#pragma unroll
    for (int j = 0; j < D - 1; ++j) {
      if (j < DX - 1) ldx(j, r.x[j]);
      ldw(j, r.w[j]);
    }
  } else {
#pragma unroll
    for (int j = 0; j < DX - 1; ++j) ldx(j, r.x[j]);
  }
  for (int i0 = 0; i0 < total; i0 += P) {
    // ring slots rotate statically: unit i0 + j uses slots j % D and j % DX
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int i = i0 + j;
      ldx(i + DX - 1, r.x[(j + DX - 1) % DX]);
      ldw(i + D - 1, r.w[(j + D - 1) % D]);
      SKINNY_PIN();
      if (i < total) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
              acc[mb][nb] = mfma16(as_bf16x8(r.x[j % DX][mb][h]), as_bf16x8(r.w[j % D][nb][h]), acc[mb][nb]);
        int c0, c1;
        const int t0 = sc.unit_tile(i, c0);
        if (i + 1 >= total || sc.unit_tile(i + 1, c1) != t0) flush(t0);
      }
      SKINNY_PIN();
    }
  }
}

}  // namespace skinny
}  // namespace vla
