// Persistent decode layer kernel (gfx950): for one decoder layer at one decode
// step, one cooperative launch of one 256-thread workgroup per CU runs
//   O projection -> residual add + MLP RMSNorm -> gate/up projection ->
//   SwiGLU -> down projection -> residual add + the next RMSNorm ->
//   the next layer's QKV projection (or the action head's projection),
// i.e. everything of the layer after attention, with a grid barrier between
// dependent phases instead of a kernel boundary.  Decode is bound by streaming
// the weights from HBM (Sec. 3.5: the rollout's batched decoding); separate
// kernels each lose a launch ramp and a tail (a plain streaming read of one
// projection's bytes reaches only 3.7-4.6 TB/s per launch), while here the
// weight loads of each projection's first units are issued before the barrier
// that its activations wait for, so the weight stream continues across the
// phases.
//
// Arithmetic is that of the separate kernels, in the same order (the skinny
// GEMM is the shared device code of skinny_dev.h; the norm's mean square is
// reduced over the same 1024-thread tree as reduce_residual_norm_kernel), so
// the results are the same bits.
//
// Cross-workgroup data: every value a later phase reads on another workgroup
// (split-K partials, the normed activations, the SwiGLU output) is stored with
// sc1 (written through to memory) and the stores are complete before the
// workgroup arrives at the barrier; a later phase reads each such address for
// the first time in the launch, so no XCD's L2 holds an older copy of it.  The
// residual x of a row is read and written by one workgroup only.
//
// Barrier: monotonic arrive counters (zeroed before each decode call), one per
// group of workgroups (g % 8, the XCD a workgroup is dispatched to) and one
// global counter that the last arriver of each group bumps; relaxed
// agent-scope atomics, no cache maintenance.  Every wait is bounded: a timeout
// sets an abort word (zeroed with the counters) that ends every workgroup at
// its next barrier, and raises VLA_FLAG_SYNC_TIMEOUT in the flags word.
#include "common.h"
#include "kernels.h"
#include "skinny_dev.h"

namespace vla {

namespace {

using skinny::NW;

constexpr unsigned kSpinLimit = 1u << 22;
constexpr uint32_t kFlagSyncTimeout = 4u;

__device__ __forceinline__ unsigned ld_agent(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every store of this thread issued so far is complete (vmcnt counts loads and
// stores in issue order on gfx9): called at the end of a phase, before the
// next projection's weight prefetch and the grid barrier.
__device__ __forceinline__ void stores_complete() { __builtin_amdgcn_s_waitcnt(0); }

// Grid barrier number `idx` (1-based within the decode call); the caller's
// stores are complete (stores_complete).  Returns false when the wait timed out
// or another workgroup raised the abort word.
__device__ bool grid_barrier(unsigned* bar, unsigned idx, uint32_t* flags) {
  __shared__ int ok_s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned G = gridDim.x, grp = blockIdx.x & 7, ngrp = G < 8 ? G : 8;
    const unsigned n_in = (G - grp + 7) / 8;  // workgroups of this group
    const unsigned old = __hip_atomic_fetch_add(&bar[16 * (1 + grp)], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == idx * n_in) __hip_atomic_fetch_add(&bar[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned target = idx * ngrp;
    int ok = 1;
    unsigned spins = 0;
    while ((int)(ld_agent(&bar[0]) - target) < 0) {
      if (ld_agent(&bar[1])) {  // another workgroup timed out
        ok = 0;
        break;
      }
      if (++spins > kSpinLimit) {
        __hip_atomic_store(&bar[1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_or(flags, kFlagSyncTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    ok_s = ok;
  }
  __syncthreads();
  return ok_s != 0;
}

__device__ __forceinline__ void store_sc1_u64(bf16_t* p, uint32_t lo, uint32_t hi) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), (unsigned long long)lo | ((unsigned long long)hi << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Residual add of the split-K partials and RMSNorm of row m, by the 256 threads
// of one workgroup standing in for the 1024 threads of
// reduce_residual_norm_kernel: virtual thread t + 256 j takes columns
// 4 (t + 256 j + 1024 k), k = 0, 1, and the mean square is reduced per virtual
// wave and then over the 16 virtual waves in order.
__device__ void residual_norm_row(const float* __restrict__ part, const SkinnyPlan& p, float* __restrict__ x,
                                  bf16_t* __restrict__ u, const float* __restrict__ g, float eps, int m, int M,
                                  int d) {
  __shared__ float sh[16];
  float4 v[4][2];
  float ss[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int vt = threadIdx.x + 256 * j;
    ss[j] = 0.f;
#pragma unroll
    for (int k = 0; k < 2; ++k) {  // d <= 8192
      const int c = 4 * (vt + 1024 * k);
      if (c >= d) break;
      float4 a = *reinterpret_cast<const float4*>(x + (size_t)m * d + c);
      const int ns = skinny_slots(p, c >> 6);
      for (int sl = 0; sl < ns; ++sl) {
        const float4 q = *reinterpret_cast<const float4*>(part + ((size_t)sl * M + m) * d + c);
        a.x += q.x; a.y += q.y; a.z += q.z; a.w += q.w;
      }
      v[j][k] = a;
      ss[j] += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
    }
  }
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float s = wave_sum(ss[j]);
    if ((threadIdx.x & 63) == 0) sh[wave + 4 * j] = s;
  }
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += sh[w];
  const float r = rsqrtf(tot / (float)d + eps);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int vt = threadIdx.x + 256 * j;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int c = 4 * (vt + 1024 * k);
      if (c >= d) break;
      const float4 gv = *reinterpret_cast<const float4*>(g + c);
      *reinterpret_cast<float4*>(x + (size_t)m * d + c) = v[j][k];
      store_sc1_u64(u + frag_index(m, c, d), pack2bf(v[j][k].x * r * gv.x, v[j][k].y * r * gv.y),
                    pack2bf(v[j][k].z * r * gv.z, v[j][k].w * r * gv.w));
    }
  }
  __syncthreads();  // sh is reused by the next row
}

template <int MB>
__global__ __launch_bounds__(64 * NW, 1) void decode_layer_kernel(DecodeLayerArgs a) {
  extern __shared__ float red[];
  const int g = blockIdx.x, G = gridDim.x;
  skinny::Ring<MB> r;
  unsigned bi = a.bar_base;
  int ts = 0;  // trace stamp index
  auto stamp = [&]() {
    if (a.trace && threadIdx.x == 0) a.trace[(size_t)g * 16 + ts] = wall_clock64();
    ++ts;
  };
  stamp();
  // O projection (its activations are the attention output of the previous kernel)
  const skinny::Sched s_o = skinny::make_sched(a.p_o, g);
  skinny::run<MB, true>(s_o, a.o, a.p_o, r, red, false);
  stores_complete();
  const skinny::Sched s_gu = skinny::make_sched(a.p_gu, g);
  skinny::prefetch_w<MB>(s_gu, a.gu, r);  // streams while this workgroup waits for the others
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // residual add + MLP RMSNorm -> ua
  for (int m = g; m < a.M; m += G) residual_norm_row(a.o.part, a.p_o, a.x, a.ua, a.g_mlp, a.eps, m, a.M, a.d);
  stores_complete();
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // gate/up projection
  skinny::run<MB, true>(s_gu, a.gu, a.p_gu, r, red, true);
  stores_complete();
  const skinny::Sched s_dn = skinny::make_sched(a.p_dn, g);
  skinny::prefetch_w<MB>(s_dn, a.dn, r);
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // SwiGLU of the gate/up partial sums -> h (the arithmetic of reduce_swiglu_kernel)
  {
    const int F = a.Fp, N = a.p_gu.tiles * 64;
    const size_t n = (size_t)a.M * (F / 4);
    for (size_t i = (size_t)g * 256 + threadIdx.x; i < n; i += (size_t)G * 256) {
      const int m = (int)(i / (F / 4)), j = 4 * (int)(i % (F / 4));
      const int cg = 64 * (j >> 5) + (j & 31);  // gate columns cg .. cg+3, up columns 32 further
      const int ns = skinny_slots(a.p_gu, cg >> 6);
      float4 gs = make_float4(0.f, 0.f, 0.f, 0.f), us = gs;
      for (int sl = 0; sl < ns; ++sl) {
        const float* pr = a.gu.part + ((size_t)sl * a.M + m) * N + cg;
        const float4 q0 = *reinterpret_cast<const float4*>(pr), q1 = *reinterpret_cast<const float4*>(pr + 32);
        gs.x += q0.x; gs.y += q0.y; gs.z += q0.z; gs.w += q0.w;
        us.x += q1.x; us.y += q1.y; us.z += q1.z; us.w += q1.w;
      }
      auto sw = [](float p, float q) { return p / (1.f + expf(-p)) * q; };
      store_sc1_u64(a.h + frag_index(m, j, a.Fp), pack2bf(sw(gs.x, us.x), sw(gs.y, us.y)),
                    pack2bf(sw(gs.z, us.z), sw(gs.w, us.w)));
    }
  }
  stores_complete();
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // down projection
  skinny::run<MB, true>(s_dn, a.dn, a.p_dn, r, red, true);
  stores_complete();
  const skinny::Sched s_nx = skinny::make_sched(a.p_nx, g);
  skinny::prefetch_w<MB>(s_nx, a.nx, r);
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // residual add + the next RMSNorm -> ub
  for (int m = g; m < a.M; m += G) residual_norm_row(a.dn.part, a.p_dn, a.x, a.ub, a.g_next, a.eps, m, a.M, a.d);
  stores_complete();
  stamp();
  if (!grid_barrier(a.bar, ++bi, a.flags)) return;
  stamp();
  // the next layer's QKV projection, or the action head's (read by the next kernel)
  skinny::run<MB, false>(s_nx, a.nx, a.p_nx, r, red, true);
  stamp();
}

template <int MB>
hipError_t launch_mb(const DecodeLayerArgs& a, int G, hipStream_t s) {
  const size_t lds = skinny::red_bytes<MB>();
  static bool attr_set = false;
  if (!attr_set && lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_layer_kernel<MB>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  DecodeLayerArgs arg = a;
  void* args[] = {&arg};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&decode_layer_kernel<MB>), dim3(G), dim3(64 * NW),
                                    args, (unsigned)lds, s);
}

template <int MB>
bool fits_one_per_cu() {
  const size_t lds = skinny::red_bytes<MB>();
  if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_layer_kernel<MB>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return false;
  int n = 0;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(&decode_layer_kernel<MB>),
                                                      64 * NW, lds) == hipSuccess &&
         n >= 1;
}

}  // namespace

bool decode_layer_supported() {
  int dev = 0, coop = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop)
    return false;
  return fits_one_per_cu<1>() && fits_one_per_cu<2>() && fits_one_per_cu<4>() && fits_one_per_cu<8>();
}

hipError_t launch_decode_layer(const DecodeLayerArgs& a, int G, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.M > 128 || G < 1 || a.d % 64 != 0 || a.d > 8192 || a.Fp % 32 != 0 || a.p_o.tiles * 64 != a.d ||
      a.p_dn.tiles * 64 != a.d || a.p_gu.tiles * 64 < 2 * a.Fp || a.p_o.G > G || a.p_gu.G > G || a.p_dn.G > G ||
      a.p_nx.G > G)
    return hipErrorInvalidValue;
  // each projection as launch_skinny requires it
  const SkinnyArgs* gs[4] = {&a.o, &a.gu, &a.dn, &a.nx};
  const SkinnyPlan* ps[4] = {&a.p_o, &a.p_gu, &a.p_dn, &a.p_nx};
  for (int i = 0; i < 4; ++i) {
    const SkinnyArgs& g = *gs[i];
    const SkinnyPlan& p = *ps[i];
    if (g.M != a.M || g.N % skinny::COLS != 0 || g.K % skinny::UNIT_K != 0 || p.tiles != g.N / skinny::COLS ||
        p.chunks != g.K / skinny::UNIT_K || p.G < 1 || (long long)frag_elems(g.N, g.K) * 2 >= (1ll << 31))
      return hipErrorInvalidValue;
  }
  if (a.o.K != a.d || a.gu.K != a.d || a.dn.K != a.Fp || a.nx.K != a.d) return hipErrorInvalidValue;
  const int mb = (a.M + 15) / 16;
  if (mb <= 1) return launch_mb<1>(a, G, s);
  if (mb <= 2) return launch_mb<2>(a, G, s);
  if (mb <= 4) return launch_mb<4>(a, G, s);
  return launch_mb<8>(a, G, s);
}

}  // namespace vla
