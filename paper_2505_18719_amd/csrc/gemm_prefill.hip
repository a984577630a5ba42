// Prefill GEMM on gfx950 MFMA: C = A * W^T, A [M, K] bf16, W [N, K] bf16,
// fp32 accumulation, with fused epilogues (residual add, SwiGLU, RoPE + paged
// KV append).
//
// Tiling: a 512-thread workgroup (8 wave64s, two per SIMD) owns a 256 x 256
// output tile; each wave owns 128 x 64 of it as 8 x 4 blocks of
// v_mfma_f32_16x16x32_bf16 (128 fp32 accumulators per lane).
//
// Ping-pong: waves 0-3 and 4-7 form two groups that run half a phase apart,
// separated by workgroup barriers.  While one group issues its 32 MFMAs of a
// K step of 32, the wave of the other group on the same SIMD reads its
// operand fragments of that step from LDS and issues its share of the copies
// of a later step, so the MFMA pipe of every SIMD is fed alternately by its
// two waves and a memory instruction that stalls never holds up an MFMA.
//
// Operands: A and W are in frag layout (see frag_index), so a K step of either
// 256-row panel is sixteen 1 KB blocks, each one v_mfma_f32_16x16x32 operand,
// and every copy moves one block whole with buffer_load ... lds (global to
// LDS, no VGPR round trip, one contiguous 1 KB read per wave instruction).
// The copies run four K steps ahead through a ring of five 32 KB stages (all
// 160 KB of LDS).  An operand read is one 16-byte LDS read per lane of a
// contiguous block: free of bank conflicts without a swizzle.
//
// Why these choices: the kernel runs at the chip's power limit (the shader
// clock measured inside it is 1.2-1.75 GHz with all CUs busy, depending on the
// board), so what counts is issue efficiency per clock and energy per flop.
// The two-waves-per-SIMD ping-pong keeps the MFMA pipe fed (measured 93-96 % of
// MFMA cycles in the main loop); the 16x16x32 instruction moves half the accumulator register traffic
// per flop of the 32x32x16 one and ran ~5 % faster at the same tiling.
// Workgroup ids are remapped so that the tiles one XCD runs are contiguous in
// a grouped order (4 tile-rows high), which keeps A and W panels shared in
// that XCD's L2.  The grid is persistent (one workgroup per CU walking its
// tiles in that order): a finished tile's stores are still draining while the
// next tile's first copies are issued, where a workgroup that ended would
// hold its CU until they had drained.  With the SwiGLU epilogue the tile
// boundary overlaps further: the last four iterations copy the next tile's
// first four K steps (instead of re-copying the last one), the epilogue works
// out of the one stage those copies leave free, and since vmcnt retires in
// issue order, the next tile's first three waits count past the epilogue's
// stores (a fixed number per wave), which drain while its first steps run.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace vla {

namespace {

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int NT = 512;                // 8 waves: 2 x 4, each owning 128 x 64 of the tile
constexpr int NSTAGE = 5;              // LDS ring of K steps: A 16 KB + W 16 KB each
constexpr int AHEAD = 4;               // K steps whose copies are in flight ahead of the one read
constexpr int STAGE_U4 = 2 * 16 * 64;  // uint4 per stage: 2 operands x 16 blocks x 64 lanes
constexpr int GROUP_M = 4;

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

// SwiGLU epilogue: columns [c0, c0+32) of a 64-column group are gate rows,
// [c0+32, c0+64) the matching up rows.  v1, v2: float4 chunks q and q + 8 of
// output row `row`, group starting at column c0.
template <int EPI>
__device__ __forceinline__ void swiglu_epilogue(const GemmArgs& a, int row, int c0, int q, const float4& v1,
                                                const float4& v2) {
  const float x1[4] = {v1.x, v1.y, v1.z, v1.w}, x2[4] = {v2.x, v2.y, v2.z, v2.w};
  float o[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) o[t] = x1[t] / (1.f + expf(-x1[t])) * x2[t];
  *reinterpret_cast<uint2*>(a.H + frag_index(row, c0 / 2 + 4 * q, a.ldh)) =  // frag layout, K = ldh
      make_uint2(pack2bf(o[0], o[1]), pack2bf(o[2], o[3]));
  if constexpr (EPI == kEpiSwiGluKeep) {
    float* cr = a.C + (size_t)row * a.ldc + c0 + 4 * q;
    *reinterpret_cast<float4*>(cr) = v1;
    *reinterpret_cast<float4*>(cr + 32) = v2;
  }
}

// Epilogues that run while the next tile's first AHEAD K steps are being copied
// (they stage through one 32 KB ring stage only), and the number of vector
// memory instructions each of their waves issues (a constant, so that the next
// tile's first waits can count past them).
template <int EPI>
constexpr bool overlaps_next() { return EPI == kEpiSwiGlu; }
template <int EPI>
constexpr int epi_vm_ops() { return EPI == kEpiSwiGlu ? 8 : 0; }

// Tile `pid` of G (in the XCD-aware order of map_tile): main loop and epilogue.
// ring0: the ring stage of this tile's K step 0.  pending: -1 when no copy of
// this tile is in flight yet; otherwise the previous tile's last iterations
// copied this tile's first AHEAD steps (step 0 has landed) and `pending` is the
// number of vector memory instructions its epilogue issued after them.
template <int EPI>
__device__ __forceinline__ void gemm_tile(const GemmArgs& a, int tiles_m, int tiles_n, int pid, int G,
                                          uint4 (&lds)[NSTAGE][STAGE_U4], int& ring0, int& pending) {
  int tm, tn;
  map_tile(pid, G, tiles_m, tiles_n, tm, tn);
  const int M = a.M, N = a.N, K = a.K;
  const int m0 = tm * BM, n0 = tn * BN;
  // threadIdx.x through an opaque copy: the per-lane values below are then recomputed for
  // every tile instead of being hoisted out of the tile loop and kept live through it
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int wm = wave & 1, wn = wave >> 1;  // 128-row half, 64-column quarter of the tile
  const int KB = frag_kb(wave < 4 ? (a.ka ? a.ka : K) : (a.kw ? a.kw : K));  // frag row stride of the copied operand
  const int last_rb_a = (M + 15) / 16 - 1, last_rb_w = N / 16 - 1;

  // copies: wave w moves blocks 4 w .. 4 w + 3 of a step's 32 (waves 0-3: A, 4-7: W)
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, 0x7fffffff, 0x00020000);
  const bool copies_a = wave < 4;
  const __amdgpu_buffer_rsrc_t rsC = copies_a ? rsA : rsW;
  const int rb0 = copies_a ? (m0 >> 4) : (n0 >> 4), rb_last = copies_a ? last_rb_a : last_rb_w;
  const uint32_t voff = lane * 16;
  const uint32_t lds_base = (uint32_t)(uintptr_t)((lds_ptr_t*)&lds[0][0]);
  auto copy = [&](int j, int st, int rb, int ks) {
    const int b = wave * 4 + j;
    lds_dma16(lds_base + (st * STAGE_U4 + b * 64) * 16, voff, rsC, (min(rb + (b & 15), rb_last) * KB + ks) * 1024);
  };
  const int nk = K / BK;
  // the last AHEAD iterations copy the next tile's first steps instead of re-copying the last one
  const bool ov = overlaps_next<EPI>() && nk > AHEAD;
  const int npid = pid + (int)gridDim.x;
  const bool has_next = ov && npid < G;
  int rb0n = rb0;
  if (has_next) {
    int tmn, tnn;
    map_tile(npid, G, tiles_m, tiles_n, tmn, tnn);
    rb0n = copies_a ? (tmn * BM) >> 4 : (tnn * BN) >> 4;
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // 16x16x32 fragments: A rows 128 wm + 16 i are frag block 8 wm + i, W rows
  // 64 wn + 16 j block 4 wn + j; a lane's 16 bytes sit at 16 * lane of a block
  const int fa = (wm * 8) * 64 + lane;
  const int fw = (16 + wn * 4) * 64 + lane;
  const uint4* ring = &lds[0][0];
  bf16x8 fa_r[8], fw_r[4];

  if (pending < 0) {
#pragma unroll
    for (int st = 0; st < AHEAD; ++st)
#pragma unroll
      for (int j = 0; j < 4; ++j) copy(j, (ring0 + st) % NSTAGE, rb0, min(st, nk - 1));
    WAIT_VMCNT(4 * (AHEAD - 1));
  }
  __builtin_amdgcn_s_barrier();
  if (grp) __builtin_amdgcn_s_barrier();
  PIN();
  int cur = ring0, fill = (ring0 + AHEAD) % NSTAGE;
  // One K step.  `wide`: the previous epilogue's epi_vm_ops instructions were issued
  // after this tile's first AHEAD steps' copies, so until step AHEAD's wait they sit
  // between the copies waited for and the newer ones (vmcnt retires in issue order).
  auto k_step = [&](int kt, bool wide) {
    // ---- memory phase: operand fragments of step kt, copies of step kt + AHEAD
    const uint4* sp = ring + cur * STAGE_U4;
#pragma unroll
    for (int i = 0; i < 8; ++i) fa_r[i] = as_bf16x8(sp[fa + i * 64]);
#pragma unroll
    for (int j = 0; j < 4; ++j) fw_r[j] = as_bf16x8(sp[fw + j * 64]);
    // past the end: the next tile's first steps, or (no next tile) the last step again
    const int kk = kt + AHEAD;
    const bool past = kk >= nk;
    const int rbf = past && has_next ? rb0n : rb0;
    const int kfill = !past ? kk : (has_next ? kk - nk : nk - 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) copy(j, fill, rbf, kfill);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fragments in registers, this stage's reads done
    if (wide) WAIT_VMCNT(4 * (AHEAD - 1) + epi_vm_ops<EPI>());  // this wave's copies of step kt + 1 have landed
    else WAIT_VMCNT(4 * (AHEAD - 1));
    PIN();
    __builtin_amdgcn_s_barrier();
    PIN();
    // ---- compute phase
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(fa_r[i], fw_r[j], acc[i][j]);
    PIN();
    __builtin_amdgcn_s_barrier();
    PIN();
    cur = cur + 1 == NSTAGE ? 0 : cur + 1;
    fill = fill + 1 == NSTAGE ? 0 : fill + 1;
  };
  int kt = 0;
  if (overlaps_next<EPI>() && pending > 0)
    for (; kt < AHEAD - 1; ++kt) k_step(kt, true);
  for (; kt < nk; ++kt) k_step(kt, false);
  if (!grp) __builtin_amdgcn_s_barrier();
  if (ov) {
    // the next tile's copies stay in flight; this tile's own copies have all landed
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
  } else {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  const int stage_out = (ring0 + nk - 1) % NSTAGE;  // the last step's stage: free for staging
  if (ov) ring0 = (ring0 + nk) % NSTAGE;
  pending = has_next ? 0 : -1;

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][r] holds row 16 i + 4 (lane / 16) + r, column 16 j + lane % 16 of the wave tile
  const int c0 = n0 + wn * 64;
  if (c0 >= N) return;
  if constexpr (EPI == kEpiSwiGlu) {
    // h = silu(gate) * up straight from the accumulators: the wave's 64 columns are
    // 32 gate columns (j = 0, 1) and the matching up columns (j = 2, 3), so h of row
    // 16 i + 4 (lane / 16) + r, feature 16 j + lane % 16 (j < 2) is in this lane.  Each
    // 16-row block i of the wave's 32 features is one 1 KB frag block of H: it is
    // transposed through 1 KB of the free stage and stored whole (16 bytes per lane).
    // Stores of blocks past the last row block are dropped by the buffer's bound.
    bf16_t* stg = reinterpret_cast<bf16_t*>(&lds[stage_out][0]) + wave * 2048;  // 4 KB per wave
    const __amdgpu_buffer_rsrc_t rsH = __builtin_amdgcn_make_buffer_rsrc(
        (void*)a.H, (short)0, (int)(frag_elems(M, a.ldh) * 2), 0x00020000);
    const int kbh = frag_kb(a.ldh), fblk = c0 >> 6;
#pragma unroll
    for (int rnd = 0; rnd < 2; ++rnd) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float x1 = acc[4 * rnd + ii][j][r], x2 = acc[4 * rnd + ii][j + 2][r];
            const int rho = 4 * (lane >> 4) + r, f = 16 * j + (lane & 15);
            stg[ii * 512 + (rho + 16 * (f >> 3)) * 8 + (f & 7)] = f2bf(x1 / (1.f + expf(-x1)) * x2);
          }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const uint4 v = reinterpret_cast<const uint4*>(stg)[ii * 64 + lane];
        const int rb = (m0 + wm * 128 + 16 * (4 * rnd + ii)) >> 4;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rsH,
                                               (uint32_t)(((rb * kbh + fblk) * 64 + lane) * 16), 0, 0);
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // this round's reads are done before the next round's writes
    }
    if (has_next) pending = epi_vm_ops<EPI>();
    return;
  }
  float* st = reinterpret_cast<float*>(&lds[0][0]) + wave * (64 * 64);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int wrow0 = m0 + wm * 128 + h * 64;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rl = ii * 16 + 4 * (lane >> 4) + r;
          const int cl = jj * 16 + (lane & 15);
          st[rl * 64 + (((cl >> 2) ^ (rl & 15)) << 2) + (cl & 3)] = acc[4 * h + ii][jj][r];
        }
    // the wave's own staging area: its LDS writes and reads are ordered (no wait for global stores here)
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    if constexpr (EPI == kEpiStoreF32 || EPI == kEpiResidual) {
      const int q = lane & 15;
      float4 res[16];
      if constexpr (EPI == kEpiResidual) {
        // every residual row of the half is loaded before the first store (independent loads in flight)
#pragma unroll
        for (int it = 0; it < 16; ++it) {
          const int row = wrow0 + it * 4 + (lane >> 4);
          const float* src = a.R ? a.R : a.C;
          if (row < M) res[it] = *reinterpret_cast<const float4*>(src + (size_t)row * a.ldc + c0 + 4 * q);
        }
      }
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int rl = it * 4 + (lane >> 4);
        const int row = wrow0 + rl;
        const float4 v = *reinterpret_cast<const float4*>(st + rl * 64 + ((q ^ (rl & 15)) << 2));
        if (row < M) {
          float4* p = reinterpret_cast<float4*>(a.C + (size_t)row * a.ldc + c0 + 4 * q);
          if constexpr (EPI == kEpiResidual) {
            const float4 o = res[it];
            *p = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
          } else {
            *p = v;
          }
        }
      }
    } else if constexpr (EPI == kEpiQkvRope) {
      // RoPE + q store / paged K, V append for this half's 64 rows.  The rows' positions, pages
      // and rotary factors are loaded together first (the loads of one row depend on each other:
      // position -> page, rotary factors).
      const int d = a.d_model, hd = a.head_dim, H = a.n_heads, half = hd / 2;
      const int region = c0 / d;  // 0 q, 1 k, 2 v: one region per 64-column group
      const int cc0 = c0 - region * d;
      const int head = cc0 / hd;
      const int blk = (cc0 % hd) / 64;
      if (region < 2) {
        // q, k: the group's columns are 32 first-half features and their rotary partners; lane
        // takes 8 consecutive ones (octet q8) and their partners for 4 rows (16 rows a pass), so
        // every store is 16 bytes
        const int q8 = lane & 3;
        const int ai = 32 * blk + 8 * q8;
        int pos[4], page[4];
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int row = wrow0 + it * 16 + (lane >> 2);
          pos[it] = row < M ? a.meta.row_pos[row] : 0;
          page[it] = row < M ? a.meta.row_env[row] : 0;
        }
        if (region == 1) {
#pragma unroll
          for (int it = 0; it < 4; ++it) page[it] = a.meta.page_table[page[it] * a.meta.max_pages + pos[it] / kPage];
        }
        float4 cs[4][4];  // (cos, sin) of rotary pairs ai .. ai + 7 at each row's position
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const float4* rp = reinterpret_cast<const float4*>(a.rope + pos[it] * half + ai);
#pragma unroll
          for (int u = 0; u < 4; ++u) cs[it][u] = rp[u];
        }
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int rl = it * 16 + (lane >> 2);
          const int row = wrow0 + rl;
          float x1[8], x2[8];
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const float4 v1 = *reinterpret_cast<const float4*>(st + rl * 64 + (((2 * q8 + h2) ^ (rl & 15)) << 2));
            const float4 v2 = *reinterpret_cast<const float4*>(st + rl * 64 + (((8 + 2 * q8 + h2) ^ (rl & 15)) << 2));
            x1[4 * h2] = v1.x; x1[4 * h2 + 1] = v1.y; x1[4 * h2 + 2] = v1.z; x1[4 * h2 + 3] = v1.w;
            x2[4 * h2] = v2.x; x2[4 * h2 + 1] = v2.y; x2[4 * h2 + 2] = v2.z; x2[4 * h2 + 3] = v2.w;
          }
          if (row >= M) continue;
          float o1[8], o2[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {  // the rotation, with its fused multiply-adds spelled out
            const float c = (t & 1) ? cs[it][t >> 1].z : cs[it][t >> 1].x;
            const float sn = (t & 1) ? cs[it][t >> 1].w : cs[it][t >> 1].y;
            o1[t] = fmaf(x1[t], c, -(x2[t] * sn));
            o2[t] = fmaf(x2[t], c, x1[t] * sn);
          }
          bf16_t* dst = region == 0 ? a.q + (size_t)row * a.ldq + head * hd
                                    : a.kv.k + (((size_t)page[it] * H + head) * kPage + pos[it] % kPage) * hd;
          *reinterpret_cast<uint4*>(dst + ai) =
              make_uint4(pack2bf(o1[0], o1[1]), pack2bf(o1[2], o1[3]), pack2bf(o1[4], o1[5]), pack2bf(o1[6], o1[7]));
          *reinterpret_cast<uint4*>(dst + half + ai) =
              make_uint4(pack2bf(o2[0], o2[1]), pack2bf(o2[2], o2[3]), pack2bf(o2[4], o2[5]), pack2bf(o2[6], o2[7]));
        }
      } else {
        // v: 8 rows per lane, 4 features and the 4 of the group's second half; the cache keeps V
        // transposed (16 keys of one feature per 32 bytes), and the 8 lanes that share a feature
        // hold 8 consecutive rows, so their 2-byte stores fill 16-byte pieces
        const int q = lane & 7;
        int pos[8], page[8];
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int row = wrow0 + it * 8 + (lane >> 3);
          pos[it] = row < M ? a.meta.row_pos[row] : 0;
          page[it] = row < M ? a.meta.row_env[row] : 0;
        }
#pragma unroll
        for (int it = 0; it < 8; ++it) page[it] = a.meta.page_table[page[it] * a.meta.max_pages + pos[it] / kPage];
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int rl = it * 8 + (lane >> 3);
          const int row = wrow0 + rl;
          const float4 v1 = *reinterpret_cast<const float4*>(st + rl * 64 + ((q ^ (rl & 15)) << 2));
          const float4 v2 = *reinterpret_cast<const float4*>(st + rl * 64 + (((q + 8) ^ (rl & 15)) << 2));
          if (row >= M) continue;
          const float x1[4] = {v1.x, v1.y, v1.z, v1.w}, x2[4] = {v2.x, v2.y, v2.z, v2.w};
          bf16_t* vb = a.kv.v + ((size_t)page[it] * H + head) * hd * kPage + pos[it] % kPage;
          const int i1 = cc0 % hd + 4 * q;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            vb[(size_t)(i1 + t) * kPage] = f2bf(x1[t]);
            vb[(size_t)(i1 + t + 32) * kPage] = f2bf(x2[t]);
          }
        }
      }
    } else {
      const int q = lane & 7;
      for (int it = 0; it < 8; ++it) {
        const int rl = it * 8 + (lane >> 3);
        const int row = wrow0 + rl;
        const float4 v1 = *reinterpret_cast<const float4*>(st + rl * 64 + ((q ^ (rl & 15)) << 2));
        const float4 v2 = *reinterpret_cast<const float4*>(st + rl * 64 + (((q + 8) ^ (rl & 15)) << 2));
        if (row >= M) continue;
        swiglu_epilogue<EPI>(a, row, c0, q, v1, v2);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this half's staging reads are done before the next half's writes
  }
}

// One workgroup per CU walks the tiles pid = blockIdx.x, blockIdx.x + gridDim.x,
// ... (gridDim.x is a multiple of 8, so a workgroup's tiles stay on its XCD's
// band).  The next tile's copies are issued as soon as every wave has read its
// staged outputs, while the previous tile's stores are still draining (a
// workgroup that ended instead would hold its CU until they had drained).
template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs a, int tiles_m, int tiles_n) {
  __shared__ uint4 lds[NSTAGE][STAGE_U4];
  const int G = tiles_m * tiles_n;
  int ring0 = 0, pending = -1;
  for (int pid = blockIdx.x; pid < G; pid += gridDim.x) {
    gemm_tile<EPI>(a, tiles_m, tiles_n, pid, G, lds, ring0, pending);
    // every wave's staging reads are done (each half ends with lgkmcnt(0)) before the
    // ring is refilled; a plain barrier, so that no wait covers the stores in flight
    __builtin_amdgcn_s_barrier();
  }
}

}  // namespace

// One workgroup per CU of the current device, rounded down to a multiple of 8 (the XCDs).
static int persistent_workgroups() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 8;
  if (!cus[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8) n = 8;
    cus[dev] = n / 8 * 8;
  }
  return cus[dev];
}

hipError_t launch_gemm(const GemmArgs& a, GemmEpilogue epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  // frag-layout operands, 32-bit byte offsets into them
  const int ka = a.ka ? a.ka : a.K, kw = a.kw ? a.kw : a.K;
  if (a.K % BK != 0 || a.N % 64 != 0 || ka < a.K || kw < a.K || ka % 32 != 0 || kw % 32 != 0 ||
      (long long)frag_elems(a.M, ka) * 2 >= (1ll << 31) || (long long)frag_elems(a.N, kw) * 2 >= (1ll << 31))
    return hipErrorInvalidValue;
  const int tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  const dim3 grid(std::min(tm * tn, persistent_workgroups())), block(NT);
  switch (epi) {
    case kEpiStoreF32: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiStoreF32>, grid, block, 0, s, a, tm, tn); break;
    case kEpiResidual: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiResidual>, grid, block, 0, s, a, tm, tn); break;
    case kEpiSwiGlu: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiSwiGlu>, grid, block, 0, s, a, tm, tn); break;
    case kEpiQkvRope: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiQkvRope>, grid, block, 0, s, a, tm, tn); break;
    case kEpiSwiGluKeep:
      if (!a.C || a.ldc % 4 != 0 || a.ldc < a.N) return hipErrorInvalidValue;
      hipLaunchKernelGGL(gemm_bf16_kernel<kEpiSwiGluKeep>, grid, block, 0, s, a, tm, tn);
      break;
  }
  return hipGetLastError();
}

}  // namespace vla
