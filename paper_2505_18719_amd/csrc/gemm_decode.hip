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
//    requests per byte is what bounds this kernel).  The next unit's weights
//    are in flight while a unit's MFMAs run (32 KB per CU; deeper rings only
//    queued more loads), its activations are loaded in the step that uses
//    them, pinned in issue order.
//  - The activations (<= 128 x K bf16) are read through L2, where every
//    workgroup of an XCD shares them.  Per unit a wave loads 8 weight blocks
//    and 2 MB activation blocks (MB = 16-row blocks of A), so at 64 rows the
//    activation loads equal the weight loads in count; they hit in L2 and cost
//    about a tenth of the kernel's time (measured by leaving them out).
//  The device code is in skinny_dev.h, shared with the persistent decode
//  layer kernel.
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "skinny_dev.h"

namespace vla {

namespace {

using skinny::COLS;
using skinny::NW;
using skinny::UNIT_K;

template <int MB>
__global__ __launch_bounds__(64 * NW, 1) void skinny_kernel(SkinnyArgs a, SkinnyPlan p) {
  extern __shared__ float red[];  // [NW][MB*16][COLS]
  const skinny::Sched sc = skinny::make_sched(p, blockIdx.x);
  skinny::Ring<MB> r;
  skinny::run<MB, false>(sc, a, p, r, red, false);
}

template <int MB>
hipError_t launch_mb(const SkinnyArgs& a, const SkinnyPlan& p, hipStream_t st) {
  const size_t lds = skinny::red_bytes<MB>();
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
