// Test hooks: single kernels of the rollout path behind a C ABI.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "kernels.h"
#include "vla.h"
#include "vla_debug.h"

using namespace vla;

namespace {

// Split-K partials of vla_debug_skinny_noalloc: a file-scope device array that
// every GPU the library runs on holds until the process ends.  Host code never
// uses its name as an address: the device address is looked up once per device.
constexpr size_t kNoAllocScratchFloats = size_t(1) << 23;  // 32 MiB
__device__ __align__(256) float scratch[kNoAllocScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (looked up on the first call there).
int scratch_on_current_device(float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return set_error(VLA_EHIP, "hipGetDevice failed or device index out of range");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(VLA_EHIP, (std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e)).c_str());
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return VLA_OK;
}

}  // namespace

extern "C" {

int vla_debug_gemm(const void* A, const void* W, int32_t M, int32_t N, int32_t K, float* C, void* stream) {
  if (!A || !W || !C || M < 0 || N < 0 || K <= 0) return VLA_EINVAL;
  GemmArgs g{};
  g.A = static_cast<const bf16_t*>(A);
  g.W = static_cast<const bf16_t*>(W);
  g.M = M;
  g.N = N;
  g.K = K;
  g.C = C;
  g.ldc = N;
  return launch_gemm(g, kEpiStoreF32, static_cast<hipStream_t>(stream)) == hipSuccess ? VLA_OK : VLA_EHIP;
}

int vla_debug_skinny(const void* A, const void* W, int32_t M, int32_t N, int32_t K, int32_t workgroups,
                     float* scratch, float* C, void* stream) {
  if (!A || !W || !C || !scratch || M < 0 || N <= 0 || K <= 0 || workgroups < 1) return VLA_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const SkinnyPlan p = skinny_plan(N, K, workgroups, 16);
  SkinnyArgs a{static_cast<const bf16_t*>(A), M, static_cast<const bf16_t*>(W), N, K, scratch};
  if (launch_skinny(a, p, s) != hipSuccess) return VLA_EHIP;
  return launch_reduce_sum(scratch, p, C, M, N, s) == hipSuccess ? VLA_OK : VLA_EHIP;
}

int vla_debug_skinny_noalloc(const void* A, const void* W, int32_t M, int32_t N, int32_t K, int32_t workgroups,
                             float* C, void* stream) {
  if (!A || !W || !C || M < 0 || N <= 0 || K <= 0 || workgroups < 1)
    return set_error(VLA_EINVAL, "NULL pointer or non-positive size");
  if (M > 128 || N % 64 != 0 || K % 256 != 0)
    return set_error(VLA_EUNSUPPORTED, "needs M <= 128, N % 64 == 0, K % 256 == 0");
  // the plan of vla_debug_skinny, so that both give the same bits
  const SkinnyPlan p = skinny_plan(N, K, workgroups, 16);
  if ((size_t)p.slots * M * N > kNoAllocScratchFloats)
    return set_error(VLA_ESHAPE, "partial sums exceed the fixed scratch: slots * M * N must be <= 2^23 floats");
  float* part = nullptr;
  const int rc = scratch_on_current_device(&part);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  SkinnyArgs a{static_cast<const bf16_t*>(A), M, static_cast<const bf16_t*>(W), N, K, part};
  hipError_t e = launch_skinny(a, p, s);
  if (e == hipSuccess) e = launch_reduce_sum(part, p, C, M, N, s);
  if (e != hipSuccess) return set_error(VLA_EHIP, hipGetErrorString(e));
  return VLA_OK;
}

int vla_debug_pack_frag(const void* src, int32_t rows, int32_t K, int32_t ld, void* dst, void* stream) {
  if (!src || !dst || rows < 0 || K <= 0 || K % 32 != 0 || ld < K) return VLA_EINVAL;
  PackArgs pa{static_cast<bf16_t*>(dst), rows, K, static_cast<const bf16_t*>(src), nullptr, ld, rows, K, kPackRows, 0};
  return launch_pack_frag(pa, static_cast<hipStream_t>(stream)) == hipSuccess ? VLA_OK : VLA_EHIP;
}

int vla_debug_sample(const float* z, int32_t B, int32_t A, int32_t n_actions, int32_t step, int32_t action_begin,
                     const float* gumbel, float temperature, int32_t* tokens, int32_t* next_tok, float* logp,
                     float* entropy, float* logits_out, void* stream) {
  if (!z || !gumbel || !tokens || !next_tok || !logp || B < 0 || A < 1 || A > 256 || step < 0 ||
      step >= n_actions || !(temperature > 0.f))
    return VLA_EINVAL;
  SamplerArgs sa{};
  sa.z = z; sa.A = A; sa.temperature = temperature; sa.gumbel = gumbel; sa.step = step; sa.n_actions = n_actions;
  sa.action_begin = action_begin; sa.tokens = tokens; sa.next_tok = next_tok; sa.logp = logp; sa.entropy = entropy;
  sa.logits_out = logits_out; sa.rows = B;
  return launch_sampler(sa, static_cast<hipStream_t>(stream)) == hipSuccess ? VLA_OK : VLA_EHIP;
}

}  // extern "C"
