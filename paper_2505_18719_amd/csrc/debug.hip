// Test hooks: single kernels of the rollout path behind a C ABI.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "vla.h"
#include "vla_debug.h"

using namespace vla;

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
